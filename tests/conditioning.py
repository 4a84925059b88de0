"""CPU emulation of fp32-accumulating implementations of the partition forward.

Test infrastructure, CPU only.  It is neither the oracle (which sums in fp64
and so defines the reference) nor the GPU path: it reproduces the *class* of
arithmetic the GPU kernels belong to, so that the end-to-end error of a
correct implementation of that class can be measured on the CPU.

Every "order" below is a correct implementation of the same fused layer
(convolution + BN + residual + activation, one storage rounding per stored
output, the partition forward of the paper's MILP inputs, App. A.1, C_ldbij).
They differ only in how the fp32 sums are formed:

  * products of the stored operands are exact (16-bit x 16-bit fits fp32;
    fp32 x fp32 is formed in fp64);
  * a "chunk" of consecutive reduction terms, in (kh, kw, ci) order, is summed
    exactly and then added into an fp32 accumulator with one rounding (the
    k-step of a matrix-core instruction);
  * the reduction may be cut into ``split`` contiguous ranges whose fp32 sums
    are added in range order (split-K);
  * ``reverse`` adds the chunks last to first, ``perm`` in a seeded random
    order (any order of the fp32 additions is a correct implementation);
  * BN is an fp32 per-channel scale and shift applied with one rounding (a
    fused multiply-add), the residual is added in fp32, then the activation
    and one rounding to the storage dtype;
  * depthwise layers take their nine taps in (kh, kw) order as fp32 fused
    multiply-adds; global average pooling sums in fp32 and scales by 1/HW;
    softmax runs in fp32.

Where storage rounding turns a last-bit difference of the fp32 sum into a
one-ulp difference of a stored 16-bit activation, a deep network can amplify
it; comparing several orders with the oracle measures how far a correct
fp32-accumulating implementation lands from the fp64 reference.
"""
from dataclasses import dataclass
from typing import Dict, List, Optional, Tuple

import numpy as np
import torch


@dataclass(frozen=True)
class Order:
    """How the fp32 sums of a reduction are formed."""
    chunk: int = 32
    split: int = 1
    reverse: bool = False
    perm: int = -1          # >= 0: chunks of each range added in a seeded random order

    @property
    def name(self) -> str:
        s = f"chunk{self.chunk}"
        if self.split > 1:
            s += f"-split{self.split}"
        if self.reverse:
            s += "-rev"
        if self.perm >= 0:
            s += f"-perm{self.perm}"
        return s


# An ensemble of orders; every member is a correct fp32-accumulating
# implementation of the same layer functions.
ENSEMBLE = (Order(32), Order(32, 2), Order(32, 4), Order(8), Order(64), Order(128),
            Order(32, 1, True))
# ... and the same with 24 seeded random chunk orders (one and two K ranges)
ENSEMBLE_WIDE = ENSEMBLE + tuple(Order(32, sp, perm=k) for k in range(12) for sp in (1, 2))


def _f32(a: np.ndarray) -> np.ndarray:
    return np.asarray(a, dtype=np.float64).astype(np.float32)


def store(x32: np.ndarray, dtype: str) -> np.ndarray:
    """Round fp32 values to the storage dtype (RNE), kept as float32."""
    x32 = np.ascontiguousarray(x32, dtype=np.float32)
    if dtype == "f32":
        return x32
    t = {"f16": torch.float16, "bf16": torch.bfloat16}[dtype]
    return torch.from_numpy(x32).to(t).to(torch.float32).numpy()


def _fold_bn(L, p: Dict[str, np.ndarray], co: int) -> Tuple[np.ndarray, np.ndarray]:
    """fp32 per-channel scale and shift: (acc + b - mean)/sqrt(var + eps)*gamma + beta."""
    b0 = p["bias"].astype(np.float64) if "bias" in p else np.zeros(co)
    if L.bn:
        s = p["bn_gamma"].astype(np.float64) / np.sqrt(p["bn_var"].astype(np.float64) + 1e-5)
        t = p["bn_beta"].astype(np.float64) + (b0 - p["bn_mean"].astype(np.float64)) * s
        return _f32(s), _f32(t)
    return np.ones(co, np.float32), _f32(b0)


def _reduce(cols: np.ndarray, wk: np.ndarray, order: Order) -> np.ndarray:
    """fp32 sums of cols[M, K] @ wk[K, Co] formed in the given order."""
    cols_t = torch.from_numpy(np.ascontiguousarray(cols, dtype=np.float64))
    wk_t = torch.from_numpy(np.ascontiguousarray(wk, dtype=np.float64))
    M, K = cols_t.shape
    Co = wk_t.shape[1]
    nch = (K + order.chunk - 1) // order.chunk
    bounds = [round(nch * i / order.split) for i in range(order.split + 1)]
    total = None
    for sp in range(order.split):
        idx = list(range(bounds[sp], bounds[sp + 1]))
        if order.reverse:
            idx.reverse()
        if order.perm >= 0:
            idx = [int(i) for i in np.random.default_rng([order.perm, M, K, Co, sp]).permutation(idx)]
        acc = torch.zeros((M, Co), dtype=torch.float32)
        for c in idx:
            k0, k1 = c * order.chunk, min(K, (c + 1) * order.chunk)
            part = cols_t[:, k0:k1] @ wk_t[k0:k1]          # fp64: exact chunk sum
            acc = (acc.to(torch.float64) + part).to(torch.float32)
        total = acc if total is None else (total.to(torch.float64) + acc).to(torch.float32)
    return total.numpy()


def _im2col(x_nhwc: np.ndarray, k: int, s: int, p: int) -> Tuple[np.ndarray, int, int]:
    """[M, k*k*C] fp64 columns in (kh, kw, ci) order."""
    N, H, W, C = x_nhwc.shape
    Ho, Wo = (H + 2 * p - k) // s + 1, (W + 2 * p - k) // s + 1
    xp = np.zeros((N, H + 2 * p, W + 2 * p, C), np.float64)
    xp[:, p:p + H, p:p + W] = x_nhwc
    cols = np.empty((N, Ho, Wo, k, k, C), np.float64)
    for kh in range(k):
        for kw in range(k):
            cols[:, :, :, kh, kw] = xp[:, kh:kh + s * (Ho - 1) + 1:s, kw:kw + s * (Wo - 1) + 1:s]
    return cols.reshape(N * Ho * Wo, k * k * C), Ho, Wo


def _epilogue(acc: np.ndarray, sc: np.ndarray, sh: np.ndarray, res: Optional[np.ndarray],
              act: str) -> np.ndarray:
    a = torch.from_numpy(np.ascontiguousarray(acc))
    # acc * scale + shift with one rounding (a fused multiply-add): the fp32
    # product is exact in fp64
    v = (a.to(torch.float64) * torch.from_numpy(sc).to(torch.float64)
         + torch.from_numpy(sh).to(torch.float64)).to(torch.float32)
    if res is not None:
        v = v + torch.from_numpy(np.ascontiguousarray(res, dtype=np.float32))
    if act == "relu":
        v = v.clamp_min(0.0)
    elif act == "relu6":
        v = v.clamp(0.0, 6.0)
    return v.numpy()


def conv_layer(L, p, x_nchw: np.ndarray, res_nchw: Optional[np.ndarray], dtype: str,
               order: Order) -> np.ndarray:
    x = np.ascontiguousarray(x_nchw.transpose(0, 2, 3, 1)).astype(np.float64)
    N, H, W, C = x.shape
    w = p["weight"].astype(np.float64)
    sc, sh = _fold_bn(L, p, L.c_out)
    if L.groups == 1:
        cols, Ho, Wo = _im2col(x, L.k, L.stride, L.pad)
        wk = np.ascontiguousarray(w.transpose(2, 3, 1, 0).reshape(-1, L.c_out))
        acc = _reduce(cols, wk, order)
    elif L.groups == C == L.c_out:
        # depthwise: nine fp32 fused multiply-adds per output, taps in (kh, kw) order.
        # A product of two 16-bit values is exact in fp32, so for 16-bit storage
        # the fp32 add after it is the fused multiply-add's one rounding.
        k, s, pd = L.k, L.stride, L.pad
        Ho, Wo = (H + 2 * pd - k) // s + 1, (W + 2 * pd - k) // s + 1
        wide = torch.float64 if dtype == "f32" else torch.float32
        xp = torch.zeros((N, H + 2 * pd, W + 2 * pd, C), dtype=wide)
        xp[:, pd:pd + H, pd:pd + W] = torch.from_numpy(x).to(wide)
        wt = torch.from_numpy(w[:, 0]).to(wide)
        acc = torch.zeros((N, Ho, Wo, C), dtype=torch.float32)
        for kh in range(k):
            for kw in range(k):
                tap = xp[:, kh:kh + s * (Ho - 1) + 1:s, kw:kw + s * (Wo - 1) + 1:s]
                acc = (acc.to(wide) + tap * wt[:, kh, kw]).to(torch.float32)
        acc = acc.reshape(-1, C).numpy()
    else:
        raise ValueError("grouped convolution other than depthwise")
    res = None
    if res_nchw is not None:
        res = np.ascontiguousarray(res_nchw.transpose(0, 2, 3, 1)).reshape(-1, L.c_out)
    y = store(_epilogue(acc, sc, sh, res, L.act), dtype)
    return np.ascontiguousarray(y.reshape(N, Ho, Wo, L.c_out).transpose(0, 3, 1, 2))


def maxpool_layer(L, x: np.ndarray) -> np.ndarray:
    N, C, H, W = x.shape
    k, s, pd = L.k, L.stride, L.pad
    Ho, Wo = (H + 2 * pd - k) // s + 1, (W + 2 * pd - k) // s + 1
    xp = np.full((N, C, H + 2 * pd, W + 2 * pd), -np.inf, np.float32)
    xp[:, :, pd:pd + H, pd:pd + W] = x
    y = np.full((N, C, Ho, Wo), -np.inf, np.float32)
    for kh in range(k):
        for kw in range(k):
            y = np.maximum(y, xp[:, :, kh:kh + s * (Ho - 1) + 1:s, kw:kw + s * (Wo - 1) + 1:s])
    return y


def gap_layer(x: np.ndarray, dtype: str) -> np.ndarray:
    N, C, H, W = x.shape
    acc = np.zeros((N, C), np.float32)
    for t in range(H * W):
        acc = (acc + x[:, :, t // W, t % W]).astype(np.float32)
    return store((acc * np.float32(1.0 / (H * W))).astype(np.float32), dtype).reshape(N, C, 1, 1)


def fc_layer(L, p, x: np.ndarray, dtype: str, order: Order) -> np.ndarray:
    N = x.shape[0]
    xf = x.reshape(N, -1).astype(np.float64)                  # (c, h, w) flattening
    wk = np.ascontiguousarray(p["weight"].astype(np.float64).T)
    acc = _reduce(xf, wk, order)
    sc, sh = np.ones(L.c_out, np.float32), _f32(p["bias"]) if "bias" in p else np.zeros(L.c_out, np.float32)
    z = (acc.astype(np.float64) * sc + sh).astype(np.float32)
    if L.op == "fc_softmax":
        z = z - z.max(axis=1, keepdims=True)
        e = np.exp(z).astype(np.float32)
        return (e / e.sum(axis=1, dtype=np.float32, keepdims=True)).astype(np.float32)
    if L.act == "relu":
        z = np.maximum(z, np.float32(0))
    return store(z, dtype)


def layer(L, p, src: np.ndarray, res: Optional[np.ndarray], dtype: str,
          order: Order = Order()) -> np.ndarray:
    """One fused layer on its source (and residual) tensor, NCHW."""
    if L.op == "conv":
        return conv_layer(L, p, src, res, dtype, order)
    if L.op == "maxpool":
        return maxpool_layer(L, src)
    if L.op == "gap":
        return gap_layer(src, dtype)
    if L.op in ("fc", "fc_softmax"):
        return fc_layer(L, p, src, dtype, order)
    raise ValueError(L.op)


def forward(layers: List, params: Dict[int, Dict[str, np.ndarray]], begin: int, end: int,
            x: np.ndarray, dtype: str, order: Order = Order(),
            keep: bool = False):
    """Layers [begin, end) on x (NCHW float32 holding dtype values)."""
    outs = {begin - 1: np.ascontiguousarray(x, np.float32)}
    for i in range(begin, end):
        L = layers[i]
        res = outs[L.res_src] if L.res_src >= 0 else None
        outs[i] = layer(L, params.get(i, {}), outs[L.src], res, dtype, order)
        if not keep:
            for j in list(outs):
                if j != i and not any(layers[t].src == j or layers[t].res_src == j
                                      for t in range(i + 1, end)):
                    del outs[j]
    return (outs[end - 1], outs) if keep else outs[end - 1]


def rel_inf(got: np.ndarray, ref: np.ndarray) -> float:
    g = np.asarray(got, np.float64).reshape(-1)
    r = np.asarray(ref, np.float64).reshape(-1)
    return float(np.abs(g - r).max() / max(np.abs(r).max(), 1e-30))


def argmax_rows(p: np.ndarray) -> np.ndarray:
    return np.asarray(p).reshape(p.shape[0], -1).argmax(axis=1)


@dataclass
class EnsembleResult:
    order: str
    rel_inf: float
    argmax_agree: np.ndarray       # per image, against the oracle
    prefix: Dict[int, float]       # layer -> rel_inf of that layer's output vs the oracle's


def ensemble(layers, params, begin, end, x, dtype, ref_outs, orders=ENSEMBLE,
             prefix_layers=()) -> List[EnsembleResult]:
    """End-to-end error of each order against the oracle's stored outputs
    ``ref_outs`` (layer -> array, from the oracle with keep=True)."""
    out = []
    ref = ref_outs[end - 1]
    for o in orders:
        got, outs = forward(layers, params, begin, end, x, dtype, o, keep=True)
        pre = {j: rel_inf(outs[j], ref_outs[j]) for j in prefix_layers}
        out.append(EnsembleResult(o.name, rel_inf(got, ref),
                                  argmax_rows(got) == argmax_rows(ref), pre))
    return out
