"""Pins of the CPU oracle against what the mathematics fixes, independent of
the oracle's own code: brute-force nested loops on tiny tensors, closed
forms (1x1 convolution = matrix product, delta kernel = identity, FC = 1x1
convolution on a 1x1 map), float64 library routines (numpy, torch CPU), exact
rounding by enumeration, and invariants (softmax, composition of ranges,
batch independence).  A dropped term, wrong sign, wrong index or transposed
operand in the oracle fails at least one of these."""
import itertools
import math

import numpy as np
import pytest

import oracle
import workloads as W
from workloads.zoo import Layer

F32_REL = 2.0 ** -23   # one fp32 rounding of the oracle's fp64 result


def brute_conv(x, w, stride, pad, groups, bias=None, bn=None, eps=1e-5, res=None,
               act="none"):
    """Textbook cross-correlation with plain Python floats (fp64)."""
    N, C, H, Wd = x.shape
    Co, cig, KH, KW = w.shape
    Ho = (H + 2 * pad - KH) // stride + 1
    Wo = (Wd + 2 * pad - KW) // stride + 1
    cog = Co // groups
    y = np.zeros((N, Co, Ho, Wo))
    for n, co, ho, wo in itertools.product(range(N), range(Co), range(Ho), range(Wo)):
        g = co // cog
        s = 0.0
        for cl, kh, kw in itertools.product(range(cig), range(KH), range(KW)):
            hi, wi = ho * stride - pad + kh, wo * stride - pad + kw
            if 0 <= hi < H and 0 <= wi < Wd:
                s += float(x[n, g * cig + cl, hi, wi]) * float(w[co, cl, kh, kw])
        if bias is not None:
            s += float(bias[co])
        if bn is not None:
            gm, bt, mu, var = (float(t[co]) for t in bn)
            s = (s - mu) / math.sqrt(var + eps) * gm + bt
        if res is not None:
            s += float(res[n, co, ho, wo])
        if act == "relu":
            s = max(s, 0.0)
        elif act == "relu6":
            s = min(max(s, 0.0), 6.0)
        y[n, co, ho, wo] = s
    return y


def close_f32(got, ref64, slack=4.0):
    """got is ref64 rounded once to fp32 (up to fp64 summation order)."""
    ref64 = np.asarray(ref64, dtype=np.float64)
    tol = slack * F32_REL * np.maximum(np.abs(ref64), 1e-30) + 1e-300
    np.testing.assert_array_less(np.abs(got.astype(np.float64) - ref64), tol)


# ---------------------------------------------------------------- rounding

def test_round_f32_matches_numpy_cast():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-40, 38, 20000),
                        [0.0, -0.0, 1e-46, -1e-46, 3.4028235e38, 3.5e38, -3.5e38]])
    with np.errstate(over="ignore"):
        want = x.astype(np.float32)
    np.testing.assert_array_equal(oracle.round_to(x, "f32"), want)


def test_round_f16_matches_numpy_cast():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(20000) * 2.0 ** rng.integers(-30, 17, 20000)
    # exact halfway points between consecutive fp16 values, both parities
    h = np.arange(0x0001, 0x7bff, 37, dtype=np.uint16).view(np.float16).astype(np.float64)
    h_next = (np.arange(0x0001, 0x7bff, 37, dtype=np.uint16) + 1).view(np.float16).astype(np.float64)
    x = np.concatenate([x, (h + h_next) / 2, -(h + h_next) / 2,
                        [65504.0, 65519.99, 65520.0, -65520.0, 2.0 ** -25, 3 * 2.0 ** -26]])
    with np.errstate(over="ignore"):
        want = x.astype(np.float16).astype(np.float32)
    np.testing.assert_array_equal(oracle.round_to(x, "f16"), want)


def _all_bf16_finite():
    bits = np.arange(0, 0x7f80, dtype=np.uint32)        # +0 .. largest finite
    vals = (bits << 16).view(np.float32).astype(np.float64)
    return np.concatenate([-vals[:0:-1], vals]), np.concatenate([bits[:0:-1], bits])


def test_round_bf16_is_nearest_even_by_enumeration():
    vals, bits = _all_bf16_finite()
    rng = np.random.default_rng(2)
    x = rng.standard_normal(3000) * 2.0 ** rng.integers(-130, 127, 3000)
    mids = (vals[1:] + vals[:-1]) / 2                     # exact ties
    x = np.concatenate([x, rng.choice(mids, 2000), [1e-45, 3.0e38, -3.0e38]])
    got = oracle.round_to(x, "bf16").astype(np.float64)
    idx = np.clip(np.searchsorted(vals, x), 1, len(vals) - 1)
    lo, hi = vals[idx - 1], vals[idx]
    dlo, dhi = x - lo, hi - x
    pick_hi = (dhi < dlo) | ((dhi == dlo) & ((bits[idx] & 1) == 0))
    want = np.where(pick_hi, hi, lo)
    np.testing.assert_array_equal(got, want)


def test_round_overflow_and_specials():
    assert oracle.round_to([7e38], "bf16")[0] == np.inf      # beyond max + half ulp
    assert oracle.round_to([-1e6], "f16")[0] == -np.inf
    assert np.isnan(oracle.round_to([np.nan], "f16")[0])
    assert oracle.round_to([2.0 ** -24], "f16")[0] == 2.0 ** -24   # smallest subnormal kept


# ---------------------------------------------------------------- convolution

CASES = [
    # N, C, H, W, Co, k, s, p, groups
    (2, 3, 5, 6, 4, 3, 1, 1, 1),
    (1, 4, 6, 5, 4, 3, 2, 1, 4),      # depthwise
    (2, 4, 6, 6, 6, 2, 2, 0, 2),      # grouped
    (1, 2, 5, 5, 3, 1, 1, 0, 1),
    (2, 4, 6, 6, 4, 1, 2, 0, 1),      # strided 1x1 (downsample)
    (1, 3, 6, 6, 2, 3, 2, 2, 1),      # pad 2
    (1, 2, 4, 4, 2, 4, 1, 0, 1),      # window = input
]


@pytest.mark.parametrize("case", CASES)
def test_conv_brute_force(case):
    N, C, H, Wd, Co, k, s, p, g = case
    rng = np.random.default_rng(hash(case) % 2 ** 32)
    x = rng.standard_normal((N, C, H, Wd)).astype(np.float32)
    w = rng.standard_normal((Co, C // g, k, k)).astype(np.float32)
    bias = rng.standard_normal(Co).astype(np.float32)
    bn = (rng.uniform(0.5, 1.5, Co).astype(np.float32), rng.standard_normal(Co).astype(np.float32),
          rng.standard_normal(Co).astype(np.float32), rng.uniform(0.5, 1.5, Co).astype(np.float32))
    Ho = (H + 2 * p - k) // s + 1
    res = rng.standard_normal((N, Co, Ho, Ho if H == Wd else (Wd + 2 * p - k) // s + 1)).astype(np.float32)
    for kw in (dict(), dict(bias=bias), dict(bn=bn), dict(bn=bn, res=res, act="relu"),
               dict(bias=bias, act="relu6")):
        ref = brute_conv(x, w, s, p, g, **kw)
        got = oracle.conv2d(x, w, s, p, g, **kw)
        assert got.shape == ref.shape
        close_f32(got, ref)


def test_conv_1x1_equals_matmul():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((3, 16, 7, 5)).astype(np.float32)
    w = rng.standard_normal((8, 16, 1, 1)).astype(np.float32)
    ref = np.einsum("oc,nchw->nohw", w[:, :, 0, 0].astype(np.float64), x.astype(np.float64))
    close_f32(oracle.conv2d(x, w), ref)


def test_delta_kernel_is_identity_bitwise():
    rng = np.random.default_rng(4)
    x = W.to_dtype_values(rng.standard_normal((2, 5, 7, 6)), "f16")
    k, p = 3, 1
    w = np.zeros((5, 5, k, k), dtype=np.float32)
    for c in range(5):
        w[c, c, p, p] = 1.0
    np.testing.assert_array_equal(oracle.conv2d(x, w, 1, p, dtype="f16"), x)


def test_bn_fold_equivalence():
    """Unfolded BN equals conv(x)*s + (beta - mean*s) with s = gamma/sqrt(var+eps)."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, 6, 5, 5)).astype(np.float32)
    w = rng.standard_normal((4, 6, 1, 1)).astype(np.float32)
    g, b, m, v = (rng.uniform(0.5, 1.5, 4), rng.standard_normal(4), rng.standard_normal(4),
                  rng.uniform(0.5, 1.5, 4))
    bn = tuple(t.astype(np.float32) for t in (g, b, m, v))
    g, b, m, v = (t.astype(np.float64) for t in bn)
    s = g / np.sqrt(v + 1e-5)
    conv = np.einsum("oc,nchw->nohw", w[:, :, 0, 0].astype(np.float64), x.astype(np.float64))
    ref = conv * s[None, :, None, None] + (b - m * s)[None, :, None, None]
    close_f32(oracle.conv2d(x, w, bn=bn), ref, slack=16)


def test_conv_matches_torch_float64():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(6)
    for (N, C, H, Co, k, s, p, g) in [(2, 8, 13, 12, 3, 2, 1, 1), (1, 6, 11, 6, 3, 1, 1, 6),
                                      (2, 3, 17, 8, 7, 2, 3, 1), (1, 8, 9, 4, 1, 2, 0, 1)]:
        x = rng.standard_normal((N, C, H, H)).astype(np.float32)
        w = rng.standard_normal((Co, C // g, k, k)).astype(np.float32)
        ref = torch.nn.functional.conv2d(torch.from_numpy(x).double(), torch.from_numpy(w).double(),
                                         stride=s, padding=p, groups=g).numpy()
        close_f32(oracle.conv2d(x, w, s, p, g), ref, slack=8)


# ---------------------------------------------------------------- pooling, fc, softmax

def brute_maxpool(x, k, s, p):
    N, C, H, Wd = x.shape
    Ho, Wo = (H + 2 * p - k) // s + 1, (Wd + 2 * p - k) // s + 1
    y = np.empty((N, C, Ho, Wo))
    for n, c, ho, wo in itertools.product(range(N), range(C), range(Ho), range(Wo)):
        vals = [x[n, c, ho * s - p + i, wo * s - p + j] for i in range(k) for j in range(k)
                if 0 <= ho * s - p + i < H and 0 <= wo * s - p + j < Wd]
        y[n, c, ho, wo] = max(vals)
    return y


@pytest.mark.parametrize("k,s,p", [(3, 2, 1), (2, 2, 0), (3, 1, 1), (3, 2, 0)])
def test_maxpool_brute_force_negative_inputs(k, s, p):
    rng = np.random.default_rng(7)
    x = -np.abs(rng.standard_normal((2, 3, 7, 8))).astype(np.float32) - 0.5  # padding must not win
    np.testing.assert_array_equal(oracle.maxpool2d(x, k, s, p), brute_maxpool(x, k, s, p))


def test_pool_and_fc_match_torch_float64():
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    rng = np.random.default_rng(8)
    x = rng.standard_normal((2, 5, 11, 11)).astype(np.float32)
    np.testing.assert_array_equal(
        oracle.maxpool2d(x, 3, 2, 1), F.max_pool2d(torch.from_numpy(x), 3, 2, 1).numpy())
    close_f32(oracle.global_avgpool(x), F.adaptive_avg_pool2d(torch.from_numpy(x).double(), 1).numpy())
    a = rng.standard_normal((3, 40)).astype(np.float32)
    w = rng.standard_normal((7, 40)).astype(np.float32)
    b = rng.standard_normal(7).astype(np.float32)
    ref = F.linear(torch.from_numpy(a).double(), torch.from_numpy(w).double(), torch.from_numpy(b).double())
    close_f32(oracle.linear(a, w, b), ref.numpy())
    close_f32(oracle.linear(a, w, b, act="relu"), F.relu(ref).numpy())
    close_f32(oracle.linear(a, w, b, softmax=True), F.softmax(ref, dim=1).numpy(), slack=8)


def test_fc_equals_1x1_conv_on_1x1_map_and_flatten_order():
    rng = np.random.default_rng(9)
    x = rng.standard_normal((2, 3, 4, 5)).astype(np.float32)
    w = rng.standard_normal((6, 60)).astype(np.float32)
    # FC over the (c, h, w) flattening == valid 4x5 convolution with weights viewed as OIHW
    via_conv = oracle.conv2d(x, w.reshape(6, 3, 4, 5))
    np.testing.assert_allclose(oracle.linear(x, w), via_conv.reshape(2, 6), rtol=4 * F32_REL)
    ref = x.reshape(2, -1).astype(np.float64) @ w.T.astype(np.float64)
    close_f32(oracle.linear(x, w), ref)


def test_softmax_invariants():
    rng = np.random.default_rng(10)
    a = rng.standard_normal((4, 64)).astype(np.float32)
    w = rng.standard_normal((100, 64)).astype(np.float32)
    b = rng.standard_normal(100).astype(np.float32)
    p = oracle.linear(a, w, b, softmax=True).astype(np.float64)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-6)
    assert (p > 0).all()
    p2 = oracle.linear(a, w, b + np.float32(3.0), softmax=True)   # shift invariance
    np.testing.assert_allclose(p2, p, rtol=1e-6)
    z = a.astype(np.float64) @ w.T.astype(np.float64) + b
    assert (p.argmax(1) == z.argmax(1)).all()


def test_global_avgpool_closed_form():
    x = np.arange(2 * 3 * 4 * 4, dtype=np.float32).reshape(2, 3, 4, 4)
    want = x.reshape(2, 3, -1).astype(np.float64).mean(-1)
    np.testing.assert_array_equal(oracle.global_avgpool(x)[:, :, 0, 0], want.astype(np.float32))


# ---------------------------------------------------------------- shapes, ranges

def test_shape_arithmetic():
    assert oracle.out_dim(224, 7, 2, 3) == 112
    assert oracle.out_dim(112, 3, 2, 1) == 56
    h = 224
    for _ in range(5):
        h = oracle.out_dim(h, 2, 2, 0)
    assert h == 7
    assert oracle.out_dim(7, 3, 2, 1) == 4 and oracle.out_dim(14, 1, 2, 0) == 7


def tiny_resnet():
    """Stem + maxpool + two bottleneck-like blocks (one with a strided
    projection) + gap + fc_softmax, small enough for the oracle in ms."""
    m = W.Model("tiny", 3, 20, 20)
    x = m.add(name="stem", op="conv", src=-1, c_in=3, c_out=8, k=3, stride=2, pad=1,
              act="relu", bn=True)
    x = m.add(name="pool", op="maxpool", src=x, c_in=8, c_out=8, k=3, stride=2, pad=1)
    r = m.add(name="b1.c1", op="conv", src=x, c_in=8, c_out=4, k=1, act="relu", bn=True)
    c = m.add(name="b1.c2", op="conv", src=r, c_in=4, c_out=4, k=3, stride=2, pad=1,
              act="relu", bn=True)
    d = m.add(name="b1.ds", op="conv", src=x, c_in=8, c_out=16, k=1, stride=2, bn=True)
    x = m.add(name="b1.c3", op="conv", src=c, c_in=4, c_out=16, k=1, act="relu", bn=True,
              res_src=d)
    r = m.add(name="b2.c1", op="conv", src=x, c_in=16, c_out=4, k=1, act="relu", bn=True)
    x = m.add(name="b2.c2", op="conv", src=r, c_in=4, c_out=16, k=3, pad=1, act="relu",
              bn=True, res_src=x)
    g = m.add(name="gap", op="gap", src=x, c_in=16, c_out=16)
    m.add(name="fc", op="fc_softmax", src=g, c_in=16, c_out=12, bias=True)
    return m


def test_composition_of_ranges_is_bitwise():
    m = tiny_resnet()
    P = W.model_params(m, 11, "bf16")
    x = W.partition_input((3, 20, 20), 2, 11, "bf16", "image")
    whole = oracle.forward(m.layers, P, 0, len(m.layers), x, "bf16")
    mid = oracle.forward(m.layers, P, 0, 6, x, "bf16")
    tail = oracle.forward(m.layers, P, 6, len(m.layers), mid, "bf16")
    np.testing.assert_array_equal(whole, tail)


def test_batch_independence_is_bitwise():
    m = tiny_resnet()
    P = W.model_params(m, 12, "f16")
    x = W.partition_input((3, 20, 20), 3, 12, "f16", "image")
    full = oracle.forward(m.layers, P, 0, len(m.layers), x, "f16")
    for i in range(3):
        one = oracle.forward(m.layers, P, 0, len(m.layers), x[i:i + 1], "f16")
        np.testing.assert_array_equal(full[i:i + 1], one)


def test_forward_rejects_residual_across_boundary():
    m = tiny_resnet()
    P = W.model_params(m, 13, "f32")
    x = np.zeros((1, 8, 5, 5), dtype=np.float32)
    with pytest.raises(ValueError):
        oracle.forward(m.layers, P, 3, len(m.layers), x, "f32")   # b1.ds reads layer 1


def test_forward_matches_layerwise_brute_force():
    """End-to-end walk of the graph: each stored output is the brute-force
    layer applied to the stored inputs, rounded to the dtype."""
    m = tiny_resnet()
    P = W.model_params(m, 14, "f16")
    x = W.partition_input((3, 20, 20), 1, 14, "f16", "image")
    _, outs = oracle.forward(m.layers, P, 0, len(m.layers), x, "f16", keep=True)
    for i, L in enumerate(m.layers):
        if L.op != "conv":
            continue
        src = outs[L.src]
        res = outs[L.res_src] if L.res_src >= 0 else None
        p = P[i]
        ref = brute_conv(src, p["weight"], L.stride, L.pad, L.groups,
                         bn=(p["bn_gamma"], p["bn_beta"], p["bn_mean"], p["bn_var"]),
                         res=res, act=L.act)
        want = ref.astype(np.float32).astype(np.float16).astype(np.float32)
        # fp64 -> fp16 direct vs via fp32 differ only on double-rounding ties
        np.testing.assert_allclose(outs[i], want, rtol=2.0 ** -10, atol=2.0 ** -24)
