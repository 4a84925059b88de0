"""Parity of the five workloads at their full shapes and batch sizes,
through the C ABI, against the CPU oracle on the same seeded inputs.

Checks per workload:
 * segment parity: the range is cut at every point where exactly one feature
   map crosses (every valid partition boundary); each minimal segment is run
   on the GPU from the oracle's own stored input and compared element by
   element with the oracle's output of that segment, within a few storage
   roundings (SEG_TOL).  This pins every kernel launch at its real shape and
   batch.
 * end to end: the whole range on the GPU vs the oracle.  Tolerance: infinity-
   norm relative error <= 2e-2 for fp16/bf16 storage, 1e-4 for fp32, argmax of
   the class probabilities bit-exact.
 * two bf16 ranges amplify one-ulp storage differences through depth
   (tests/test_conditioning.py): on MobileNetV2 at batch 32 every fp32
   summation order of a correct implementation misses 2e-2 (7.2e-2 .. 9.0e-2,
   2-4 argmax flips), and on ResNet-50 [25, 56) at batch 8 correct orders
   land anywhere from 5.3e-3 to 5.1e-2 (a quarter of them above 2e-2).  Their
   2e-2 tests are expected failures with that reason; in addition the GPU
   must land inside the envelope of those correct orders (error no larger
   than the worst order's, no more argmax flips than the worst order's).
Where the oracle cannot afford the whole batch it checks sampled images of
the batch the GPU ran (each image's output is independent of the others)."""
import functools

import numpy as np
import pytest

import oracle
import workloads as W

from gpu_util import gpu_forward, rel_inf, argmax_rows

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "f16": 2e-2, "bf16": 2e-2}
# a segment is one to four fused layers, each rounding its output once
SEG_TOL = {"f32": 1e-5, "f16": 2.0 ** -9, "bf16": 2.0 ** -7}


@functools.lru_cache(maxsize=None)
def _setup(name):
    wl = W.workload(name)
    m = wl.build_model()
    return wl, m, wl.params(m)


@functools.lru_cache(maxsize=None)
def _oracle_image(name, index):
    wl, m, P = _setup(name)
    x = wl.input(index + 1)[index:index + 1]
    return oracle.forward(m.layers, P, wl.begin, wl.end, x, wl.dtype)[0]


def boundaries(layers, begin, end):
    """Points j in (begin, end) where a partition may start: every layer of
    [j, end) reads only layers >= j - 1."""
    out = []
    for j in range(begin + 1, end):
        if all(L.src >= j - 1 and (L.res_src == -1 or L.res_src >= j - 1)
               for L in layers[j:end]):
            out.append(j)
    return out


def _partition(m, P, a, b, dtype, batch):
    from paper_2507_18748_amd import Partition
    return Partition(m.layers, P, (m.in_c, m.in_h, m.in_w), a, b, dtype, max_batch=batch)


def _end_to_end(name, batch, sample=None):
    wl, m, P = _setup(name)
    x = wl.input(batch)
    print(f"[config-parity] {name} [{wl.begin},{wl.end}) {wl.dtype} batch={batch}", flush=True)
    with _partition(m, P, wl.begin, wl.end, wl.dtype, batch) as part:
        got = gpu_forward(part, x)
    if sample is None:
        ref = oracle.forward(m.layers, P, wl.begin, wl.end, x, wl.dtype)
        got = got.reshape(ref.shape)
    else:
        ref = np.stack([_oracle_image(name, i) for i in sample])
        got = got.reshape((batch,) + ref.shape[1:])[list(sample)]
    e = rel_inf(got, ref)
    r = ref.reshape(ref.shape[0], -1)
    top2 = np.sort(r, axis=1)[:, -2:]
    gap = top2[:, 1] - top2[:, 0]
    agree = argmax_rows(got) == argmax_rows(ref)
    print(f"    rel_inf = {e:.3e} (tol {TOL[wl.dtype]:.0e}); argmax {int(agree.sum())}/{len(agree)}; "
          f"min top1-top2 gap {float(gap.min()):.3e}", flush=True)
    return e, agree, gap, float(np.abs(r).max())


def _check_end_to_end(name, batch, sample=None):
    wl = W.workload(name)
    e, agree, gap, _ = _end_to_end(name, batch, sample)
    assert e <= TOL[wl.dtype]
    assert agree.all()


def _check_within_fp32_orders(name, orders):
    """The GPU's end-to-end error against the envelope of correct
    fp32-accumulating implementations that differ only in summation order."""
    import conditioning as C
    wl, m, P = _setup(name)
    e, agree, _, _ = _end_to_end(name, wl.batch)
    x = wl.input(wl.batch)
    _, outs = oracle.forward(m.layers, P, wl.begin, wl.end, x, wl.dtype, keep=True)
    res = C.ensemble(m.layers, P, wl.begin, wl.end, x, wl.dtype, outs, orders)
    errs = [r.rel_inf for r in res]
    flips = [int((~r.argmax_agree).sum()) for r in res]
    print(f"    {len(res)} fp32 orders: rel_inf {min(errs):.3e} .. {max(errs):.3e}, argmax flips "
          f"{min(flips)} .. {max(flips)}; GPU {e:.3e}, {int((~agree).sum())} flips", flush=True)
    assert e <= max(errs)
    assert int((~agree).sum()) <= max(flips)


def _check_segments(name, batch, sample=None):
    """Element-wise parity of every minimal segment from the oracle's input."""
    wl, m, P = _setup(name)
    x = wl.input(batch)
    if sample is not None:
        x = x[list(sample)]
    _, outs = oracle.forward(m.layers, P, wl.begin, wl.end, x, wl.dtype, keep=True)
    cuts = [wl.begin] + boundaries(m.layers, wl.begin, wl.end) + [wl.end]
    worst = 0.0
    for a, b in zip(cuts[:-1], cuts[1:]):
        with _partition(m, P, a, b, wl.dtype, x.shape[0]) as part:
            got = gpu_forward(part, outs[a - 1])
        ref = outs[b - 1]
        got = got.reshape(ref.shape)
        if m.layers[a].op == "maxpool" and b == a + 1:
            np.testing.assert_array_equal(got, ref)       # a max introduces no rounding
            e = 0.0
        else:
            e = rel_inf(got, ref)
        worst = max(worst, e)
        print(f"    segment [{a},{b}) {m.layers[a].name}..{m.layers[b - 1].name}: rel_inf {e:.2e}",
              flush=True)
        assert e <= SEG_TOL[wl.dtype], f"segment [{a},{b}) rel_inf {e:.3e}"
        if m.layers[b - 1].op == "fc_softmax":
            assert (argmax_rows(got) == argmax_rows(ref)).all()
    print(f"[segment-parity] {name} batch {x.shape[0]}: {len(cuts) - 1} segments, "
          f"worst rel_inf {worst:.2e}", flush=True)


def _check_segments_at_batch(name, batch, sample):
    """Element-wise parity of every minimal segment in the launch configuration
    of `batch` (the plans the benchmark times), on sampled images: the oracle
    computes the sampled images only; the other rows of each segment's input
    repeat the first sample (each image is computed independently)."""
    wl, m, P = _setup(name)
    xs = wl.input(batch)[list(sample)]
    _, outs = oracle.forward(m.layers, P, wl.begin, wl.end, xs, wl.dtype, keep=True)
    cuts = [wl.begin] + boundaries(m.layers, wl.begin, wl.end) + [wl.end]
    rows = list(sample)
    worst = 0.0
    for a, b in zip(cuts[:-1], cuts[1:]):
        src = outs[a - 1]
        xin = np.repeat(src[:1], batch, axis=0)
        xin[rows] = src
        with _partition(m, P, a, b, wl.dtype, batch) as part:
            got = gpu_forward(part, xin)
        ref = outs[b - 1]
        got = got.reshape((batch,) + ref.shape[1:])[rows]
        e = rel_inf(got, ref)
        worst = max(worst, e)
        print(f"    segment [{a},{b}) {m.layers[a].name}..{m.layers[b - 1].name} at batch {batch}: "
              f"rel_inf {e:.2e}", flush=True)
        assert e <= SEG_TOL[wl.dtype], f"segment [{a},{b}) rel_inf {e:.3e}"
    print(f"[segment-parity] {name} batch {batch}, images {rows}: {len(cuts) - 1} segments, "
          f"worst rel_inf {worst:.2e}", flush=True)


# ---- end to end ----

def test_resnet18_stem_layer1_fp32_batch1():
    _check_end_to_end("resnet18_stem_layer1", 1)


def test_resnet50_layer4_head_bf16_batch8():
    _check_end_to_end("resnet50_layer4_head", 8)


@pytest.mark.xfail(strict=False, reason=(
    "whether a correct fp32-accumulating implementation meets 2e-2 on ResNet-50 [25,56) at "
    "batch 8 (seed 2) depends on its summation order only: 31 orders land at 5.3e-3 .. 5.1e-2, "
    "26% above 2e-2 (tests/test_conditioning.py); the GPU measured 3.2e-2, 8/8 argmax"))
def test_resnet50_layer3_layer4_head_bf16_batch8():
    _check_end_to_end("resnet50_layer3_layer4_head", 8)


def test_resnet50_layer3_layer4_head_within_fp32_orders():
    import conditioning as C
    _check_within_fp32_orders("resnet50_layer3_layer4_head", C.ENSEMBLE_WIDE)


def test_vgg16_fp16_batch16():
    _check_end_to_end("vgg16", 16, sample=(0, 7, 15))


@pytest.mark.xfail(strict=True, reason=(
    "no fp32-accumulating implementation meets 2e-2 on MobileNetV2 at batch 32 (seed 4): every "
    "summation order lands at 7.2e-2 .. 9.0e-2 with 2-4 argmax flips in 32 "
    "(tests/test_conditioning.py); the GPU measured 6.4e-2 .. 7.0e-2 with 2-3 flips"))
def test_mobilenet_v2_bf16_batch32():
    _check_end_to_end("mobilenet_v2", 32)


def test_mobilenet_v2_within_fp32_orders():
    import conditioning as C
    _check_within_fp32_orders("mobilenet_v2", C.ENSEMBLE)


@pytest.mark.parametrize("batch", [1, 4, 16, 64])
def test_resnet152_fp16(batch):
    _check_end_to_end("resnet152", batch, sample=sorted({0, batch - 1}))


# ---- segment parity at full shape ----

def test_segments_resnet18_stem_layer1():
    _check_segments("resnet18_stem_layer1", 1)


def test_segments_resnet50_layer3_layer4_head():
    _check_segments("resnet50_layer3_layer4_head", 8)


def test_segments_vgg16():
    _check_segments("vgg16", 16)


def test_segments_mobilenet_v2():
    _check_segments("mobilenet_v2", 32)


def test_segments_resnet152_batch16():
    _check_segments("resnet152", 16)


def test_segments_resnet152_batch64_sampled():
    """The benchmark's configuration (ResNet-152 fp16 at batch 64), segment by
    segment, on the first and last image."""
    _check_segments_at_batch("resnet152", 64, (0, 63))
