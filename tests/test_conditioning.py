"""How far a correct fp32-accumulating implementation lands from the fp64
oracle on the two bf16 ranges whose end-to-end error the stored 16-bit
activations amplify: MobileNetV2 [0, 54) at batch 32 (seed 4) and ResNet-50
[25, 56) (layer3 + layer4 + head) at batch 8 (seed 2).

The emulation (tests/conditioning.py) forms the same layer functions as the
GPU kernels with fp32 sums and one storage rounding per layer; its members
differ only in the order of the fp32 additions.  These CPU tests

  * pin the emulation as a correct implementation: every layer, fed the
    oracle's own stored input, lands within one storage rounding of the
    oracle's output of that layer;
  * show that on MobileNetV2 no member meets the 2e-2 end-to-end bar (all
    land at 7.2e-2 or above with 2-4 argmax flips in 32), so the bar is out of
    reach for any fp32-accumulating implementation at this seed;
  * show that on ResNet-50 [25, 56) the members straddle 2e-2: whether a
    correct implementation passes depends on its summation order only.

The GPU tests (test_gpu_configs.py) bound the GPU by the same ensembles."""
import numpy as np
import pytest

import conditioning as C
import oracle
import workloads as W

LAYER_TOL = {"f32": 1e-5, "f16": 2.0 ** -9, "bf16": 2.0 ** -7}


def _setup(name):
    wl = W.workload(name)
    m = wl.build_model()
    P = wl.params(m)
    x = wl.input(wl.batch)
    ref, outs = oracle.forward(m.layers, P, wl.begin, wl.end, x, wl.dtype, keep=True)
    return wl, m, P, x, outs


@pytest.fixture(scope="module")
def mbv2():
    return _setup("mobilenet_v2")


@pytest.fixture(scope="module")
def r50():
    return _setup("resnet50_layer3_layer4_head")


def _layer_local(setup, order):
    """Each emulated layer on the oracle's stored inputs vs the oracle's output."""
    wl, m, P, x, outs = setup
    worst = 0.0
    for i in range(wl.begin, wl.end):
        L = m.layers[i]
        src = outs[L.src]
        res = outs[L.res_src] if L.res_src >= 0 else None
        got = C.layer(L, P.get(i, {}), src, res, wl.dtype, order)
        e = C.rel_inf(got, outs[i])
        worst = max(worst, e)
        assert e <= LAYER_TOL[wl.dtype], f"layer {i} {L.name}: {e:.3e}"
    return worst


@pytest.mark.parametrize("order", [C.Order(32), C.Order(32, 4), C.Order(128, 1, True)],
                         ids=lambda o: o.name)
def test_emulation_is_layer_locally_correct_mobilenet_v2(mbv2, order):
    worst = _layer_local(mbv2, order)
    print(f"mobilenet_v2 {order.name}: worst layer-local rel_inf {worst:.2e}")


@pytest.mark.parametrize("order", [C.Order(32), C.Order(32, 4), C.Order(128, 1, True)],
                         ids=lambda o: o.name)
def test_emulation_is_layer_locally_correct_resnet50_layer3_layer4(r50, order):
    worst = _layer_local(r50, order)
    print(f"resnet50 [25,56) {order.name}: worst layer-local rel_inf {worst:.2e}")


def test_emulation_detects_a_planted_error(r50):
    """A one-term mistake in a layer (a dropped input channel) is caught by the
    layer-local check, so passing it is not vacuous."""
    wl, m, P, x, outs = r50
    i = 26                                       # layer3.0.conv2, 3x3
    L = m.layers[i]
    p = dict(P[i])
    w = p["weight"].copy()
    w[:, 5] = 0.0                                # drop input channel 5
    p["weight"] = w
    got = C.conv_layer(L, p, outs[L.src], None, wl.dtype, C.Order(32))
    assert C.rel_inf(got, outs[i]) > 2 * LAYER_TOL[wl.dtype]


def _end_to_end(setup, orders):
    wl, m, P, x, outs = setup
    res = C.ensemble(m.layers, P, wl.begin, wl.end, x, wl.dtype, outs, orders)
    for r in res:
        print(f"  {r.order:24s} rel_inf {r.rel_inf:.3e}  argmax {int(r.argmax_agree.sum())}/"
              f"{len(r.argmax_agree)}")
    return res


def test_mobilenet_v2_no_fp32_order_meets_2e_2(mbv2):
    res = _end_to_end(mbv2, C.ENSEMBLE)
    errs = [r.rel_inf for r in res]
    print(f"mobilenet_v2 batch 32: fp32 orders span {min(errs):.3e} .. {max(errs):.3e}")
    assert min(errs) > 2e-2
    assert all(not r.argmax_agree.all() for r in res)


def test_resnet50_layer3_layer4_orders_straddle_2e_2(r50):
    res = _end_to_end(r50, C.ENSEMBLE_WIDE)
    errs = np.array([r.rel_inf for r in res])
    print(f"resnet50 [25,56) batch 8: {len(errs)} fp32 orders, min {errs.min():.3e} "
          f"median {np.median(errs):.3e} max {errs.max():.3e}; "
          f"{(errs > 2e-2).mean():.0%} above 2e-2")
    assert errs.min() < 2e-2 < errs.max()
    assert all(r.argmax_agree.all() for r in res)


def test_per_layer_growth_is_reported(r50, mbv2):
    """Error of each stored activation against the oracle's, layer by layer,
    for one order: a one-ulp difference at the first layers grows with depth."""
    for setup in (r50, mbv2):
        wl, m, P, x, outs = setup
        got, gouts = C.forward(m.layers, P, wl.begin, wl.end, x, wl.dtype, C.Order(32),
                               keep=True)
        first = C.rel_inf(gouts[wl.begin], outs[wl.begin])
        growth = [(i, C.rel_inf(gouts[i], outs[i])) for i in range(wl.begin, wl.end)]
        print(f"{wl.name}: " + ", ".join(f"{i}:{e:.1e}" for i, e in growth[::4]))
        assert first <= LAYER_TOL[wl.dtype]
        assert max(e for _, e in growth) > 4 * first
