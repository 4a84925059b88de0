"""Two partitions chained on one GPU (the step on either side of the path)
and the partition-boundary quantisation of the Implementation section:
fp32 feature maps cross a boundary as fp16."""
import numpy as np
import pytest

import oracle
import workloads as W

from gpu_util import gpu_forward, rel_inf, upload_nhwc, empty_out

pytestmark = pytest.mark.gpu


def _special_f32(n_random: int, seed: int) -> np.ndarray:
    sp = [0.0, -0.0, 1.0, -1.0, 65504.0, -65504.0, 65505.0, 65519.0, 65519.99, 65520.0,
          65536.0, 1e30, -1e30, np.inf, -np.inf, np.nan,
          2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -26, 2.0 ** -14, 2.0 ** -14 * (1 - 2.0 ** -11),
          1e-45, -1e-45, 2.0 ** -126, 3.3895314e38, -3.3895314e38]
    rng = np.random.default_rng(seed)
    r = rng.standard_normal(n_random) * np.exp2(rng.integers(-30, 20, n_random))
    # values on and next to the fp16 and bf16 rounding midpoints
    m = rng.standard_normal(n_random // 4).astype(np.float32)
    mid16 = (m.astype(np.float16).astype(np.float32).view(np.uint32) + (1 << 12)).view(np.float32)
    mid_b = ((m.view(np.uint32) & 0xFFFF0000) | 0x8000).view(np.float32)
    return np.concatenate([np.array(sp, np.float32), r.astype(np.float32), mid16, mid_b])


def _device_cast(x: np.ndarray, src: str, dst: str) -> np.ndarray:
    import torch
    from paper_2507_18748_amd import cast
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
    xd = torch.from_numpy(x).to(tdt[src]).cuda() if src != "f32" else \
        torch.from_numpy(np.ascontiguousarray(x, np.float32)).cuda()
    y = torch.empty(x.size, dtype=tdt[dst], device="cuda")
    cast(xd.data_ptr(), src, y.data_ptr(), dst, x.size, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return y.float().cpu().numpy()


def _same_bits(got: np.ndarray, want: np.ndarray):
    got = np.asarray(got, np.float32)
    want = np.asarray(want, np.float32)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    np.testing.assert_array_equal(got[~nan].view(np.uint32), want[~nan].view(np.uint32))


@pytest.mark.parametrize("n_random", [0, 1, 1003])
def test_cast_f32_to_f16_and_back_bit_exact(n_random):
    x = _special_f32(n_random, 3)[: max(1, 26 + n_random)]
    with np.errstate(over="ignore"):
        want16 = x.astype(np.float16).astype(np.float32)      # IEEE round-to-nearest-even
    _same_bits(_device_cast(x, "f32", "f16"), want16)
    # widening is exact
    _same_bits(_device_cast(want16, "f16", "f32"), want16)


@pytest.mark.parametrize("n_random", [1, 1003])
def test_cast_f32_to_bf16_bit_exact(n_random):
    x = _special_f32(n_random, 5)
    _same_bits(_device_cast(x, "f32", "bf16"), oracle.round_to(x, "bf16"))


def test_empty_cast_is_a_no_op():
    import torch
    from paper_2507_18748_amd import cast
    cast(0, "f32", 0, "f16", 0, torch.cuda.current_stream().cuda_stream)


def test_fp32_partitions_chained_through_an_fp16_boundary():
    """ResNet-18 [0,6) fp32 at batch 1 split at a valid boundary, the first
    partition's fp32 output quantised to fp16 and widened back before the
    second partition.

    The fp16 rounding of a boundary value is a discrete decision that a 1e-6
    difference between two correct fp32 results can flip, so the chains are
    not compared with each other directly:
    * the second partition on the oracle's quantised boundary (rounded on the
      host) matches the oracle to the fp32 tolerance;
    * the all-GPU chain and the oracle chain each lie within 2^-11 (the
      quantisation's half-ulp) of the unsplit oracle result, which bounds
      their difference by 2^-10."""
    import torch
    from paper_2507_18748_amd import Partition, split_points, cast
    wl = W.workload("resnet18_stem_layer1")
    m = wl.build_model()
    P = wl.params(m)
    ok = split_points(m.layers)
    p = max(q for q in range(wl.begin + 1, wl.end) if ok[q])
    x = wl.input(1)
    chw = (m.in_c, m.in_h, m.in_w)
    s = torch.cuda.current_stream().cuda_stream
    mid = oracle.forward(m.layers, P, wl.begin, p, x, "f32")
    mid_q = mid.astype(np.float16).astype(np.float32)
    ref = oracle.forward(m.layers, P, p, wl.end, mid_q, "f32")
    whole = oracle.forward(m.layers, P, wl.begin, wl.end, x, "f32")
    with Partition(m.layers, P, chw, wl.begin, p, "f32", max_batch=1) as a, \
            Partition(m.layers, P, chw, p, wl.end, "f32", max_batch=1) as b:
        # second partition alone on the oracle's quantised boundary
        assert rel_inf(gpu_forward(b, mid_q), ref) <= 1e-4
        # the whole chain on the GPU, boundary quantised by ppipe_cast
        xa = upload_nhwc(x, "f32")
        ya = empty_out(a, 1)
        a.run(1, xa.data_ptr(), ya.data_ptr(), s)
        h = torch.empty(ya.numel(), dtype=torch.float16, device="cuda")
        cast(ya.data_ptr(), "f32", h.data_ptr(), "f16", ya.numel(), s)
        yb_in = torch.empty_like(ya)
        cast(h.data_ptr(), "f16", yb_in.data_ptr(), "f32", ya.numel(), s)
        out = empty_out(b, 1)
        b.run(1, yb_in.data_ptr(), out.data_ptr(), s)
        torch.cuda.synchronize()
        got = out.cpu().numpy().transpose(0, 3, 1, 2)
    # the boundary's fp16 rounding carried to the output: 3.4e-4 on the
    # oracle for every valid split of this range
    assert rel_inf(ref, whole) < 2.0 ** -11
    assert rel_inf(got, whole) < 2.0 ** -11


def test_bf16_partitions_chained_match_the_whole_model_bitwise():
    """ResNet-50 [0,44) then [44,56) in bf16 (16-bit boundaries travel
    unchanged) against [0,56) run as one partition, batch 2."""
    import torch
    from paper_2507_18748_amd import Partition
    m = W.zoo.resnet50()
    P = W.model_params(m, 2, "bf16")
    x = W.partition_input((3, 224, 224), 2, 2, "bf16", "image")
    chw = (3, 224, 224)
    s = torch.cuda.current_stream().cuda_stream
    with Partition(m.layers, P, chw, 0, 56, "bf16", max_batch=2) as whole:
        ref = gpu_forward(whole, x)
    with Partition(m.layers, P, chw, 0, 44, "bf16", max_batch=2) as a, \
            Partition(m.layers, P, chw, 44, 56, "bf16", max_batch=2) as b:
        xa = upload_nhwc(x, "bf16")
        ya = empty_out(a, 2)
        a.run(2, xa.data_ptr(), ya.data_ptr(), s)
        out = empty_out(b, 2)
        b.run(2, ya.data_ptr(), out.data_ptr(), s)
        torch.cuda.synchronize()
        got = out.float().cpu().numpy().transpose(0, 3, 1, 2)
    np.testing.assert_array_equal(got.reshape(ref.shape), ref)
