"""Runtime behaviour through the C ABI: repeatability, graph replay,
batch-size sweep on one handle, profiling tables and error paths."""
import numpy as np
import pytest

import oracle
import workloads as W

from gpu_util import gpu_forward, rel_inf, upload_nhwc, empty_out

pytestmark = pytest.mark.gpu


def _small():
    wl = W.workload("resnet50_layer4_head")
    m = wl.build_model()
    return wl, m, wl.params(m)


def test_bitwise_repeatable_and_graph_replay_matches_eager():
    import torch
    from paper_2507_18748_amd import Partition
    wl, m, P = _small()
    x = wl.input(8)
    with Partition(m.layers, P, (3, 224, 224), wl.begin, wl.end, wl.dtype, max_batch=8) as part:
        a = gpu_forward(part, x)
        b = gpu_forward(part, x)
        np.testing.assert_array_equal(a, b)
        xd = upload_nhwc(x, wl.dtype)
        out = empty_out(part, 8)
        part.capture(8, xd.data_ptr(), out.data_ptr())
        s = torch.cuda.current_stream().cuda_stream
        for _ in range(4):
            out.zero_()
            part.run(8, xd.data_ptr(), out.data_ptr(), s)
            torch.cuda.synchronize()
            _ = (xd.float() * 2).sum().item()      # unrelated eager work between replays
            got = out.float().cpu().numpy().transpose(0, 3, 1, 2)
            np.testing.assert_array_equal(got, a)


def test_timed_runs_match_plain_runs_and_time_every_launch():
    """Timed runs (events recorded by every launch) give the same bits as
    plain runs, and one record per launch with a positive duration."""
    import torch
    from paper_2507_18748_amd import Partition
    wl, m, P = _small()
    x = wl.input(8)
    with Partition(m.layers, P, (3, 224, 224), wl.begin, wl.end, wl.dtype, max_batch=8) as part:
        ref = gpu_forward(part, x)
        xd = upload_nhwc(x, wl.dtype)
        out = empty_out(part, 8)
        part.timing_setup(8, xd.data_ptr(), out.data_ptr())
        s = torch.cuda.current_stream().cuda_stream
        for _ in range(3):
            out.zero_()
            part.run_timed(s)
            torch.cuda.synchronize()
            got = out.float().cpu().numpy().transpose(0, 3, 1, 2)
            np.testing.assert_array_equal(got, ref)
        recs = part.timing_read()
        launches = sum(part.layer_info(i, 8)["kernel_count"] for i in range(wl.begin, wl.end))
        assert len(recs) == launches
        assert all(r["mean_us"] > 0 for r in recs)
        assert [r["layer"] for r in recs] == sorted(r["layer"] for r in recs)


def test_batch_sweep_on_one_handle():
    from paper_2507_18748_amd import Partition
    wl, m, P = _small()
    x = wl.input(16)
    ref0 = oracle.forward(m.layers, P, wl.begin, wl.end, x[:1], wl.dtype)
    with Partition(m.layers, P, (3, 224, 224), wl.begin, wl.end, wl.dtype, max_batch=16) as part:
        for b in (1, 2, 3, 5, 8, 13, 16):
            got = gpu_forward(part, x[:b])
            assert rel_inf(got[:1].reshape(ref0.shape), ref0) <= 2e-2
        from paper_2507_18748_amd import PpipeError
        with pytest.raises(PpipeError):
            part.run(17, 1, 2, 0)
        with pytest.raises(PpipeError):
            part.run(0, 1, 2, 0)


def test_profile_tables():
    from paper_2507_18748_amd import Partition
    wl, m, P = _small()
    with Partition(m.layers, P, (3, 224, 224), wl.begin, wl.end, wl.dtype, max_batch=8) as part:
        table, whole = part.profile_layers([1, 2, 8], warmup=3, reps=10)
        assert table.shape == (12, 3)
        assert np.isfinite(table).all() and (table > 0).all()
        assert (whole > 0).all()
        # the partition time is the sum of its layers up to launch gaps
        ratio = whole / table.sum(axis=0)
        print("partition / sum(layers):", ratio)
        assert ((ratio > 0.3) & (ratio < 1.5)).all()
        recs = part.profile_kernels(8, warmup=3, reps=10)
        assert len(recs) >= 12 and all(r["mean_us"] > 0 for r in recs)
        info = part.layer_info(44, 8)
        assert info["out_bytes_b1"] == 512 * 14 * 14 * 2 and info["flops_b1"] > 0


def test_isolated_cold_profile_records_every_launch():
    from paper_2507_18748_amd import Partition
    wl, m, P = _small()
    with Partition(m.layers, P, (3, 224, 224), wl.begin, wl.end, wl.dtype, max_batch=8) as part:
        recs = part.profile_kernels_cold(8, reps=2, sweep_bytes=64 << 20)
        launches = sum(part.layer_info(i, 8)["kernel_count"] for i in range(wl.begin, wl.end))
        assert len(recs) == launches
        assert all(r["min_us"] > 0 and r["min_us"] <= r["median_us"] for r in recs)


def test_chained_blocks_match_the_whole_range_bitwise():
    """Pre-partitioned blocks run one after another give the same bits as the
    range run as one partition (every launch plan depends on the layer shape
    and batch only), and close the range exactly."""
    import torch
    from paper_2507_18748_amd import Partition, split_points, prepartition
    wl, m, P = _small()
    x = wl.input(8)
    ok = split_points(m.layers)
    flops = []
    with Partition(m.layers, P, (3, 224, 224), wl.begin, wl.end, wl.dtype, max_batch=8) as part:
        ref = gpu_forward(part, x)
        flops = [part.layer_info(i, 1)["flops_b1"] + 1e6 for i in range(wl.begin, wl.end)]
    local_ok = [1] + [ok[p] for p in range(wl.begin + 1, wl.end)] + [1]
    bounds = [wl.begin + b for b in prepartition(flops, local_ok, 3)]
    assert bounds[0] == wl.begin and bounds[-1] == wl.end and len(bounds) >= 3
    cur = upload_nhwc(x, wl.dtype)
    s = torch.cuda.current_stream().cuda_stream
    for bb, be in zip(bounds, bounds[1:]):
        with Partition(m.layers, P, (3, 224, 224), bb, be, wl.dtype, max_batch=8) as bp:
            out = empty_out(bp, 8)
            bp.run(8, cur.data_ptr(), out.data_ptr(), s)
            torch.cuda.synchronize()
        cur = out
    got = cur.float().cpu().numpy().transpose(0, 3, 1, 2)
    np.testing.assert_array_equal(got.reshape(ref.shape), ref)


@pytest.mark.parametrize("parts", [2, 4])
def test_handles_planned_for_a_cu_share(parts):
    """A handle created for one of `parts` CU shares plans its grids for that
    share's compute units: fewer CUs in its info, K splits and tiles chosen
    for them (some layer of ResNet-50 [44,56) at batch 8 changes plan), and
    its output on a share stream matches the oracle at the end-to-end bar."""
    import torch
    from paper_2507_18748_amd import Partition, stream_cu_share, stream_destroy
    wl, m, P = _small()
    x = wl.input(8)
    ref = oracle.forward(m.layers, P, wl.begin, wl.end, x, wl.dtype)
    with Partition(m.layers, P, (3, 224, 224), wl.begin, wl.end, wl.dtype, max_batch=8) as whole:
        whole_plans = [whole.layer_info(i, 8)["kernel"] for i in range(wl.begin, wl.end)]
        whole_cus = whole.info["cus"]
    st = stream_cu_share(0, parts)
    try:
        with Partition(m.layers, P, (3, 224, 224), wl.begin, wl.end, wl.dtype, max_batch=8,
                       cu_share_parts=parts) as h:
            assert h.info["cus"] == whole_cus // 8 // parts * 8
            plans = [h.layer_info(i, 8)["kernel"] for i in range(wl.begin, wl.end)]
            print("changed:", [(a, b) for a, b in zip(whole_plans, plans) if a != b])
            assert plans != whole_plans
            xd = upload_nhwc(x, wl.dtype)
            o = empty_out(h, 8)
            h.run(8, xd.data_ptr(), o.data_ptr(), st)
            torch.cuda.synchronize()
            got = o.float().cpu().numpy().transpose(0, 3, 1, 2).reshape(ref.shape)
            assert rel_inf(got, ref) <= 2e-2
            assert (got.reshape(8, -1).argmax(1) == ref.reshape(8, -1).argmax(1)).all()
    finally:
        torch.cuda.synchronize()
        stream_destroy(st)


@pytest.mark.parametrize("parts", [1, 2, 3, 4])
def test_runs_on_cu_share_streams_match_the_default_stream(parts):
    """Virtual GPUs: each share's stream runs its own handle side by side
    with the others and gives the same bits as a run on the default stream."""
    import torch
    from paper_2507_18748_amd import Partition, stream_cu_share, stream_destroy
    wl, m, P = _small()
    x = wl.input(4)
    hs = [Partition(m.layers, P, (3, 224, 224), wl.begin, wl.end, wl.dtype, max_batch=4)
          for _ in range(parts)]
    streams = [stream_cu_share(j, parts) for j in range(parts)]
    try:
        ref = gpu_forward(hs[0], x)
        xd = upload_nhwc(x, wl.dtype)
        outs = [empty_out(h, 4) for h in hs]
        for _ in range(3):
            for h, o, st in zip(hs, outs, streams):
                h.run(4, xd.data_ptr(), o.data_ptr(), st)
        torch.cuda.synchronize()
        for o in outs:
            got = o.float().cpu().numpy().transpose(0, 3, 1, 2)
            np.testing.assert_array_equal(got.reshape(ref.shape), ref)
    finally:
        torch.cuda.synchronize()
        for st in streams:
            stream_destroy(st)
        for h in hs:
            h.close()
