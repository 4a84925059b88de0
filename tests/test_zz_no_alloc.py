"""ppipe_partition_run_static_scratch: the allocation-free variant of
ppipe_partition_run, whose kernels take their scratch memory (split-K
partials, softmax logits, the channel-padded stem input) from the library's
fixed per-device array.  Its output must equal ppipe_partition_run's bit for
bit (same kernels, same plans), on two calls in a row with the second on a
smaller batch, and it must refuse a batch whose scratch exceeds the array."""
import numpy as np
import pytest

import workloads as W
from workloads.zoo import Model

from gpu_util import upload_nhwc, empty_out

pytestmark = pytest.mark.gpu


def _run_both(part, x_nchw, dtype):
    import torch
    b = x_nchw.shape[0]
    xd = upload_nhwc(x_nchw, dtype)
    st = torch.cuda.current_stream().cuda_stream
    outs = []
    for fn in (part.run, part.run_static_scratch):
        o = empty_out(part, b)
        o.fill_(float("nan"))
        fn(b, xd.data_ptr(), o.data_ptr(), st)
        torch.cuda.synchronize()
        outs.append(o.float().cpu().numpy())
    return outs


@pytest.mark.parametrize("name,batches", [("resnet50_layer4_head", (8, 3)),
                                          ("resnet18_stem_layer1", (2, 1))])
def test_static_scratch_matches_run(name, batches):
    from paper_2507_18748_amd import Partition
    wl = W.workload(name)
    m = wl.build_model()
    P = wl.params(m)
    with Partition(m.layers, P, (m.in_c, m.in_h, m.in_w), wl.begin, wl.end, wl.dtype,
                   max_batch=max(batches)) as part:
        for b in batches:                       # the second call on a smaller batch
            print(f"[no-alloc] {name} batch {b}", flush=True)
            ref, got = _run_both(part, wl.input(b), wl.dtype)
            assert np.isfinite(ref).all()
            np.testing.assert_array_equal(got, ref)


def test_static_scratch_refuses_more_than_it_holds():
    """A 1x1 layer forced to two K splits needs 2 * M * Co fp32 partials:
    102.8 MB at batch 64 (refused, nothing launched), 25.7 MB at batch 16
    (accepted, equal to run())."""
    from paper_2507_18748_amd import Partition, PpipeError
    m = Model("t", 256, 28, 28)
    m.add(name="c", op="conv", src=-1, c_in=256, c_out=256, act="relu", bn=True)
    P = W.model_params(m, 0, "bf16")
    with Partition(m.layers, P, (256, 28, 28), 0, 1, "bf16", max_batch=64,
                   tuning={"gemm_plan": (9, 0, 2)}) as part:
        assert "splits=2" in part.layer_info(0, 64)["kernel"]
        x = W.partition_input((256, 28, 28), 64, 1, "bf16", "relu_normal")
        xd = upload_nhwc(x, "bf16")
        o = empty_out(part, 64)
        print("[no-alloc] refusal at batch 64", flush=True)
        with pytest.raises(PpipeError) as e:
            part.run_static_scratch(64, xd.data_ptr(), o.data_ptr(), 0)
        assert e.value.status == -1
        print("[no-alloc] forced split at batch 16", flush=True)
        ref, got = _run_both(part, x[:16], "bf16")
        np.testing.assert_array_equal(got, ref)


def test_static_scratch_on_resnet152():
    """ResNet-152 (the default workload) fits the array at batch 64 (its
    scratch is layer4's split-K partials; the stem kernel reads the
    3-channel image as it is) and equals run() there and then at batch 32."""
    from paper_2507_18748_amd import Partition
    wl = W.workload("resnet152")
    m = wl.build_model()
    P = wl.params(m)
    with Partition(m.layers, P, (m.in_c, m.in_h, m.in_w), wl.begin, wl.end, wl.dtype,
                   max_batch=64) as part:
        assert part.layer_info(0, 64)["kernel"].startswith("stem_conv<")
        x = wl.input(64)
        for b in (64, 32):                      # the second call on a smaller batch
            print(f"[no-alloc] resnet152 batch {b}", flush=True)
            ref, got = _run_both(part, x[:b], wl.dtype)
            assert np.isfinite(ref).all()
            np.testing.assert_array_equal(got, ref)
