"""Helpers for the GPU parity tests: upload NCHW host data as NHWC device
tensors, run a partition through the C ABI, and compare with the oracle."""
import numpy as np

TORCH_DT = {}


def _torch():
    import torch
    if not TORCH_DT:
        TORCH_DT.update({"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16})
    return torch


def upload_nhwc(x_nchw: np.ndarray, dtype: str):
    torch = _torch()
    if x_nchw.ndim == 2:                       # an FC output: [N, K] is N x K x 1 x 1
        x_nchw = x_nchw.reshape(x_nchw.shape + (1, 1))
    t = torch.from_numpy(np.ascontiguousarray(x_nchw.transpose(0, 2, 3, 1)))
    return t.to(TORCH_DT[dtype]).cuda().contiguous()


def empty_out(part, batch: int):
    torch = _torch()
    i = part.info
    dt = torch.float32 if i["out_dtype"] == 0 else TORCH_DT[part.dtype]
    return torch.empty((batch, i["out_h"], i["out_w"], i["out_c"]), dtype=dt, device="cuda")


def gpu_forward(part, x_nchw: np.ndarray, capture: bool = False, reps: int = 1) -> np.ndarray:
    """Run the partition on x (NCHW host array); returns NCHW (or [N, classes]) float32."""
    torch = _torch()
    b = x_nchw.shape[0]
    x = upload_nhwc(x_nchw, part.dtype)
    out = empty_out(part, b)
    stream = torch.cuda.current_stream().cuda_stream
    if capture:
        part.capture(b, x.data_ptr(), out.data_ptr())
    for _ in range(reps):
        part.run(b, x.data_ptr(), out.data_ptr(), stream)
    torch.cuda.synchronize()
    return np.ascontiguousarray(out.float().cpu().numpy().transpose(0, 3, 1, 2))


def rel_inf(got: np.ndarray, ref: np.ndarray) -> float:
    """max |g - r| / max |r| (the infinity-norm relative error)."""
    g = np.asarray(got, np.float64).reshape(-1)
    r = np.asarray(ref, np.float64).reshape(-1)
    assert g.shape == r.shape, (got.shape, ref.shape)
    assert np.isfinite(g).all(), "non-finite GPU output"
    return float(np.abs(g - r).max() / max(np.abs(r).max(), 1e-30))


def argmax_rows(p: np.ndarray) -> np.ndarray:
    return np.asarray(p).reshape(p.shape[0], -1).argmax(axis=1)
