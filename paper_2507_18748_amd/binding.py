"""ctypes binding of libppipe.so: argument marshalling only.

Every step of the forward pass runs in the library's HIP kernels; PyTorch is
used by callers only for device memory (tensor.data_ptr()) and streams
(torch.cuda.Stream.cuda_stream).  The binding raises when the library is not
built: there is no fallback implementation.
"""
import ctypes
import os
from typing import Dict, Iterable, List, Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libppipe.so")

OPS = {"conv": 0, "maxpool": 1, "gap": 2, "fc": 3, "fc_softmax": 4}
ACTS = {"none": 0, "relu": 1, "relu6": 2}
DTYPES = {"f32": 0, "f16": 1, "bf16": 2}

_fp = ctypes.POINTER(ctypes.c_float)
_dp = ctypes.POINTER(ctypes.c_double)


class LayerDesc(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("src", ctypes.c_int32), ("res_src", ctypes.c_int32),
                ("c_in", ctypes.c_int32), ("c_out", ctypes.c_int32), ("k", ctypes.c_int32),
                ("stride", ctypes.c_int32), ("pad", ctypes.c_int32), ("groups", ctypes.c_int32),
                ("act", ctypes.c_int32), ("weight", _fp), ("bias", _fp), ("bn_gamma", _fp),
                ("bn_beta", _fp), ("bn_mean", _fp), ("bn_var", _fp), ("bn_eps", ctypes.c_float),
                ("name", ctypes.c_char_p)]


class Tuning(ctypes.Structure):
    """Planner overrides (kernel tests and tuning sweeps only)."""
    _fields_ = [("gemm_cfg", ctypes.c_int32), ("gemm_waves", ctypes.c_int32),
                ("gemm_splits", ctypes.c_int32), ("no_pointwise", ctypes.c_int32),
                ("no_stem", ctypes.c_int32), ("stream_grid", ctypes.c_int32),
                ("no_pair", ctypes.c_int32), ("dw_outputs", ctypes.c_int32)]


class ModelDesc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("layers", ctypes.POINTER(LayerDesc)),
                ("in_c", ctypes.c_int32), ("in_h", ctypes.c_int32), ("in_w", ctypes.c_int32),
                ("max_batch", ctypes.c_int32)]


def _records(recs, count: int, cap: int) -> List[dict]:
    return [{"layer": r.layer, "launch": r.launch, "kernel": r.kernel.decode(),
             "flops": r.flops, "bytes": r.bytes, "mean_us": r.mean_us,
             "median_us": r.median_us, "min_us": r.min_us} for r in recs[:min(count, cap)]]


class PartitionInfo(ctypes.Structure):
    _fields_ = [("layer_begin", ctypes.c_int32), ("layer_end", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("max_batch", ctypes.c_int32),
                ("in_c", ctypes.c_int32), ("in_h", ctypes.c_int32), ("in_w", ctypes.c_int32),
                ("out_c", ctypes.c_int32), ("out_h", ctypes.c_int32), ("out_w", ctypes.c_int32),
                ("out_dtype", ctypes.c_int32), ("in_bytes_per_image", ctypes.c_int64),
                ("out_bytes_per_image", ctypes.c_int64), ("weight_bytes", ctypes.c_int64),
                ("workspace_bytes", ctypes.c_int64), ("tuned", ctypes.c_int32),
                ("cus", ctypes.c_int32)]


class LayerInfo(ctypes.Structure):
    _fields_ = [("index", ctypes.c_int32), ("op", ctypes.c_int32), ("out_c", ctypes.c_int32),
                ("out_h", ctypes.c_int32), ("out_w", ctypes.c_int32),
                ("kernel_count", ctypes.c_int32), ("out_bytes_b1", ctypes.c_int64),
                ("flops_b1", ctypes.c_double), ("act_bytes_b1", ctypes.c_double),
                ("param_bytes", ctypes.c_double), ("kernel", ctypes.c_char * 96),
                ("name", ctypes.c_char * 64), ("forced", ctypes.c_int32)]


class KernelRecord(ctypes.Structure):
    _fields_ = [("layer", ctypes.c_int32), ("launch", ctypes.c_int32),
                ("kernel", ctypes.c_char * 96), ("flops", ctypes.c_double),
                ("bytes", ctypes.c_double), ("mean_us", ctypes.c_float),
                ("median_us", ctypes.c_float), ("min_us", ctypes.c_float)]


STATUS = {0: "OK", -1: "INVALID", -2: "SPLIT", -3: "UNSUPPORTED", -4: "NOMEM", -5: "HIP"}


MAX_STAGES = 16
DECISIONS = {0: "idle", 1: "dispatch", 2: "drop", 3: "wait"}


class PipelineDesc(ctypes.Structure):
    _fields_ = [("n_stages", ctypes.c_int32),
                ("stage_n_gpus", ctypes.POINTER(ctypes.c_int32)),
                ("stage_gpus", ctypes.POINTER(ctypes.c_int32)),
                ("max_bs", ctypes.c_int32),
                ("unified_bs", ctypes.c_int32),
                ("infer_us", ctypes.POINTER(ctypes.c_double)),
                ("net_us", ctypes.POINTER(ctypes.c_double))]


class Decision(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("pipeline", ctypes.c_int32),
                ("bs", ctypes.c_int32), ("probes", ctypes.c_int32),
                ("first_id", ctypes.c_int64),
                ("start_us", ctypes.c_double), ("finish_us", ctypes.c_double),
                ("deadline_us", ctypes.c_double), ("wake_us", ctypes.c_double),
                ("path", ctypes.c_int32 * MAX_STAGES)]


class SimStats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in ("requests", "dispatched", "dropped", "late",
                                              "batches", "decisions", "probes",
                                              "dispatch_probes")] + \
               [(n, ctypes.c_double) for n in ("decision_us", "dispatch_us", "max_finish_us")]


class PpipeError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"ppipe error {status} ({STATUS.get(status, '?')}): {msg}")
        self.status = status


_lib = None


def load_library() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    # One HIP runtime per process: PyTorch ships its own libamdhip64.so.7 and
    # libhsa-runtime64.so.1.  Loading torch first makes the dynamic linker bind
    # this library to those already-loaded copies (same SONAMEs) instead of a
    # second runtime from /opt/rocm, which would fight torch over the device.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    if not os.path.exists(LIB_PATH):
        raise PpipeError(-5, f"{LIB_PATH} is not built; run __graft_entry__.build() "
                              "or python paper_2507_18748_amd/build.py")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32 = ctypes.c_void_p, ctypes.c_int32
    lib.ppipe_partition_create.restype = vp
    lib.ppipe_partition_create.argtypes = [ctypes.POINTER(ModelDesc), i32, i32, i32]
    lib.ppipe_partition_create_tuned.restype = vp
    lib.ppipe_partition_create_tuned.argtypes = [ctypes.POINTER(ModelDesc), i32, i32, i32,
                                                 ctypes.POINTER(Tuning)]
    lib.ppipe_partition_create_on_share.restype = vp
    lib.ppipe_partition_create_on_share.argtypes = [ctypes.POINTER(ModelDesc), i32, i32, i32, i32]
    lib.ppipe_partition_run.restype = ctypes.c_int
    lib.ppipe_partition_run.argtypes = [vp, i32, vp, vp, vp]
    lib.ppipe_partition_run_static_scratch.restype = ctypes.c_int
    lib.ppipe_partition_run_static_scratch.argtypes = [vp, i32, vp, vp, vp]
    lib.ppipe_partition_capture.restype = ctypes.c_int
    lib.ppipe_partition_capture.argtypes = [vp, i32, vp, vp]
    lib.ppipe_profile_layers.restype = ctypes.c_int
    lib.ppipe_profile_layers.argtypes = [vp, ctypes.POINTER(i32), i32, i32, i32, _fp, _fp]
    lib.ppipe_profile_kernels.restype = ctypes.c_int
    lib.ppipe_profile_kernels.argtypes = [vp, i32, i32, i32, ctypes.POINTER(KernelRecord), i32,
                                          ctypes.POINTER(i32)]
    lib.ppipe_profile_kernels_cold.restype = ctypes.c_int
    lib.ppipe_profile_kernels_cold.argtypes = [vp, i32, i32, ctypes.c_int64,
                                               ctypes.POINTER(KernelRecord), i32,
                                               ctypes.POINTER(i32)]
    lib.ppipe_timing_setup.restype = ctypes.c_int
    lib.ppipe_timing_setup.argtypes = [vp, i32, vp, vp]
    lib.ppipe_partition_run_timed.restype = ctypes.c_int
    lib.ppipe_partition_run_timed.argtypes = [vp, vp]
    lib.ppipe_timing_read.restype = ctypes.c_int
    lib.ppipe_timing_read.argtypes = [vp, ctypes.POINTER(KernelRecord), i32,
                                      ctypes.POINTER(i32)]
    lib.ppipe_partition_info.restype = ctypes.c_int
    lib.ppipe_partition_info.argtypes = [vp, ctypes.POINTER(PartitionInfo)]
    lib.ppipe_layer_info.restype = ctypes.c_int
    lib.ppipe_layer_info.argtypes = [vp, i32, i32, ctypes.POINTER(LayerInfo)]
    lib.ppipe_partition_destroy.restype = None
    lib.ppipe_partition_destroy.argtypes = [vp]
    lib.ppipe_stream_create_cu_share.restype = ctypes.c_int
    lib.ppipe_stream_create_cu_share.argtypes = [i32, i32, ctypes.POINTER(vp)]
    lib.ppipe_stream_destroy.restype = ctypes.c_int
    lib.ppipe_stream_destroy.argtypes = [vp]
    lib.ppipe_cast.restype = ctypes.c_int
    lib.ppipe_cast.argtypes = [vp, i32, vp, i32, ctypes.c_int64, vp]
    lib.ppipe_split_points.restype = ctypes.c_int
    lib.ppipe_split_points.argtypes = [ctypes.POINTER(ModelDesc), ctypes.POINTER(i32)]
    lib.ppipe_prepartition.restype = ctypes.c_int
    lib.ppipe_prepartition.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i32), i32,
                                       i32, ctypes.POINTER(i32), ctypes.POINTER(i32)]
    lib.ppipe_batcher_create.restype = vp
    lib.ppipe_batcher_create.argtypes = [i32, ctypes.POINTER(i32), i32, ctypes.POINTER(PipelineDesc)]
    lib.ppipe_batcher_destroy.restype = None
    lib.ppipe_batcher_destroy.argtypes = [vp]
    lib.ppipe_batcher_submit.restype = ctypes.c_int
    lib.ppipe_batcher_submit.argtypes = [vp, ctypes.c_int64, ctypes.c_double, ctypes.c_double]
    lib.ppipe_batcher_step.restype = ctypes.c_int
    lib.ppipe_batcher_step.argtypes = [vp, ctypes.c_double, i32, ctypes.POINTER(Decision)]
    lib.ppipe_batcher_probe.restype = ctypes.c_int
    lib.ppipe_batcher_probe.argtypes = [vp, i32, i32, ctypes.c_double, _dp, _dp, ctypes.POINTER(i32)]
    lib.ppipe_batcher_check.restype = ctypes.c_int
    lib.ppipe_batcher_check.argtypes = [vp, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64)]
    lib.ppipe_batcher_simulate.restype = ctypes.c_int
    lib.ppipe_batcher_simulate.argtypes = [vp, _dp, ctypes.c_int64, ctypes.c_double,
                                           ctypes.POINTER(SimStats), ctypes.POINTER(Decision),
                                           ctypes.c_int64, ctypes.POINTER(ctypes.c_int64)]
    lib.ppipe_last_error.restype = ctypes.c_char_p
    lib.ppipe_last_error.argtypes = []
    lib.ppipe_last_status.restype = ctypes.c_int32
    lib.ppipe_last_status.argtypes = []
    _lib = lib
    return lib


def _err(lib, status: int):
    return PpipeError(status, lib.ppipe_last_error().decode(errors="replace"))


def _attr(L, name, default=None):
    return L[name] if isinstance(L, dict) else getattr(L, name, default)


def stream_cu_share(part: int, parts: int) -> int:
    """hipStream_t (as an int) restricted to share `part` of `parts` of the CUs."""
    lib = load_library()
    st = ctypes.c_void_p()
    status = lib.ppipe_stream_create_cu_share(part, parts, ctypes.byref(st))
    if status != 0:
        raise _err(lib, status)
    return st.value


def stream_destroy(stream: int):
    lib = load_library()
    status = lib.ppipe_stream_destroy(stream)
    if status != 0:
        raise _err(lib, status)


def cast(x_ptr: int, in_dtype: str, y_ptr: int, out_dtype: str, n: int, stream: int = 0):
    """Boundary quantisation: n elements converted on the device (ppipe_cast)."""
    lib = load_library()
    status = lib.ppipe_cast(x_ptr, DTYPES[in_dtype], y_ptr, DTYPES[out_dtype], n, stream)
    if status != 0:
        raise _err(lib, status)


def split_points(layers: Sequence) -> List[int]:
    """ok[p] for p = 0 .. len(layers): 1 when a partition may start at layer p
    (ppipe_split_points)."""
    lib = load_library()
    arr = (LayerDesc * len(layers))()
    for i, L in enumerate(layers):
        arr[i].op = OPS[_attr(L, "op")]
        arr[i].src = _attr(L, "src")
        arr[i].res_src = _attr(L, "res_src", -1)
    desc = ModelDesc(len(layers), arr, 0, 0, 0, 1)
    ok = (ctypes.c_int32 * (len(layers) + 1))()
    status = lib.ppipe_split_points(ctypes.byref(desc), ok)
    if status != 0:
        raise _err(lib, status)
    return list(ok)


def prepartition(layer_us: Sequence[float], split_ok: Sequence[int], n_blocks: int) -> List[int]:
    """Block boundaries [b0 = 0, b1, ..., n_layers] of the pre-partitioning
    (ppipe_prepartition)."""
    lib = load_library()
    n = len(layer_us)
    t = (ctypes.c_double * n)(*layer_us)
    ok = (ctypes.c_int32 * (n + 1))(*split_ok)
    out = (ctypes.c_int32 * (n + 1))()
    nb = ctypes.c_int32(0)
    status = lib.ppipe_prepartition(t, ok, n, n_blocks, out, ctypes.byref(nb))
    if status != 0:
        raise _err(lib, status)
    return list(out[:nb.value + 1])


def _decision(d: Decision, n_stages: int = MAX_STAGES) -> dict:
    out = {"kind": DECISIONS[d.kind], "pipeline": d.pipeline, "bs": d.bs, "probes": d.probes}
    if d.kind == 1:
        out.update(id=d.first_id, start=d.start_us, finish=d.finish_us, deadline=d.deadline_us,
                   path=[g for g in d.path[:n_stages] if g >= 0])
    elif d.kind == 2:
        out["id"] = d.first_id
    elif d.kind == 3:
        out["wake"] = d.wake_us
    return out


class Batcher:
    """Resource-reservation adaptive batching scheduler (ppipe_batcher_*,
    Sec. 5.4).

    gpu_node: node of each GPU (GPUs of a node share its uplink/downlink).
    pipelines: list of {"stages": [{"gpus": [...], "infer": [l(1)..l(B)],
      "net": [l(1)..l(B)]}, ...], "bs": unified batch size}; every stage of a
      pipeline has tables of the same length B (net of stage 0 is unused).
    """

    def __init__(self, gpu_node: Sequence[int], pipelines: Sequence[dict]):
        self._lib = load_library()
        self._h = None
        keep = []
        descs = (PipelineDesc * len(pipelines))()
        for d, p in zip(descs, pipelines):
            st = p["stages"]
            nb = len(st[0]["infer"])
            if any(len(x["infer"]) != nb or len(x["net"]) != nb for x in st):
                raise PpipeError(-1, "stage tables of one pipeline must have equal length")
            n_g = np.array([len(x["gpus"]) for x in st], np.int32)
            gp = np.array([g for x in st for g in x["gpus"]], np.int32)
            inf = np.ascontiguousarray([x["infer"] for x in st], np.float64)
            net = np.ascontiguousarray([x["net"] for x in st], np.float64)
            keep += [n_g, gp, inf, net]
            d.n_stages, d.max_bs, d.unified_bs = len(st), nb, int(p["bs"])
            d.stage_n_gpus = n_g.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
            d.stage_gpus = gp.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
            d.infer_us = inf.ctypes.data_as(_dp)
            d.net_us = net.ctypes.data_as(_dp)
        nodes = (ctypes.c_int32 * len(gpu_node))(*gpu_node)
        h = self._lib.ppipe_batcher_create(len(gpu_node), nodes, len(pipelines), descs)
        if not h:
            raise _err(self._lib, self._lib.ppipe_last_status())
        self._h = h
        self._stages = [len(p["stages"]) for p in pipelines]

    def _check(self, status):
        if status != 0:
            raise _err(self._lib, status)

    def submit(self, rid: int, arrival: float, deadline: float):
        self._check(self._lib.ppipe_batcher_submit(self._h, rid, arrival, deadline))

    def step(self, now: float, deadline_wake: bool = False) -> dict:
        d = Decision()
        self._check(self._lib.ppipe_batcher_step(self._h, now, int(deadline_wake), ctypes.byref(d)))
        return _decision(d)

    def probe(self, pipeline: int, bs: int, now: float):
        """(finish, wait, path) of a probe that reserves nothing."""
        f, w = ctypes.c_double(), ctypes.c_double()
        path = (ctypes.c_int32 * MAX_STAGES)()
        self._check(self._lib.ppipe_batcher_probe(self._h, pipeline, bs, now, ctypes.byref(f),
                                                  ctypes.byref(w), path))
        return f.value, w.value, list(path[:self._stages[pipeline]])

    def check(self):
        """(overlapping reservation pairs, reservations held)."""
        o, n = ctypes.c_int64(), ctypes.c_int64()
        self._check(self._lib.ppipe_batcher_check(self._h, ctypes.byref(o), ctypes.byref(n)))
        return o.value, n.value

    def simulate(self, arrivals: Sequence[float], slo: float, log_capacity: int = 0):
        """Native event loop (ppipe_batcher_simulate); returns (stats dict,
        list of decisions)."""
        arr = np.ascontiguousarray(arrivals, np.float64)
        st = SimStats()
        log = (Decision * max(log_capacity, 1))()
        cnt = ctypes.c_int64()
        self._check(self._lib.ppipe_batcher_simulate(
            self._h, arr.ctypes.data_as(_dp), len(arr), slo, ctypes.byref(st),
            log if log_capacity > 0 else None, log_capacity, ctypes.byref(cnt)))
        stats = {n: getattr(st, n) for n, _ in SimStats._fields_}
        return stats, [_decision(log[i]) for i in range(cnt.value)]

    def close(self):
        if self._h:
            self._lib.ppipe_batcher_destroy(self._h)
            self._h = None

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Partition:
    """Layers [begin, end) of a model on the current HIP device.

    layers: sequence of objects (or dicts) with fields op, src, res_src, c_in,
      c_out, k, stride, pad, groups, act (op / act as names, see OPS / ACTS).
    params: {layer index: {"weight", "bias", "bn_gamma", "bn_beta", "bn_mean",
      "bn_var"}} of float32 numpy arrays (OIHW weights); read during create.
    tuning: planner overrides for kernel tests and tuning sweeps, a dict of
      Tuning fields (gemm_plan=(cfg, waves, splits) sets the first three);
      None (the default) leaves every choice to the planner.
    cu_share_parts: plan the kernel grids for one of this many CU shares
      (the handle will run on stream_cu_share(i, cu_share_parts) streams);
      None or 1 plans for the whole device.  Not combined with tuning.
    """

    def __init__(self, layers: Sequence, params: Dict[int, Dict[str, np.ndarray]],
                 in_chw: Sequence[int], begin: int, end: int, dtype: str,
                 max_batch: int = 64, bn_eps: float = 1e-5, tuning: Optional[dict] = None,
                 cu_share_parts: Optional[int] = None):
        self._lib = load_library()
        self.begin, self.end, self.dtype = begin, end, dtype
        keep: List[np.ndarray] = []

        def ptr(a: Optional[np.ndarray]):
            if a is None:
                return None
            a = np.ascontiguousarray(a, dtype=np.float32)
            keep.append(a)
            return a.ctypes.data_as(_fp)

        arr = (LayerDesc * len(layers))()
        for i, L in enumerate(layers):
            d = arr[i]
            d.op = OPS[_attr(L, "op")]
            d.src = _attr(L, "src")
            d.res_src = _attr(L, "res_src", -1)
            d.c_in, d.c_out = _attr(L, "c_in"), _attr(L, "c_out")
            d.k, d.stride = _attr(L, "k", 1), _attr(L, "stride", 1)
            d.pad, d.groups = _attr(L, "pad", 0), _attr(L, "groups", 1)
            d.act = ACTS[_attr(L, "act", "none")]
            d.bn_eps = bn_eps
            nm = _attr(L, "name")
            if nm:
                b = str(nm).encode()
                keep.append(b)
                d.name = b
            p = params.get(i, {}) if begin <= i < end else {}
            d.weight = ptr(p.get("weight"))
            d.bias = ptr(p.get("bias"))
            d.bn_gamma = ptr(p.get("bn_gamma"))
            d.bn_beta = ptr(p.get("bn_beta"))
            d.bn_mean = ptr(p.get("bn_mean"))
            d.bn_var = ptr(p.get("bn_var"))
        desc = ModelDesc(len(layers), arr, int(in_chw[0]), int(in_chw[1]), int(in_chw[2]),
                         int(max_batch))
        if tuning and cu_share_parts not in (None, 1):
            raise ValueError("tuning overrides plan for the whole device; drop cu_share_parts")
        if tuning:
            t = Tuning(-1, 0, 1, 0, 0, 0, 0, 0)
            for k, v in tuning.items():
                if k == "gemm_plan":
                    v = [int(q) for q in v]
                    t.gemm_cfg = v[0]
                    t.gemm_waves = v[1] if len(v) > 1 else 0
                    t.gemm_splits = v[2] if len(v) > 2 else 1
                elif k in dict(Tuning._fields_):
                    setattr(t, k, int(v))
                else:
                    raise ValueError(f"unknown tuning field {k!r}")
            h = self._lib.ppipe_partition_create_tuned(ctypes.byref(desc), begin, end,
                                                       DTYPES[dtype], ctypes.byref(t))
        elif cu_share_parts is not None:
            h = self._lib.ppipe_partition_create_on_share(ctypes.byref(desc), begin, end,
                                                          DTYPES[dtype], int(cu_share_parts))
        else:
            h = self._lib.ppipe_partition_create(ctypes.byref(desc), begin, end, DTYPES[dtype])
        if not h:
            raise _err(self._lib, self._lib.ppipe_last_status())
        self._h = ctypes.c_void_p(h)
        info = PartitionInfo()
        self._check(self._lib.ppipe_partition_info(self._h, ctypes.byref(info)))
        self.info = {f: getattr(info, f) for f, _ in PartitionInfo._fields_}

    def _check(self, status: int):
        if status != 0:
            raise _err(self._lib, status)

    # --- execution ---
    def run(self, batch: int, x_ptr: int, out_ptr: int, stream: int = 0):
        """x_ptr / out_ptr: device addresses (tensor.data_ptr()); stream: hipStream_t."""
        self._check(self._lib.ppipe_partition_run(self._h, batch, x_ptr, out_ptr, stream))

    def run_static_scratch(self, batch: int, x_ptr: int, out_ptr: int, stream: int = 0):
        """run() with the kernels' scratch in the library's fixed per-device
        array (allocates nothing; overlapping calls on one device race)."""
        self._check(self._lib.ppipe_partition_run_static_scratch(self._h, batch, x_ptr,
                                                                 out_ptr, stream))

    def capture(self, batch: int, x_ptr: int, out_ptr: int):
        self._check(self._lib.ppipe_partition_capture(self._h, batch, x_ptr, out_ptr))

    # --- profiling ---
    def profile_layers(self, batch_sizes: Iterable[int], warmup: int = 10, reps: int = 50):
        bs = list(batch_sizes)
        nl = self.end - self.begin
        b_arr = (ctypes.c_int32 * len(bs))(*bs)
        table = np.zeros((nl, len(bs)), dtype=np.float32)
        whole = np.zeros(len(bs), dtype=np.float32)
        self._check(self._lib.ppipe_profile_layers(self._h, b_arr, len(bs), warmup, reps,
                                                   table.ctypes.data_as(_fp),
                                                   whole.ctypes.data_as(_fp)))
        return table, whole

    def profile_kernels(self, batch: int, warmup: int = 10, reps: int = 50) -> List[dict]:
        count = ctypes.c_int32(0)
        cap = 4 * (self.end - self.begin) + 8
        recs = (KernelRecord * cap)()
        self._check(self._lib.ppipe_profile_kernels(self._h, batch, warmup, reps, recs, cap,
                                                    ctypes.byref(count)))
        return _records(recs, count.value, cap)

    def profile_kernels_cold(self, batch: int, reps: int = 10,
                             sweep_bytes: int = 1 << 30) -> List[dict]:
        """Isolated-cold per-launch timing (caches swept before every repetition)."""
        count = ctypes.c_int32(0)
        cap = 4 * (self.end - self.begin) + 8
        recs = (KernelRecord * cap)()
        self._check(self._lib.ppipe_profile_kernels_cold(self._h, batch, reps, sweep_bytes,
                                                         recs, cap, ctypes.byref(count)))
        return _records(recs, count.value, cap)

    # --- launch timing inside runs ---
    def timing_setup(self, batch: int, x_ptr: int, out_ptr: int):
        self._check(self._lib.ppipe_timing_setup(self._h, batch, x_ptr, out_ptr))

    def run_timed(self, stream: int = 0):
        self._check(self._lib.ppipe_partition_run_timed(self._h, stream))

    def timing_read(self) -> List[dict]:
        count = ctypes.c_int32(0)
        cap = 4 * (self.end - self.begin) + 8
        recs = (KernelRecord * cap)()
        self._check(self._lib.ppipe_timing_read(self._h, recs, cap, ctypes.byref(count)))
        return _records(recs, count.value, cap)

    def layer_info(self, index: int, batch: int = 1) -> dict:
        li = LayerInfo()
        self._check(self._lib.ppipe_layer_info(self._h, index, batch, ctypes.byref(li)))
        d = {f: getattr(li, f) for f, _ in LayerInfo._fields_}
        d["kernel"] = li.kernel.decode()
        d["name"] = li.name.decode()
        return d

    # --- lifetime ---
    def close(self):
        if getattr(self, "_h", None):
            self._lib.ppipe_partition_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
