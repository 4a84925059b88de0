"""The C-ABI library: builds for gfx950, exports every symbol the header
declares, keeps torch and the oracle out of its interface, and validates
model descriptions on the host before touching a device."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ppipe.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ppipe_[a-z_]+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for must in ("ppipe_partition_create", "ppipe_partition_run", "ppipe_profile_layers",
                 "ppipe_partition_info", "ppipe_layer_info", "ppipe_partition_destroy",
                 "ppipe_last_error", "ppipe_profile_kernels", "ppipe_partition_capture",
                 "ppipe_batcher_create", "ppipe_batcher_step", "ppipe_batcher_simulate"):
        assert must in names
    text = open(HEADER).read()
    assert "torch" not in text.lower().replace("pytorch", "") or "at::" not in text
    assert "at::Tensor" not in text and "c10" not in text


def test_library_exports_every_declared_symbol():
    from paper_2507_18748_amd import load_library
    lib = load_library()
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_library_does_not_contain_the_oracle():
    from paper_2507_18748_amd import LIB_PATH
    out = subprocess.run(["nm", "-D", "--defined-only", LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    assert "oracle" not in out
    needed = subprocess.run(["readelf", "-d", LIB_PATH], capture_output=True, text=True,
                            check=True).stdout
    assert "liboracle" not in needed and "torch" not in needed


def test_header_compiles_as_c():
    src = '#include "ppipe.h"\nint main(void){ppipe_partition_info_t i; (void)i; return 0;}\n'
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.dirname(HEADER),
                        "-x", "c", "-", "-fsyntax-only"], input=src, text=True,
                       capture_output=True)
    assert r.returncode == 0, r.stderr


def _tiny_layers():
    from workloads.zoo import Layer
    return [Layer("c0", "conv", -1, 8, 16, 3, 1, 1, act="relu", bn=True),
            Layer("c1", "conv", 0, 16, 16, 1, bn=True),
            Layer("c2", "conv", 1, 16, 16, 3, 1, 1, act="relu", bn=True, res_src=0),
            Layer("gap", "gap", 2, 16, 16),
            Layer("fc", "fc_softmax", 3, 16, 12, bias=True)]


def _params(layers, seed=0):
    import workloads as W
    return {i: W.layer_params(L, i, seed, "f16") for i, L in enumerate(layers)}


def _status_of(fn):
    from paper_2507_18748_amd import PpipeError
    with pytest.raises(PpipeError) as e:
        fn()
    return e.value.status


def test_create_rejects_residual_across_the_boundary():
    from paper_2507_18748_amd import Partition
    L = _tiny_layers()
    # layer 2 adds layer 0's output: a split before 1 or 2 crosses that edge
    assert _status_of(lambda: Partition(L, _params(L), (8, 9, 9), 2, 5, "f16")) == -2
    assert _status_of(lambda: Partition(L, _params(L), (8, 9, 9), 0, 2, "f16")) == -2


def test_create_rejects_bad_descriptions():
    from paper_2507_18748_amd import Partition
    from workloads.zoo import Layer
    L = _tiny_layers()
    P = _params(L)
    assert _status_of(lambda: Partition(L, P, (8, 9, 9), 3, 3, "f16")) == -1       # empty range
    assert _status_of(lambda: Partition(L, P, (4, 9, 9), 0, 5, "f16")) == -1       # c_in mismatch
    bad = list(L)
    bad[1] = Layer("g", "conv", 0, 16, 16, 3, 1, 1, groups=4, bn=True)             # grouped
    assert _status_of(lambda: Partition(bad, _params(bad), (8, 9, 9), 0, 5, "f16")) == -3
    bad = list(L)
    bad[3] = Layer("fc", "fc_softmax", 2, 16 * 81, 12, bias=True)                  # not last
    assert _status_of(lambda: Partition(bad[:4] + [Layer("x", "fc", 3, 12, 8)], {
        **_params(bad[:4]), 4: {"weight": np.zeros((8, 12), np.float32)}}, (8, 9, 9), 0, 5,
        "f16")) == -3
    odd = list(L)
    odd[0] = Layer("c0", "conv", -1, 8, 18, 3, 1, 1, act="relu", bn=True)         # Co % 4 != 0
    odd[1] = Layer("c1", "conv", 0, 18, 16, 1, bn=True)
    odd[2] = Layer("c2", "conv", 1, 16, 16, 3, 1, 1, bn=True)
    assert _status_of(lambda: Partition(odd, _params(odd), (8, 9, 9), 0, 5, "f16")) == -3
    miss = _params(L)
    del miss[2]["weight"]
    assert _status_of(lambda: Partition(L, miss, (8, 9, 9), 0, 5, "f16")) == -1


def test_timing_calls_reject_a_null_handle():
    """Error paths of the timed-run entry points need no device."""
    import ctypes
    from paper_2507_18748_amd.binding import load_library, KernelRecord
    lib = load_library()
    n = ctypes.c_int32(0)
    assert lib.ppipe_partition_run_timed(None, None) == -1
    assert lib.ppipe_timing_read(None, (KernelRecord * 1)(), 1, ctypes.byref(n)) == -1
    assert lib.ppipe_timing_setup(None, 1, None, None) == -1


def test_cast_rejects_bad_arguments():
    from paper_2507_18748_amd.binding import load_library
    lib = load_library()
    assert lib.ppipe_cast(None, 0, None, 7, 4, None) == -1      # bad output dtype
    assert lib.ppipe_cast(None, 0, None, 1, -1, None) == -1     # negative count
    assert lib.ppipe_cast(None, 0, None, 1, 8, None) == -1      # null buffers


def test_cu_share_stream_rejects_bad_shares():
    import ctypes
    from paper_2507_18748_amd.binding import load_library
    lib = load_library()
    st = ctypes.c_void_p()
    assert lib.ppipe_stream_create_cu_share(2, 2, ctypes.byref(st)) == -1
    assert lib.ppipe_stream_create_cu_share(0, 0, ctypes.byref(st)) == -1
    assert lib.ppipe_stream_destroy(None) == 0


def test_product_sources_read_no_environment():
    """Kernel choice is deterministic in the layer shape and the create-time
    tuning argument: no library source reads an environment variable."""
    csrc = os.path.join(ROOT, "paper_2507_18748_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        text = open(os.path.join(csrc, f)).read()
        assert "getenv" not in text, f


def test_create_tuned_rejects_out_of_range_overrides():
    from paper_2507_18748_amd import Partition
    layers = _tiny_layers()
    for bad in ({"gemm_cfg": 999}, {"dw_outputs": 3}, {"gemm_plan": (0, 0, 100)},
                {"stream_grid": -1}):
        st = _status_of(lambda: Partition(layers, _params(layers), (8, 6, 6), 0, 5, "f16",
                                          max_batch=4, tuning=bad))
        assert st == -1, bad
    with pytest.raises(ValueError):
        Partition(layers, _params(layers), (8, 6, 6), 0, 5, "f16", max_batch=4,
                  tuning={"no_such_field": 1})


def test_create_on_share_rejects_out_of_range_parts():
    """CU-share-sized planning takes 1..8 shares; the check comes before any
    device work, and tuning overrides cannot be combined with it."""
    from paper_2507_18748_amd import Partition
    layers = _tiny_layers()
    for bad in (0, 9, -1):
        st = _status_of(lambda: Partition(layers, _params(layers), (8, 6, 6), 0, 5, "f16",
                                          max_batch=4, cu_share_parts=bad))
        assert st == -1, bad
    with pytest.raises(ValueError):
        Partition(layers, _params(layers), (8, 6, 6), 0, 5, "f16", max_batch=4,
                  tuning={"no_pair": 1}, cu_share_parts=2)
