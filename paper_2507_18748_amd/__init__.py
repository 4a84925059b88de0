"""MI355X-native forward pass of a CNN pipeline partition and its per-layer
latency table (the data-parallel computation that dominates PPipe's run
time).  The compute lives in hand-written gfx950 HIP kernels behind the C ABI
declared in include/ppipe.h; this package is the thin ctypes binding."""
from .binding import (Partition, PpipeError, load_library, LIB_PATH, OPS, ACTS,
                      DTYPES, split_points, prepartition, cast,
                      stream_cu_share, stream_destroy, Batcher)

__all__ = ["Partition", "PpipeError", "load_library", "LIB_PATH", "OPS", "ACTS", "DTYPES",
           "split_points", "prepartition", "cast", "stream_cu_share", "stream_destroy", "Batcher"]
