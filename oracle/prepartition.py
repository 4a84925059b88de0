"""Oracle for DNN pre-partitioning (Sec. 5.2).

TEST INFRASTRUCTURE ONLY: imported by the test suite, never by the GPU
library.  Plain Python, written from the paper's description and the
problem statement's partition rule, independent of the library's code.

* A partition [p, q) receives exactly one feature map, the output of layer
  p - 1 (the MILP's Y_bj): it may start at p only if no layer from p on reads
  an output produced before layer p - 1 (the model input counts as "layer
  -1").
* Pre-partitioning groups consecutive layers, from the first one on, into a
  block whose summed runtime is as close as possible to 1/N of the whole
  model's runtime, and repeats from the next layer until the last one.  Here
  every block must itself be a valid partition, so a block may end only at a
  valid start of the next; among equally close ends the earliest is taken.
"""
from typing import List, Sequence


def _refs(layer):
    get = (lambda k, d=None: layer.get(k, d)) if isinstance(layer, dict) else \
          (lambda k, d=None: getattr(layer, k, d))
    out = [get("src")]
    res = get("res_src", -1)
    if res is not None and res >= 0:
        out.append(res)
    return out


def split_points(layers: Sequence) -> List[int]:
    """ok[p], p = 0 .. n: 1 if a partition may start at layer p."""
    n = len(layers)
    ok = []
    for p in range(n + 1):
        good = True
        for j in range(p, n):
            for r in _refs(layers[j]):
                if r < p - 1:        # produced before the partition's input
                    good = False
        ok.append(1 if (p == 0 or p == n or good) else 0)
    return ok


def prepartition(layer_us: Sequence[float], split_ok: Sequence[int], n_blocks: int) -> List[int]:
    """Block starts followed by n (the paper's greedy grouping)."""
    n = len(layer_us)
    target = sum(layer_us) / n_blocks
    starts = []
    start = 0
    while start < n:
        starts.append(start)
        # every admissible end of the block and how close its runtime gets
        cands = [q for q in range(start + 1, n + 1) if q == n or split_ok[q]]
        gaps = [abs(sum(layer_us[start:q]) - target) for q in cands]
        best = min(gaps)
        start = cands[gaps.index(best)]      # earliest of the closest
    return starts + [n]
