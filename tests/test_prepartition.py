"""Pre-partitioning (Sec. 5.2): oracle pins, and the library's host functions
(ppipe_split_points, ppipe_prepartition; no device needed) against the
oracle."""
import numpy as np
import pytest

import workloads as W
from oracle import prepartition as O


def test_oracle_worked_example():
    # target 5: from layer 0, sums 1, 2, 3, 4, 10 -> the block closes after 4 layers
    assert O.prepartition([1, 1, 1, 1, 6], [1] * 6, 2) == [0, 4, 5]
    # equal layers divide evenly
    assert O.prepartition([2.0] * 20, [1] * 21, 10) == list(range(0, 21, 2))
    # a block cannot end at an invalid boundary: the nearest valid one is taken
    assert O.prepartition([1] * 6, [1, 1, 0, 0, 1, 1, 1], 3) == [0, 1, 4, 6]
    # ties go to the earlier end (sums 1 and 2 are equally close to 1.5), which
    # can leave more than N blocks
    assert O.prepartition([1, 1, 1], [1, 1, 1, 1], 2) == [0, 1, 2, 3]


def test_oracle_split_points_resnet50():
    """Valid partition starts of ResNet-50 from the architecture: stem conv,
    max pool, then [3, 4, 6, 3] bottlenecks of 3 fused layers (4 for the
    first of each stage, which carries the downsample projection), global
    average pool, FC."""
    starts, i = [0, 1, 2], 2
    for stage, blocks in enumerate([3, 4, 6, 3]):
        for b in range(blocks):
            i += 4 if b == 0 else 3
            starts.append(i)
    starts += [i + 1, i + 2]          # after avgpool, after fc (= n)
    m = W.zoo.resnet50()
    assert len(m.layers) == 56 and i == 54
    ok = O.split_points(m.layers)
    assert [p for p, v in enumerate(ok) if v] == starts
    assert ok[44] and ok[25] and not ok[45]


def test_oracle_blocks_cover_and_are_closest_by_brute_force():
    rng = np.random.default_rng(7)
    for _ in range(200):
        n = int(rng.integers(1, 14))
        t = [float(v) for v in rng.exponential(1.0, n)]
        if rng.random() < 0.3:
            t[int(rng.integers(0, n))] = 0.0
        ok = [1] + [int(rng.random() < 0.6) for _ in range(n - 1)] + [1]
        N = int(rng.integers(1, 6))
        b = O.prepartition(t, ok, N)
        assert b[0] == 0 and b[-1] == n and all(x < y for x, y in zip(b, b[1:]))
        assert all(ok[x] for x in b)
        target = sum(t) / N
        for s, e in zip(b, b[1:]):
            # brute force: no admissible end is strictly closer, none earlier equally close
            for q in range(s + 1, n + 1):
                if q != n and not ok[q]:
                    continue
                g, ge = abs(sum(t[s:q]) - target), abs(sum(t[s:e]) - target)
                assert g > ge or (g == ge and q >= e)


@pytest.mark.parametrize("model", ["resnet18", "resnet50", "resnet152", "vgg16", "mobilenet_v2"])
def test_library_split_points_match_oracle(model):
    from paper_2507_18748_amd import split_points
    m = W.zoo.model(model)
    assert split_points(m.layers) == O.split_points(m.layers)


def test_library_split_points_match_partition_create_rule():
    """A partition the library accepts starts at a valid point and vice versa
    (create rejects a range whose input is not one feature map)."""
    from paper_2507_18748_amd import split_points
    m = W.zoo.resnet50()
    ok = split_points(m.layers)
    assert ok[44] == 1 and ok[45] == 0 and ok[46] == 0


def test_library_prepartition_matches_oracle():
    from paper_2507_18748_amd import prepartition
    rng = np.random.default_rng(11)
    for _ in range(300):
        n = int(rng.integers(1, 40))
        t = [float(v) for v in rng.exponential(5.0, n)]
        if rng.random() < 0.3:
            t[int(rng.integers(0, n))] = 0.0
        ok = [1] + [int(rng.random() < 0.5) for _ in range(n - 1)] + [1]
        N = int(rng.integers(1, 12))
        assert prepartition(t, ok, N) == O.prepartition(t, ok, N), (t, ok, N)


def test_library_prepartition_rejects_bad_input():
    from paper_2507_18748_amd import prepartition, PpipeError
    with pytest.raises(PpipeError):
        prepartition([1.0, -1.0], [1, 1, 1], 2)
    with pytest.raises(PpipeError):
        prepartition([1.0], [1, 1], 0)
