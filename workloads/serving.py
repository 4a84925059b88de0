"""Seeded synthetic serving workloads for the adaptive batching scheduler:
request arrival traces, cluster layouts and pooled-pipeline plans.

Inputs only: nothing here schedules, probes or reserves.  Poisson arrivals
stand in for the production traces the paper replays, which are not
available here.
"""
from typing import List, Sequence

import numpy as np


def poisson_arrivals(rate_per_us: float, n: int, seed: int, start: float = 0.0) -> np.ndarray:
    """n arrival times (us) of a Poisson process of the given rate: the
    cumulative sum of exponential gaps with mean 1 / rate."""
    rng = np.random.default_rng(seed)
    return start + np.cumsum(rng.exponential(1.0 / rate_per_us, size=n))


def bursty_arrivals(rate_per_us: float, n: int, seed: int, burst: int = 8) -> np.ndarray:
    """n arrival times with the same mean rate in bursts: Poisson burst
    starts at rate / burst, each burst a geometric number (mean `burst`) of
    requests a microsecond apart."""
    rng = np.random.default_rng(seed)
    out: List[float] = []
    t = 0.0
    while len(out) < n:
        t += rng.exponential(burst / rate_per_us)
        k = int(rng.geometric(1.0 / burst))
        out += [t + i for i in range(k)]
        t += k
    return np.array(out[:n])


def node_layout(n_nodes: int, gpus_per_node: int) -> List[int]:
    """gpu_node list: GPU g lives on node g // gpus_per_node."""
    return [g // gpus_per_node for g in range(n_nodes * gpus_per_node)]


def random_tables(rng: np.random.Generator, n_stages: int, max_bs: int, integer: bool) -> dict:
    """Per-stage latency tables that grow with the batch size: a fixed part
    plus a per-sample part (inference), and a per-sample transfer size."""
    infer, net = [], []
    for _ in range(n_stages):
        a, c = rng.uniform(5, 40), rng.uniform(1, 12)
        x, y = rng.uniform(0, 5), rng.uniform(0.2, 3)
        bs = np.arange(1, max_bs + 1)
        li, ln = a + c * bs, x + y * bs
        if integer:
            li, ln = np.ceil(li), np.ceil(ln)
        infer.append([float(v) for v in li])
        net.append([float(v) for v in ln])
    return {"infer": infer, "net": net}


def random_plan(seed: int, integer: bool = False, max_bs: int = 8):
    """A small random cluster and plan: (gpu_node, pipelines) with pipelines
    as [{"bs": .., "stages": [{"gpus", "infer", "net"}]}]; GPUs are dealt
    out to pools without sharing, nodes hold 1-3 GPUs."""
    rng = np.random.default_rng(seed)
    n_pipes = int(rng.integers(1, 4))
    shapes = [[int(rng.integers(1, 4)) for _ in range(int(rng.integers(1, 4)))]
              for _ in range(n_pipes)]
    n_gpus = sum(sum(s) for s in shapes)
    per_node = int(rng.integers(1, 4))
    gpu_node = [g // per_node for g in range(n_gpus)]
    order = rng.permutation(n_gpus)
    pipes, k = [], 0
    for s in shapes:
        tab = random_tables(rng, len(s), max_bs, integer)
        stages = []
        for i, m in enumerate(s):
            stages.append({"gpus": [int(g) for g in order[k:k + m]],
                           "infer": tab["infer"][i], "net": tab["net"][i]})
            k += m
        pipes.append({"bs": int(rng.integers(1, max_bs + 1)), "stages": stages})
    return gpu_node, pipes


def plan_capacity_per_us(pipes: Sequence[dict]) -> float:
    """Requests per us the plan sustains at its unified batch sizes: per
    pipeline the slowest pool (pool GPUs x bs / stage latency), summed."""
    tot = 0.0
    for p in pipes:
        b = p["bs"]
        tot += min(len(s["gpus"]) * b / s["infer"][b - 1] for s in p["stages"])
    return tot
