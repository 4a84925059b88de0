"""Oracle for resource-reservation adaptive batching (Sec. 5.4; Alg. 1 and
Alg. 2 of the appendix).

TEST INFRASTRUCTURE ONLY: imported by the test suite, never by the library.
Plain Python written from the paper's prose and pseudocode, sharing no code
with the library.  Times are plain floats (microseconds).

Model.
* Resources: every GPU, and the uplink and the downlink of every node (the
  GPUs of a node share them).  Each resource keeps a list of reserved
  half-open intervals [start, end).
* A pooled pipeline is a list of stages; a stage has a pool of GPUs and
  latency tables infer[bs] and net[bs] (the transfer of its input feature
  map; unused for the first stage).  `bs` is the pipeline's unified batch
  size.

Readings (where the pseudocode is loose):
* earliestSlot(res, t, l) is the smallest time >= t at which all listed
  resources are free for [time, time + l).  The answer is t itself or the
  end of some reserved interval, so those candidates are tried in order.
* waitTime of a probe is the sum, over every earliestSlot call on the chosen
  path, of (slot start - time asked for).
* In a pool the first GPU (pool order) with the earliest completion wins;
  between pipelines the first with the least waiting time wins.
* Alg. 1's batch-size loop runs down to 1; no feasible size means drop.  The
  drop test is on the chosen size bs*, and what gets reserved is the probe of
  bs* (the pseudocode's `bs == 0` and `reserve(r)` are slips).
* "Wait until the queued requests are about to miss their deadline": probe
  the chosen pipeline with the queued count; the slack of the oldest deadline
  over that completion is how long the scheduler may wait.  At that wake-up
  the requests must go, so that one decision caps the batch size at the
  queue length (without the cap it would wait forever).
* Event loop: a decision round at every arrival (an arrival at the wake-up
  time is taken first) and at a pending wake-up; a round repeats decisions
  until the queue is empty or a wait is chosen.
"""
import math
from typing import Dict, List, Optional, Sequence, Tuple

INF = math.inf


class Cluster:
    """GPUs with their nodes and the reservation tables (Sec. 5.4, resource
    reservation tables for GPUs, uplinks and downlinks)."""

    def __init__(self, gpu_node: Sequence[int]):
        self.gpu_node = list(gpu_node)
        self.table: Dict[Tuple[str, int], List[Tuple[float, float]]] = {}

    def gpu(self, g):
        return ("gpu", g)

    def uplink(self, g):
        return ("ul", self.gpu_node[g])

    def downlink(self, g):
        return ("dl", self.gpu_node[g])

    def intervals(self, res):
        return self.table.get(res, [])

    def is_free(self, res, start, dur):
        """No reserved interval of `res` meets [start, start + dur)."""
        end = start + dur
        for (a, b) in self.intervals(res):
            if dur > 0:
                if a < end and start < b:
                    return False
            elif a < start < b:   # an instant is blocked only strictly inside
                return False
        return True

    def earliest_slot(self, resources, t, l):
        """Appendix A.3: earliest time >= t at which every resource in
        `resources` is free for duration l."""
        candidates = {t}
        for r in resources:
            for (_, b) in self.intervals(r):
                if b >= t:
                    candidates.add(b)
        for c in sorted(candidates):
            if all(self.is_free(r, c, l) for r in resources):
                return c
        raise AssertionError("the last interval end is always free")

    def mark_reserved(self, res, start, dur):
        if dur > 0:
            self.table.setdefault(res, []).append((start, start + dur))


class Pipeline:
    def __init__(self, stages, bs):
        """stages: list of dicts {"gpus": [...], "infer": [l(1), l(2), ...],
        "net": [...]}; bs: the unified batch size of the plan."""
        self.stages = stages
        self.bs = bs


def probe(cluster: Cluster, pipe: Pipeline, bs: int, now: float):
    """Alg. 2, probe(): stage by stage, the pool's GPU that completes the
    stage earliest given the resources' reservations.  Returns
    (path, resv, finish, wait) with resv a list of (resource, start, dur)."""
    t_g = now
    path, resv, wait = [], [], 0.0
    last = None
    for si, st in enumerate(pipe.stages):
        l_n = st["net"][bs - 1]
        l_i = st["infer"][bs - 1]
        best = None
        for g in st["gpus"]:
            t, r, w = t_g, [], 0.0
            if si > 0:   # the feature map moves over last GPU's uplink and g's downlink at once
                u, d = cluster.uplink(last), cluster.downlink(g)
                slot = cluster.earliest_slot([u, d], t, l_n)
                w += slot - t
                r += [(u, slot, l_n), (d, slot, l_n)]
                t = slot + l_n
            slot = cluster.earliest_slot([cluster.gpu(g)], t, l_i)
            w += slot - t
            r.append((cluster.gpu(g), slot, l_i))
            t = slot + l_i
            if best is None or t < best[0]:
                best = (t, g, r, w)
        t_g, last = best[0], best[1]
        path.append(best[1])
        resv += best[2]
        wait += best[3]
    return path, resv, t_g, wait


def reserve(cluster: Cluster, resv):
    """Alg. 2, reserve(): mark every probed interval as reserved."""
    for (res, start, dur) in resv:
        cluster.mark_reserved(res, start, dur)


def decide(cluster: Cluster, pipes: Sequence[Pipeline], queue: List[dict], now: float,
           deadline_wake: bool = False) -> dict:
    """One pass of Alg. 1's loop.  queue: list of {"id", "arrival",
    "deadline"} sorted by arrival; modified in place (dispatched or dropped
    requests are removed)."""
    if not queue:
        return {"kind": "idle"}
    # choose the pooled pipeline: least waiting time at its unified batch size
    p_star, t_star = None, INF
    for i, p in enumerate(pipes):
        wait = probe(cluster, p, p.bs, now)[3]
        if wait < t_star:
            p_star, t_star = i, wait
    pipe = pipes[p_star]
    deadline = queue[0]["deadline"]
    top = min(pipe.bs, len(queue)) if deadline_wake else pipe.bs
    # choose the batch size and path: the largest that meets the oldest deadline
    bs_star, found = 0, None
    for bs in range(top, 0, -1):
        path, resv, finish, _ = probe(cluster, pipe, bs, now)
        if finish <= deadline:
            bs_star, found = bs, (path, resv, finish)
            break
    if bs_star == 0:
        gone = queue.pop(0)
        return {"kind": "drop", "pipeline": p_star, "id": gone["id"]}
    if len(queue) < bs_star:
        finish_now = probe(cluster, pipe, len(queue), now)[2]
        return {"kind": "wait", "pipeline": p_star, "bs": bs_star,
                "wake": now + max(0.0, deadline - finish_now)}
    path, resv, finish = found
    reserve(cluster, resv)
    batch = queue[:bs_star]
    del queue[:bs_star]
    return {"kind": "dispatch", "pipeline": p_star, "bs": bs_star, "id": batch[0]["id"],
            "path": path, "start": resv[0][1], "finish": finish, "deadline": deadline,
            "ids": [r["id"] for r in batch], "resv": resv}


def simulate(cluster: Cluster, pipes: Sequence[Pipeline], arrivals: Sequence[float],
             slo: float) -> List[dict]:
    """Event loop over requests i = 0.. arriving at arrivals[i] with deadline
    arrivals[i] + slo; returns every non-idle decision with its time."""
    queue: List[dict] = []
    log: List[dict] = []
    nxt, wake = 0, INF
    while nxt < len(arrivals) or queue:
        ta = arrivals[nxt] if nxt < len(arrivals) else INF
        if ta <= wake:
            now, forced = ta, False
            queue.append({"id": nxt, "arrival": ta, "deadline": ta + slo})
            nxt += 1
        else:
            now, forced = wake, True
        wake = INF
        while True:
            d = decide(cluster, pipes, queue, now, forced)
            forced = False
            if d["kind"] == "idle":
                break
            d["now"] = now
            log.append(d)
            if d["kind"] == "wait":
                wake = d["wake"]
                break
    return log


def reserved_overlaps(cluster: Cluster) -> int:
    """Pairs of overlapping reservations on any resource (brute force)."""
    n = 0
    for ivs in cluster.table.values():
        for i in range(len(ivs)):
            for j in range(i + 1, len(ivs)):
                a, b = ivs[i], ivs[j]
                if a[0] < b[1] and b[0] < a[1]:
                    n += 1
    return n
