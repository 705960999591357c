"""Oracle of the ahead-of-time planner -- TEST INFRASTRUCTURE ONLY.

Only the test suite and ``bench.py``'s timing of the planner may import this
module (through the ``oracle`` package).  It shares no code with the native
planner in ``paper_2607_19893_amd``.  Plain Python sets, dicts and loops,
in the order the paper describes the steps; every floating-point result is
one IEEE double operation sequence written out below, so a native planner
that performs the same operations in the same order agrees bit for bit.

What each function follows:
  * ``rlg_build``: the relative locality graph (Section 4.1.1, Eq. 1): the
    weight of two views is the Jaccard similarity of their track sets; an
    empty union gives 0 and a missing edge means weight 0.  Shared-track
    counts come from the inverse track-to-view mapping; tracks seen by more
    than ``track_cap`` views are left out of both views' sets (the outlier
    cap); each view keeps its ``top_k`` strongest neighbours (weight
    descending, then view id ascending) and an edge is retained when either
    end keeps it.
  * ``lp_partition``: logical partitioning (Section 4.2, LP) into K groups
    by balanced k-means over the camera centres (MacQueen / Lloyd
    iterations with a capacity of ceil(n / K) views per group), seeded by
    farthest-point selection from view 0, then refined on the RLG so that
    strong coupling stays within groups: in passes over the views in
    ascending order, a view moves to the group its retained edges weigh most
    towards when that weight exceeds the weight towards its own group, within
    a balance band of the group sizes (floor(n / K) - s .. ceil(n / K) + s,
    s = max(1, ceil(n / K) // 16)), until a pass moves nothing (at most
    ``REFINE_PASSES``); the region-level coupling summary is the sum of
    retained edge weights between (and within) groups.
  * ``sds_order``: static data scheduling (Section 4.2, SDS, Eq. 2): a cyclic
    traversal of the non-empty groups that starts at the first one and
    repeatedly moves to the least-coupled unvisited group; task units of
    ``unit_size`` views take turns over that cycle, each filled from its
    group with the candidates of lowest score s(v | U_prev) = sum of w_uv
    over the previous unit (view id breaks ties), topped up from the next
    groups of the cycle when its group runs out; two consecutive units are
    summarized by their largest retained view-pair weight.
"""
from __future__ import annotations

import dataclasses
from typing import List, Sequence

import numpy as np


def _mut() -> int:
    from . import _MUT      # the package's current planted-mistake switch
    return _MUT


@dataclasses.dataclass
class RLG:
    edge_ptr: np.ndarray     # [n + 1] int64
    edge_dst: np.ndarray     # int32, ascending within a view
    edge_w: np.ndarray       # float64

    def weight(self, i: int, j: int) -> float:
        a, b = int(self.edge_ptr[i]), int(self.edge_ptr[i + 1])
        k = np.searchsorted(self.edge_dst[a:b], j)
        if k < b - a and int(self.edge_dst[a + k]) == j:
            return float(self.edge_w[a + k])
        return 0.0

    def neighbours(self, i: int):
        a, b = int(self.edge_ptr[i]), int(self.edge_ptr[i + 1])
        return [(int(j), float(w)) for j, w in zip(self.edge_dst[a:b], self.edge_w[a:b])]


def track_sets(item_tracks: Sequence[Sequence[int]], n_tracks: int, track_cap: int) -> List[set]:
    """Each view's set of tracks after the outlier cap (tracks seen by more
    than ``track_cap`` views are dropped; ``track_cap`` <= 0 keeps all)."""
    length = [0] * n_tracks
    for ts in item_tracks:
        for t in ts:
            length[int(t)] += 1
    keep = [track_cap <= 0 or length[t] <= track_cap for t in range(n_tracks)]
    if _mut() == 16:                             # planted: the cap keeps only the long tracks
        keep = [not k for k in keep]
    return [set(int(t) for t in ts if keep[int(t)]) for ts in item_tracks]


def jaccard(Pi: set, Pj: set) -> float:
    """Eq. 1; an empty union gives 0."""
    union = len(Pi | Pj)
    if union == 0:
        return 0.0
    if _mut() == 17:                             # planted: intersection over the smaller set
        return len(Pi & Pj) / min(len(Pi), len(Pj))
    return len(Pi & Pj) / union


def rlg_build(item_tracks: Sequence[Sequence[int]], n_tracks: int, track_cap: int, top_k: int) -> RLG:
    n = len(item_tracks)
    P = track_sets(item_tracks, n_tracks, track_cap)
    # inverse mapping: the views of each kept track
    views_of = {}
    for i, s in enumerate(P):
        for t in s:
            views_of.setdefault(t, []).append(i)
    # candidate neighbours: views that share at least one kept track
    cand = [set() for _ in range(n)]
    for vs in views_of.values():
        for i in vs:
            for j in vs:
                if i != j:
                    cand[i].add(j)
    keep = [set() for _ in range(n)]
    for i in range(n):
        ranked = sorted(((jaccard(P[i], P[j]), j) for j in cand[i]), key=lambda x: (-x[0], x[1]))
        if top_k > 0:
            ranked = ranked[:top_k]
        for _, j in ranked:
            keep[i].add(j)
            if _mut() != 18:                     # planted: an edge kept by one end only is one-sided
                keep[j].add(i)
    ptr = np.zeros(n + 1, np.int64)
    dst, wts = [], []
    for i in range(n):
        for j in sorted(keep[i]):
            dst.append(j)
            wts.append(jaccard(P[i], P[j]))
        ptr[i + 1] = len(dst)
    return RLG(ptr, np.array(dst, np.int32), np.array(wts, np.float64))


def _sqdist(p, c) -> float:
    dx = p[0] - c[0]
    dy = p[1] - c[1]
    dz = p[2] - c[2]
    return dx * dx + dy * dy + dz * dz


REFINE_PASSES = 16


def refine_groups(group: List[int], rlg: RLG, K: int) -> None:
    """The LP refinement (module docstring), in place.  A view's weight
    towards each group is the sum of its retained edge weights, neighbours in
    ascending order; the move goes to the group of largest gain over the own
    group (the lowest such group on ties), if the gain is positive, that group
    is below the band's top and the own group above its bottom."""
    n = len(group)
    if n == 0 or K < 2:
        return
    base, top = n // K, -(-n // K)
    slack = max(1, top // 16)
    lo, hi = base - slack, top + slack
    size = [0] * K
    for g in group:
        size[g] += 1
    for _ in range(REFINE_PASSES):
        moved = False
        for u in range(n):
            a = group[u]
            W = [0.0] * K
            for j, w in rlg.neighbours(u):
                W[group[j]] += w
            best, gain = -1, 0.0
            for b in range(K):
                if b != a and (size[b] < hi or _mut() == 28):      # planted (28): no top of the band
                    d = W[b] - W[a]
                    if d > gain:
                        best, gain = b, d
            if best >= 0 and size[a] > lo:
                group[u] = best
                size[a] -= 1
                size[best] += 1
                moved = True
        if not moved:
            break


@dataclasses.dataclass
class Partition:
    group: np.ndarray          # [n] int32
    coupling: np.ndarray       # [K, K] float64
    iters: int                 # assignment rounds run


def lp_partition(position: np.ndarray, rlg: RLG, K: int, max_iters: int) -> Partition:
    pos = [tuple(float(x) for x in row) for row in np.asarray(position, np.float64).reshape(-1, 3)]
    n = len(pos)
    if n == 0:
        return Partition(np.zeros(0, np.int32), np.zeros((K, K)), 0)
    cap = -(-n // K)
    # farthest-point seeds: view 0, then the view farthest from every seed so far
    centres = [pos[0]]
    near = [_sqdist(p, pos[0]) for p in pos]
    while len(centres) < K:
        far = max(range(n), key=lambda i: (near[i], -i))
        centres.append(pos[far])
        near = [min(near[i], _sqdist(pos[i], pos[far])) for i in range(n)]
    assign = None
    rounds = 0
    for _ in range(max_iters):
        rounds += 1
        # balanced assignment: (distance, view, group) ascending, each group up to its capacity
        triples = sorted((_sqdist(pos[i], centres[g]), i, g) for i in range(n) for g in range(K))
        new = [-1] * n
        count = [0] * K
        for _, i, g in triples:
            if new[i] < 0 and (count[g] < cap or _mut() == 19):   # planted (19): no capacity
                new[i] = g
                count[g] += 1
        if new == assign:
            break
        assign = new
        # centres: mean of the members, summed in ascending view order
        for g in range(K):
            sx = sy = sz = 0.0
            c = 0
            for i in range(n):
                if assign[i] == g:
                    sx += pos[i][0]
                    sy += pos[i][1]
                    sz += pos[i][2]
                    c += 1
            if c:
                centres[g] = (sx / c, sy / c, sz / c)
    if _mut() != 27:                                  # planted (27): no refinement
        refine_groups(assign, rlg, K)
    C = [[0.0] * K for _ in range(K)]
    for i in range(n):
        for j, w in rlg.neighbours(i):
            if j > i:
                a, b = assign[i], assign[j]
                C[a][b] += w
                if a != b:
                    C[b][a] += w
    return Partition(np.array(assign, np.int32), np.array(C, np.float64), rounds)


@dataclasses.dataclass
class Schedule:
    cycle: np.ndarray          # group traversal (non-empty groups)
    order: np.ndarray          # [n] views, unit after unit
    unit_group: np.ndarray     # group each unit was started from
    transition: np.ndarray     # [units] coupling with the previous unit (0 for the first)


def group_cycle(group: np.ndarray, coupling: np.ndarray, K: int) -> List[int]:
    present = sorted(set(int(g) for g in group))
    if not present:
        return []
    cycle = [present[0]]
    left = set(present[1:])
    while left:
        last = cycle[-1]
        if _mut() == 20:                         # planted: the most coupled successor
            nxt = min(left, key=lambda g: (-float(coupling[last][g]), g))
        else:
            nxt = min(left, key=lambda g: (float(coupling[last][g]), g))
        cycle.append(nxt)
        left.remove(nxt)
    return cycle


def score(v: int, prev: Sequence[int], rlg: RLG) -> float:
    """Eq. 2: sum of the retained weights between v and the previous unit (ascending view order)."""
    s = 0.0
    for u in sorted(prev):
        s += rlg.weight(u, v)
    return s


def sds_order(group: np.ndarray, coupling: np.ndarray, K: int, rlg: RLG, unit_size: int) -> Schedule:
    n = len(group)
    cycle = group_cycle(group, coupling, K)
    remaining = {g: sorted(int(i) for i in np.nonzero(np.asarray(group) == g)[0]) for g in cycle}
    left = n
    order, unit_group, transition = [], [], []
    prev: List[int] = []
    pos = 0
    L = len(cycle)
    while left:
        while not remaining[cycle[pos % L]]:
            pos += 1
        start = pos % L
        pos += 1
        unit: List[int] = []
        k = start
        while len(unit) < unit_size and left:
            while not remaining[cycle[k % L]]:
                k += 1
            g = cycle[k % L]
            ranked = sorted(remaining[g], key=lambda v: (score(v, prev, rlg), v))
            if _mut() == 21:                     # planted: highest score first
                ranked = sorted(remaining[g], key=lambda v: (-score(v, prev, rlg), v))
            take = ranked[:unit_size - len(unit)]
            for v in take:
                remaining[g].remove(v)
            unit += take
            left -= len(take)
        t = 0.0
        for u in prev:
            for v in unit:
                t = max(t, rlg.weight(u, v))
        order += unit
        unit_group.append(cycle[start])
        transition.append(t)
        prev = unit
    return Schedule(np.array(cycle, np.int32), np.array(order, np.int32), np.array(unit_group, np.int32),
                    np.array(transition, np.float64))
