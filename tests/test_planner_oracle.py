"""Pins of the oracle's ahead-of-time planner against facts that do not come
from the oracle itself:
  * Eq. 1 on a hand-worked five-view example (weights, top-k retention with
    a tie, the outlier cap), each value derived by hand from the track sets;
  * brute force over every view pair of tiny random track lists with exact
    fractions, without the inverse track mapping;
  * logical partitioning on hand-worked point sets (the capacity decides one
    view), well-separated blobs recovered exactly, the coupling summary of a
    hand graph;
  * static data scheduling: a hand-derived group cycle, a worked six-view
    schedule of Eq. 2 with its transition summaries, the top-up of a unit
    from the next group, and the Eq. 2 rule checked unit by unit on dyadic
    weights (exact sums) of larger random schedules;
  * each planted mistake (16-21) fails at least one pin.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest


def graph_dict(R):
    return {i: dict(R.neighbours(i)) for i in range(len(R.edge_ptr) - 1)}


# ---------------------------------------------------------------------------
# relative locality graph (Section 4.1.1, Eq. 1)
# ---------------------------------------------------------------------------

# track sets: v0 {0,1,2}, v1 {1,2,3}, v2 {3,4}, v3 {} (no tracks), v4 {0,1,2}
EX_TRACKS = [[0, 1, 2], [1, 2, 3], [3, 4], [], [0, 1, 2]]


def check_rlg_example(o):
    # all neighbours: w01 = 2/4, w04 = 3/3, w12 = 1/4, w14 = 2/4; v0-v2 share nothing, v3 has no tracks
    g = graph_dict(o.rlg_build(EX_TRACKS, 6, 0, 0))
    assert g == {0: {1: 0.5, 4: 1.0}, 1: {0: 0.5, 2: 0.25, 4: 0.5}, 2: {1: 0.25}, 3: {}, 4: {0: 1.0, 1: 0.5}}
    # top-1: v0 keeps v4 (1.0), v1 keeps v0 (0.5, tie with v4 broken by id), v2 keeps v1, v4 keeps v0;
    # v1-v4 is kept by neither end and drops out; v1-v2 stays because v2 keeps it
    g = graph_dict(o.rlg_build(EX_TRACKS, 6, 0, 1))
    assert g == {0: {1: 0.5, 4: 1.0}, 1: {0: 0.5, 2: 0.25}, 2: {1: 0.25}, 3: {}, 4: {0: 1.0}}
    # cap 2: tracks 1 and 2 (three views each) are outliers; P0 = P4 = {0}, P1 = {3}, P2 = {3, 4}
    g = graph_dict(o.rlg_build(EX_TRACKS, 6, 2, 0))
    assert g == {0: {4: 1.0}, 1: {2: 0.5}, 2: {1: 0.5}, 3: {}, 4: {0: 1.0}}
    # Eq. 1 directly; an empty union gives 0
    assert o.jaccard({1, 2}, {2, 3}) == 1 / 3 and o.jaccard(set(), set()) == 0.0


def test_rlg_worked_example(orc):
    check_rlg_example(orc)


def brute_force_graph(tracks, n_tracks, cap, k):
    """Every view pair, exact fractions, no inverse mapping."""
    n = len(tracks)
    length = [sum(t in set(ts) for ts in tracks) for t in range(n_tracks)]
    P = [set(t for t in ts if cap <= 0 or length[t] <= cap) for ts in tracks]
    w = {}
    for i, j in itertools.permutations(range(n), 2):
        inter = len(P[i] & P[j])
        if inter:
            w[i, j] = Fraction(inter, len(P[i] | P[j]))
    kept = set()
    for i in range(n):
        ranked = sorted((j for j in range(n) if (i, j) in w), key=lambda j: (-w[i, j], j))
        for j in (ranked[:k] if k > 0 else ranked):
            kept.add(frozenset((i, j)))
    g = {i: {} for i in range(n)}
    for e in kept:
        i, j = sorted(e)
        g[i][j] = float(w[i, j])
        g[j][i] = float(w[i, j])
    return g


def check_rlg_brute_force(o, trials=60):
    rng = np.random.default_rng(7)
    for _ in range(trials):
        n = int(rng.integers(1, 8))
        nt = int(rng.integers(1, 12))
        tracks = [sorted(set(rng.integers(0, nt, int(rng.integers(0, 6))).tolist())) for _ in range(n)]
        cap = int(rng.integers(0, 5))
        k = int(rng.integers(0, 4))
        assert graph_dict(o.rlg_build(tracks, nt, cap, k)) == brute_force_graph(tracks, nt, cap, k), (tracks, cap, k)


def test_rlg_brute_force(orc):
    check_rlg_brute_force(orc)


def test_rlg_invariants(orc):
    from paper_2607_19893_amd import scenes
    c = scenes.capture_tracks(300, seed=3)
    tracks = [c.tracks_of(i) for i in range(c.n)]
    full = orc.rlg_build(tracks, c.n_tracks, 64, 0)
    for k in (1, 4, 16):
        R = orc.rlg_build(tracks, c.n_tracks, 64, k)
        g = graph_dict(R)
        for i, nb in g.items():
            for j, w in nb.items():
                assert 0.0 < w <= 1.0 and g[j][i] == w and full.weight(i, j) == w
            # at least min(k, candidates) neighbours, and every retained edge is some end's top-k choice
            assert len(nb) >= min(k, len(full.neighbours(i)))
    # k >= n - 1 keeps every pair that shares a track
    R = orc.rlg_build(tracks, c.n_tracks, 64, c.n)
    assert graph_dict(R) == graph_dict(full)


# ---------------------------------------------------------------------------
# logical partitioning (Section 4.2, LP)
# ---------------------------------------------------------------------------

def empty_graph(o, n):
    return o.RLG(np.zeros(n + 1, np.int64), np.zeros(0, np.int32), np.zeros(0))


def line(xs):
    xs = np.asarray(xs, float)
    return np.stack([xs, np.zeros_like(xs), np.zeros_like(xs)], 1)


def check_lp_examples(o):
    # x = 0, 1, 10, 11, K = 2: seeds v0 and v3 (farthest), pairs by distance, then a repeat ends it
    P = o.lp_partition(line([0, 1, 10, 11]), empty_graph(o, 4), 2, 10)
    assert list(P.group) == [0, 0, 1, 1] and P.iters == 2
    # capacity ceil(5/2) = 3: v3 at 0.3 goes to the far group because the near one is full
    P = o.lp_partition(line([0, 0.1, 0.2, 0.3, 100]), empty_graph(o, 5), 2, 10)
    assert list(P.group) == [0, 0, 0, 1, 1]
    # K = 1: everything in group 0
    P = o.lp_partition(line(np.arange(7.0)), empty_graph(o, 7), 1, 10)
    assert list(P.group) == [0] * 7
    # coupling summary of a hand graph: 0-1 (1/2), 1-2 (1/4), 2-3 (1/2); groups {0,1}, {2,3}
    R = o.RLG(np.array([0, 1, 3, 5, 6]), np.array([1, 0, 2, 1, 3, 2], np.int32),
              np.array([0.5, 0.5, 0.25, 0.25, 0.5, 0.5]))
    P = o.lp_partition(line([0, 1, 10, 11]), R, 2, 10)
    assert list(P.group) == [0, 0, 1, 1]
    assert P.coupling.tolist() == [[0.5, 0.25], [0.25, 0.5]]


def check_lp_refinement(o):
    # two clusters of four on a line, K = 2: k-means puts views 0-3 and 4-7 together; view 3's
    # retained edges go mostly to views 4-6 (7/8 each) and weakly to view 0 (1/8), so the
    # refinement moves it (band 4 +- 1: group sizes 3 and 5 allowed) and nothing else moves
    edges = [(0, 1, 0.5), (1, 2, 0.5), (0, 2, 0.5), (0, 3, 0.125), (3, 4, 0.875), (3, 5, 0.875),
             (3, 6, 0.875), (4, 5, 0.5), (5, 6, 0.5), (6, 7, 0.5)]
    R = hand_graph(o, 8, edges)
    pos = line([0, 0.1, 0.2, 0.3, 10, 10.1, 10.2, 10.3])
    P = o.lp_partition(pos, R, 2, 10)
    assert list(P.group) == [0, 0, 0, 1, 1, 1, 1, 1]
    # within: {0,1,2} 3 x 1/2; {3..7} 3 x 7/8 + 3 x 1/2; across: the 0-3 edge
    assert P.coupling.tolist() == [[1.5, 0.125], [0.125, 4.125]]
    # three clusters of four at x = 0, 10, 20, K = 3 (k-means groups 0, 2, 1 by the seeding order):
    # the first cluster's views tied to each other (1 each) and to every other view (3/4 each),
    # so they gain nothing by moving; the others gain 3 by joining group 0, but only view 4 (the
    # first in ascending order) may: group 0 is then at the band's top (4 + 1)
    edges = [(i, j, 1.0) for i in range(4) for j in range(i + 1, 4)]
    edges += [(i, j, 0.75) for i in range(4) for j in range(4, 12)]
    pos3 = line([0, 0.1, 0.2, 0.3, 10, 10.1, 10.2, 10.3, 20, 20.1, 20.2, 20.3])
    P = o.lp_partition(pos3, hand_graph(o, 12, edges), 3, 10)
    assert [int(g) for g in P.group] == [0, 0, 0, 0, 0, 2, 2, 2, 1, 1, 1, 1], list(P.group)


def cut_weight(R, group):
    return sum(w for i in range(len(group)) for j, w in R.neighbours(i) if j > i and group[i] != group[j])


def test_lp_worked_examples(orc):
    check_lp_examples(orc)
    check_lp_refinement(orc)


def test_lp_refinement_lowers_the_cut(orc):
    """On random captures the refinement never raises the weight across
    groups, keeps the sizes in the band, and leaves a partition in which no
    single move within the band would lower the cut."""
    for seed in range(4):
        rng = np.random.default_rng(seed)
        n = 60
        pos = rng.normal(0, 1, (n, 3))
        edges = [(i, j, float(rng.integers(1, 9)) / 8.0) for i in range(n) for j in range(i + 1, n)
                 if rng.random() < 0.08]
        R = hand_graph(orc, n, edges)
        K = 3
        orc.set_mutation(27)
        try:
            P0 = orc.lp_partition(pos, R, K, 20)
        finally:
            orc.set_mutation(0)
        P = orc.lp_partition(pos, R, K, 20)
        assert cut_weight(R, P.group) <= cut_weight(R, P0.group)
        top = -(-n // K)
        slack = max(1, top // 16)
        sizes = np.bincount(P.group, minlength=K)
        assert sizes.min() >= n // K - slack and sizes.max() <= top + slack
        # local optimality within the band (when the passes ended by themselves)
        g = list(P.group)
        for u in range(n):
            W = np.zeros(K)
            for j, w in R.neighbours(u):
                W[g[j]] += w
            for b in range(K):
                if b != g[u] and sizes[b] < top + slack and sizes[g[u]] > n // K - slack:
                    assert W[b] <= W[g[u]], (seed, u, b)


def test_lp_blobs_and_balance(orc):
    rng = np.random.default_rng(0)
    cent = np.array([[0, 0, 0], [100, 0, 0], [0, 100, 0], [0, 0, 100]], float)
    for sizes in ([5, 5, 5, 5], [4, 4, 4, 4]):
        pts = np.concatenate([c + rng.normal(0, 1, (s, 3)) for c, s in zip(cent, sizes)])
        lab = np.repeat(np.arange(4), sizes)
        o_ = rng.permutation(len(pts))
        P = orc.lp_partition(pts[o_], empty_graph(orc, len(pts)), 4, 50)
        got = {frozenset(np.nonzero(P.group == g)[0]) for g in range(4)}
        want = {frozenset(np.nonzero(lab[o_] == b)[0]) for b in range(4)}
        assert got == want
    # balance on a random cloud: no group above ceil(n / K)
    pts = rng.normal(0, 1, (103, 3))
    for K in (2, 3, 4, 7):
        P = orc.lp_partition(pts, empty_graph(orc, 103), K, 30)
        assert np.bincount(P.group, minlength=K).max() <= -(-103 // K)


# ---------------------------------------------------------------------------
# static data scheduling (Section 4.2, SDS, Eq. 2)
# ---------------------------------------------------------------------------

def hand_graph(o, n, edges):
    nb = {i: {} for i in range(n)}
    for i, j, w in edges:
        nb[i][j] = w
        nb[j][i] = w
    ptr, dst, wt = [0], [], []
    for i in range(n):
        for j in sorted(nb[i]):
            dst.append(j)
            wt.append(nb[i][j])
        ptr.append(len(dst))
    return o.RLG(np.array(ptr, np.int64), np.array(dst, np.int32), np.array(wt))


def check_sds_examples(o):
    # cycle: from group 0 the least coupled is 2 (1), then from 2: 1 (5) before 3 (6), then 3
    C = np.array([[0, 3, 1, 2], [3, 0, 5, 4], [1, 5, 0, 6], [2, 4, 6, 0]], float)
    assert o.group_cycle(np.array([0, 1, 2, 3]), C, 4) == [0, 2, 1, 3]
    # six views, groups {0,1,2} and {3,4,5}, edges 0-3 (1/2), 1-4 (1/4), 2-5 (3/4), 1-5 (1/8), units of one view:
    #   U1 = {0} (no previous unit); U2 from group 1 against {0}: s(3) = 1/2, s(4) = s(5) = 0 -> 4;
    #   U3 against {4}: s(1) = 1/4, s(2) = 0 -> 2; U4 against {2}: s(3) = 0, s(5) = 3/4 -> 3;
    #   U5 = {1}; U6 = {5}, and the last transition carries w(1, 5) = 1/8
    R = hand_graph(o, 6, [(0, 3, 0.5), (1, 4, 0.25), (2, 5, 0.75), (1, 5, 0.125)])
    S = o.sds_order(np.array([0, 0, 0, 1, 1, 1]), np.array([[0, 1.625], [1.625, 0]]), 2, R, 1)
    assert list(S.cycle) == [0, 1]
    assert list(S.order) == [0, 4, 2, 3, 1, 5]
    assert list(S.unit_group) == [0, 1, 0, 1, 0, 1]
    assert list(S.transition) == [0, 0, 0, 0, 0, 0.125]
    # the same with units of three: U1 = {0, 1, 2}; U2 = group 1 against it, s = 1/2, 1/4, 7/8 -> all three;
    # the transition is the largest single weight, 3/4
    S = o.sds_order(np.array([0, 0, 0, 1, 1, 1]), np.array([[0, 1.625], [1.625, 0]]), 2, R, 3)
    assert list(S.order) == [0, 1, 2, 4, 3, 5] and list(S.transition) == [0, 0.75]
    # top-up: group 0 holds one view, units of two: U1 = {0} + the first of group 1, then group 1 alone
    S = o.sds_order(np.array([0, 1, 1, 1, 1]), np.zeros((2, 2)), 2, empty_graph(o, 5), 2)
    assert list(S.order) == [0, 1, 2, 3, 4] and list(S.unit_group) == [0, 1, 1]
    # an empty group is left out of the cycle
    S = o.sds_order(np.array([2, 0, 2, 0]), np.zeros((3, 3)), 3, empty_graph(o, 4), 1)
    assert list(S.cycle) == [0, 2] and list(S.order) == [1, 0, 3, 2]


def test_sds_worked_examples(orc):
    check_sds_examples(orc)


def check_sds_rule(o, seed=3):
    """Unit by unit on dyadic weights (exact sums): every view a unit takes from
    a group scores no higher than any view that group keeps (Eq. 2, id breaks
    ties), units take turns over the cycle, and the transition is the largest
    weight between consecutive units."""
    rng = np.random.default_rng(seed)
    n, K, B = 60, 3, 4
    edges = {}
    for _ in range(200):
        i, j = rng.integers(0, n, 2)
        if i != j:
            edges[min(i, j), max(i, j)] = float(rng.integers(1, 9)) / 8.0
    R = hand_graph(o, n, [(i, j, w) for (i, j), w in edges.items()])
    group = rng.integers(0, K, n)
    C = rng.integers(0, 10, (K, K)).astype(float)
    C = C + C.T
    S = o.sds_order(group, C, K, R, B)
    assert sorted(S.order) == list(range(n))
    w = lambda u, v: edges.get((min(u, v), max(u, v)), 0.0)
    left = set(range(n))
    prev = []
    for t in range(len(S.unit_group)):
        unit = list(S.order[t * B:(t + 1) * B])
        assert len(unit) == B or t == len(S.unit_group) - 1
        s = lambda v: sum(Fraction(w(u, v)) for u in prev)
        for g in set(group[unit]):
            took = [v for v in unit if group[v] == g]
            kept = [v for v in left if group[v] == g and v not in unit]
            for a in took:
                for b in kept:
                    assert (s(a), a) < (s(b), b), (t, a, b)
        assert S.transition[t] == max([w(u, v) for u in prev for v in unit], default=0.0)
        left -= set(unit)
        prev = unit
    # units take turns: each unit starts at the cycle's next group that still has views
    assert S.unit_group[0] == S.cycle[0]


def test_sds_rule_on_random_schedules(orc):
    for seed in range(4):
        check_sds_rule(orc, seed)


# ---------------------------------------------------------------------------
# planted mistakes
# ---------------------------------------------------------------------------

PLANNER_MUTATIONS = {16: check_rlg_example, 17: check_rlg_example, 18: check_rlg_brute_force,
                     19: check_lp_examples, 20: check_sds_examples, 21: check_sds_examples,
                     27: check_lp_refinement, 28: check_lp_refinement}


@pytest.mark.parametrize("k", sorted(PLANNER_MUTATIONS))
def test_pins_catch_planted_mistake(orc, k):
    orc.set_mutation(k)
    try:
        with pytest.raises(AssertionError):
            PLANNER_MUTATIONS[k](orc)
    finally:
        orc.set_mutation(0)
