"""The native planner (gs_rlg_build, gs_lp_partition, gs_sds_order: host C++
behind the C ABI) against the oracle, bit for bit: retained graph and
weights, groups, coupling summary and rounds, group cycle, view order, unit
groups and transition summaries.  Synthetic aerial captures (flight-grid
tracks with long outliers) of 1 to 1000 views and hand-made edge cases;
at 50,000 views (the largest capture the paper times) sampled views and
units are checked one by one against the oracle's Eq. 1 and the Eq. 2 rule.
These run on the CPU: the planner is host code."""
import numpy as np
import pytest


@pytest.fixture(scope="module")
def gs():
    from paper_2607_19893_amd import gsmi
    return gsmi


def run_native(gs, c, cap, k, K, iters, B):
    G = gs.gs_rlg_build(c.item_ptr, c.item_tracks, c.n_tracks, cap, k)
    group, C, rounds = gs.gs_lp_partition(c.position, G, K, iters)
    cycle, order, ug, tr = gs.gs_sds_order(group, C, G, B)
    return G, group, C, rounds, cycle, order, ug, tr


def run_oracle(orc, c, cap, k, K, iters, B):
    R = orc.rlg_build([c.tracks_of(i) for i in range(c.n)], c.n_tracks, cap, k)
    P = orc.lp_partition(c.position, R, K, iters)
    S = orc.sds_order(P.group, P.coupling, K, R, B)
    return R, P, S


def bits(a):
    return np.ascontiguousarray(a, np.float64).view(np.int64)


def assert_same(nat, ref):
    G, group, C, rounds, cycle, order, ug, tr = nat
    R, P, S = ref
    np.testing.assert_array_equal(G.edge_ptr, R.edge_ptr)
    np.testing.assert_array_equal(G.edge_dst, R.edge_dst)
    np.testing.assert_array_equal(bits(G.edge_w), bits(R.edge_w))
    np.testing.assert_array_equal(group, P.group)
    np.testing.assert_array_equal(bits(C), bits(P.coupling))
    assert rounds == P.iters
    np.testing.assert_array_equal(cycle, S.cycle)
    np.testing.assert_array_equal(order, S.order)
    np.testing.assert_array_equal(ug, S.unit_group)
    np.testing.assert_array_equal(bits(tr), bits(S.transition))


CASES = [  # n, seed, track cap, top-k, K, rounds, unit size
    (1, 0, 64, 16, 4, 20, 2),
    (2, 1, 0, 0, 1, 5, 1),
    (7, 2, 0, 0, 3, 20, 2),
    (30, 3, 1, 4, 4, 20, 2),
    (100, 4, 40, 8, 4, 20, 3),
    (257, 5, 64, 16, 5, 20, 7),
    (220, 6, 0, 0, 4, 3, 2),
    (1000, 7, 64, 16, 4, 20, 2),
    (1000, 8, 64, 1, 8, 20, 1),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "n%d-cap%d-k%d-K%d-B%d" % (c[0], c[2], c[3], c[4], c[6]))
def test_native_matches_oracle(gs, orc, case):
    from paper_2607_19893_amd import scenes
    n, seed, cap, k, K, iters, B = case
    c = scenes.capture_tracks(n, seed=seed)
    assert_same(run_native(gs, c, cap, k, K, iters, B), run_oracle(orc, c, cap, k, K, iters, B))


def test_edge_cases(gs, orc):
    from paper_2607_19893_amd import scenes
    # views without tracks, K above n, a unit larger than the capture, a track cap that drops everything shared
    c = scenes.capture_tracks(40, seed=9)
    lists = [c.tracks_of(i) for i in range(c.n)]
    for i in (0, 5, 6, 39):
        lists[i] = lists[i][:0]
    ptr = np.zeros(c.n + 1, np.int64)
    np.cumsum([len(x) for x in lists], out=ptr[1:])
    c2 = scenes.Capture("holes", c.position, ptr, np.concatenate(lists).astype(np.int32), c.n_tracks)
    for cap, k, K, B in ((0, 0, 4, 2), (64, 3, 50, 1), (1, 2, 3, 100), (0, 5, 1, 40)):
        assert_same(run_native(gs, c2, cap, k, K, 20, B), run_oracle(orc, c2, cap, k, K, 20, B))
    # no views at all
    G = gs.gs_rlg_build(np.zeros(1, np.int64), np.zeros(0, np.int32), 0, 0, 4)
    assert G.edge_ptr.tolist() == [0] and G.edge_dst.size == 0
    group, C, rounds = gs.gs_lp_partition(np.zeros((0, 3)), G, 3, 5)
    assert group.size == 0 and rounds == 0 and not C.any()
    cycle, order, ug, tr = gs.gs_sds_order(group, C, G, 2)
    assert cycle.size == 0 and order.size == 0 and ug.size == 0


def test_malformed_inputs_rejected(gs):
    import ctypes
    L = gs.raw()
    ptr = np.array([0, 2, 3], np.int64)
    bad_order = np.array([3, 1, 2], np.int32)            # view 0's tracks not ascending
    with pytest.raises(gs.GsmiError, match="ascending"):
        gs.gs_rlg_build(ptr, bad_order, 4, 0, 0)
    with pytest.raises(gs.GsmiError, match="outside"):
        gs.gs_rlg_build(ptr, np.array([0, 1, 9], np.int32), 4, 0, 0)
    with pytest.raises(gs.GsmiError, match="decreases"):
        gs.gs_rlg_build(np.array([0, 2, 1], np.int64), np.array([0, 1], np.int32), 4, 0, 0)
    G = gs.gs_rlg_build(ptr, np.array([0, 1, 1], np.int32), 4, 0, 0)
    with pytest.raises(gs.GsmiError, match="K and max_iters"):
        gs.gs_lp_partition(np.zeros((2, 3)), G, 0, 5)
    with pytest.raises(gs.GsmiError, match="not finite"):
        gs.gs_lp_partition(np.array([[0, 0, 0], [np.nan, 0, 0]]), G, 2, 5)
    with pytest.raises(gs.GsmiError, match="outside"):
        gs.gs_sds_order(np.array([0, 3], np.int32), np.zeros((2, 2)), G, 1)
    asym = gs.PlanGraph(np.array([0, 1, 1], np.int64), np.array([0], np.int32), np.array([0.5]))
    with pytest.raises(gs.GsmiError, match="neighbour"):
        gs.gs_sds_order(np.array([0, 1], np.int32), np.zeros((2, 2)), asym, 1)
    # a graph too large for the caller's arrays: the needed count comes back, nothing is written
    ne = ctypes.c_int64(0)
    ep = np.full(3, -7, np.int64)
    st = L.gs_rlg_build(2, 4, ctypes.c_void_p(ptr.ctypes.data), ctypes.c_void_p(np.array([0, 1, 1], np.int32).ctypes.data),
                        0, 0, ctypes.c_void_p(ep.ctypes.data), None, None, 0, ctypes.byref(ne))
    assert st == gs.GS_ERR_WORKSPACE and ne.value == 2 and ep.tolist() == [-7, -7, -7]


def test_full_capture_sampled(gs, orc):
    """50,000 views: sampled views' retained weights equal the oracle's Eq. 1
    on their kept track sets and each holds its own top-k; groups in the
    refinement's size band;
    the order a permutation with full units; sampled units follow Eq. 2."""
    from paper_2607_19893_amd import scenes
    n, cap, k, K, B = 50_000, 64, 16, 4, 2
    c = scenes.capture_tracks(n, seed=5)
    G, group, C, rounds, cycle, order, ug, tr = run_native(gs, c, cap, k, K, 20, B)
    length = np.bincount(c.item_tracks, minlength=c.n_tracks)
    keep = length <= cap
    P = lambda i: set(int(t) for t in c.tracks_of(i) if keep[t])
    rng = np.random.default_rng(1)
    for i in rng.choice(n, 40, replace=False):
        Pi = P(i)
        nb = {int(j): float(w) for j, w in zip(G.edge_dst[G.edge_ptr[i]:G.edge_ptr[i + 1]],
                                                G.edge_w[G.edge_ptr[i]:G.edge_ptr[i + 1]])}
        for j, w in nb.items():
            assert orc.jaccard(Pi, P(j)) == w
        # candidates of view i: every view sharing one of its kept tracks (searched in the CSR)
        own = np.zeros(c.n_tracks, bool)
        own[list(Pi)] = True
        hit = own[c.item_tracks]
        cand = set(np.searchsorted(c.item_ptr, np.nonzero(hit)[0], side="right") - 1) - {i}
        ranked = sorted(((orc.jaccard(Pi, P(j)), j) for j in cand), key=lambda x: (-x[0], x[1]))[:k]
        for w, j in ranked:
            assert nb.get(int(j)) == w
    top = -(-n // K)
    slack = max(1, top // 16)
    sizes = np.bincount(group, minlength=K)
    assert sizes.max() <= top + slack and sizes.min() >= n // K - slack     # the refinement's band
    assert np.array_equal(np.sort(order), np.arange(n))
    assert len(ug) == -(-n // B)
    edges = lambda u: dict(zip(G.edge_dst[G.edge_ptr[u]:G.edge_ptr[u + 1]].tolist(),
                               G.edge_w[G.edge_ptr[u]:G.edge_ptr[u + 1]].tolist()))
    pos_of = np.empty(n, np.int64)
    pos_of[order] = np.arange(n)
    for t in sorted(rng.choice(len(ug) - 1, 30, replace=False) + 1):
        prev, unit = order[(t - 1) * B:t * B], order[t * B:(t + 1) * B]
        s = lambda v: orc.score(int(v), [int(u) for u in prev], orc.RLG(G.edge_ptr, G.edge_dst, G.edge_w))
        for g in set(group[unit].tolist()):
            later = [v for v in np.nonzero(group == g)[0] if pos_of[v] >= (t + 1) * B]
            best_later = min(((s(v), int(v)) for v in later), default=None)
            for a in unit[group[unit] == g]:
                if best_later is not None:
                    assert (s(a), int(a)) < best_later
        w_max = max([edges(int(u)).get(int(v), 0.0) for u in prev for v in unit], default=0.0)
        assert tr[t] == w_max
