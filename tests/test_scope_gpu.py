"""GPU parity of the primitive-scope entry points (scope bitmaps, hazard sets,
throughput-first admission; Section 4.3) against the CPU oracle, through the
C ABI.  Sizes span several workgroups (8192 ids each) with ragged tails; the
full-size case takes the scopes of two consecutive views of the room workload
(1M primitives, 1920x1080) exactly as the benchmark does."""
import sys

import numpy as np
import pytest
from parity_util import target_of

pytestmark = pytest.mark.gpu

SIZES = [1, 31, 33, 8192, 100003, 1 << 20]


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_gpu():
    import torch
    assert torch.cuda.is_available(), "GPU parity tests need an MI355X"
    return torch


@pytest.fixture(scope="module")
def gs():
    from paper_2607_19893_amd import gsmi
    return gsmi


def dev_u32(torch, a):
    a = np.ascontiguousarray(a, np.uint32)
    return torch.from_numpy(a.view(np.int32).copy() if a.size else np.zeros(1, np.int32)).cuda()


def host_u32(t, k=None):
    a = t.detach().cpu().numpy().view(np.uint32)
    return a if k is None else a[:k]


def scope_on_gpu(torch, gs, ids, n, accumulate_into=None):
    """Build a scope from an id list on the GPU (ids uploaded as given)."""
    words = gs.scope_words(n)
    sc = accumulate_into if accumulate_into is not None else torch.full((max(1, words),), -1, dtype=torch.int32,
                                                                        device="cuda")
    idx = dev_u32(torch, ids)
    cnt = dev_u32(torch, [len(ids)])
    gs.gs_scope_from_ids(idx, cnt, len(ids), n, 1 if accumulate_into is not None else 0, sc)
    return sc


def random_scopes(rng, n, structured):
    """Four scopes (RA, WA, RB, WB).  structured: W+ within R+ for both units
    and B overlapping A the way consecutive views do."""
    if structured:
        RA = np.flatnonzero(rng.random(n) < 0.4)
        WA = RA[rng.random(RA.size) < 0.6]
        shift = max(1, n // 7)
        RB = np.unique(np.concatenate([(RA[rng.random(RA.size) < 0.5] + shift) % n,
                                       np.flatnonzero(rng.random(n) < 0.1)]))
        WB = RB[rng.random(RB.size) < 0.6]
        return RA, WA, RB, WB
    return tuple(np.flatnonzero(rng.random(n) < rng.random()) for _ in range(4))


@pytest.mark.parametrize("n", SIZES)
def test_scope_from_ids_and_pred(n, torch_gpu, gs, orc):
    torch = torch_gpu
    rng = np.random.default_rng(n)
    ids = rng.integers(0, n + 40, size=max(1, n // 3)).astype(np.uint32)   # unsorted, repeats, some >= n
    sc = scope_on_gpu(torch, gs, ids, n)
    torch.cuda.synchronize()
    words = gs.scope_words(n)
    np.testing.assert_array_equal(host_u32(sc, words), orc.scope_bitmap(ids, n))
    # union with a second list
    ids2 = rng.integers(0, n, size=max(1, n // 5)).astype(np.uint32)
    scope_on_gpu(torch, gs, ids2, n, accumulate_into=sc)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host_u32(sc, words), orc.scope_bitmap(np.concatenate([ids, ids2]), n))
    # from predicate arrays (uint32 and uint8), plain and accumulated
    p32 = (rng.random(n) < 0.3).astype(np.uint32) * rng.integers(1, 9, n).astype(np.uint32)
    p8 = (rng.random(n) < 0.2).astype(np.uint8)
    s2 = torch.full((max(1, words),), -1, dtype=torch.int32, device="cuda")
    gs.gs_scope_from_pred(gs.GS_PRED_U32_NONZERO, dev_u32(torch, p32), n, 0, s2)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host_u32(s2, words), orc.scope_bitmap(np.flatnonzero(p32), n))
    gs.gs_scope_from_pred(gs.GS_PRED_U8_NONZERO, torch.from_numpy(p8).cuda(), n, 1, s2)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host_u32(s2, words),
                                  orc.scope_bitmap(np.flatnonzero((p32 != 0) | (p8 != 0)), n))
    # compaction of a bitmap into ascending ids (gs_visible_set on a scope)
    out = torch.zeros(max(1, n), dtype=torch.int32, device="cuda")
    cnt = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.zeros(gs.gs_workspace_bytes(gs.GS_WS_VISIBLE_SET, n), dtype=torch.uint8, device="cuda")
    gs.gs_visible_set(gs.GS_PRED_BITMAP, s2, n, out, cnt, ws)
    torch.cuda.synchronize()
    expect = np.flatnonzero((p32 != 0) | (p8 != 0)).astype(np.uint32)
    k = int(host_u32(cnt)[0])
    assert k == expect.size
    np.testing.assert_array_equal(host_u32(out, k), expect)


def run_conflicts(torch, gs, scopes, n, want_bitmaps=True, want_ids=True):
    RA, WA, RB, WB = (scope_on_gpu(torch, gs, s, n) for s in scopes)
    words = max(1, gs.scope_words(n))
    bm = [torch.full((words,), -1, dtype=torch.int32, device="cuda") for _ in range(3)] if want_bitmaps \
        else [None] * 3
    il = [torch.full((max(1, n),), -1, dtype=torch.int32, device="cuda") for _ in range(3)] if want_ids \
        else [None] * 3
    counts = torch.full((4,), -1, dtype=torch.int32, device="cuda")
    ws = torch.zeros(gs.gs_workspace_bytes(gs.GS_WS_SCOPE, n), dtype=torch.uint8, device="cuda")
    gs.gs_scope_conflicts(RA, WA, RB, WB, n, bm[0], bm[1], bm[2], il[0], il[1], il[2], counts, ws)
    torch.cuda.synchronize()
    return (RA, WA, RB, WB), bm, il, host_u32(counts), ws


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("structured", [True, False])
def test_scope_conflicts(n, structured, torch_gpu, gs, orc):
    torch = torch_gpu
    rng = np.random.default_rng(1000 + n)
    scopes = random_scopes(rng, n, structured)
    _, bm, il, counts, _ = run_conflicts(torch, gs, scopes, n)
    ref = orc.scope_conflicts(*scopes)
    words = gs.scope_words(n)
    assert list(counts) == [r.size for r in ref] + [len(set(scopes[2].tolist()))]
    for b, l, r in zip(bm, il, ref):
        np.testing.assert_array_equal(host_u32(b, words), orc.scope_bitmap(r, n))
        np.testing.assert_array_equal(host_u32(l, r.size), r)


def test_scope_conflicts_edge_cases(torch_gpu, gs, orc):
    torch = torch_gpu
    E = np.zeros(0, np.int64)
    for n in (0, 1, 64, 8193):
        full = np.arange(n)
        for scopes in ((E, E, E, E), (full, full, full, full), (full, E, full, E), (full, E, E, full)):
            _, bm, il, counts, _ = run_conflicts(torch, gs, scopes, n)
            ref = orc.scope_conflicts(*scopes)
            assert list(counts) == [r.size for r in ref] + [len(scopes[2])]
            if n:
                for l, r in zip(il, ref):
                    np.testing.assert_array_equal(host_u32(l, r.size), r)
    # hazards without any output list or bitmap: counts only
    rng = np.random.default_rng(5)
    scopes = random_scopes(rng, 50000, True)
    _, _, _, counts, _ = run_conflicts(torch, gs, scopes, 50000, want_bitmaps=False, want_ids=False)
    assert list(counts[:3]) == [r.size for r in orc.scope_conflicts(*scopes)]


def gate_on_gpu(torch, gs, n, RB, D, CA, g, tau, evidence=None, skip=None, version=0):
    RBs, Ds, CAs = (scope_on_gpu(torch, gs, s, n) for s in (RB, D, CA))
    Es = scope_on_gpu(torch, gs, evidence, n) if evidence is not None else None
    gd = torch.from_numpy(np.ascontiguousarray(g, np.float32)).cuda()
    sk = dev_u32(torch, skip) if skip is not None else None
    res = torch.full((16,), -1, dtype=torch.int32, device="cuda")
    ws = torch.zeros(gs.gs_workspace_bytes(gs.GS_WS_SCOPE, n), dtype=torch.uint8, device="cuda")
    args = gs.make_gate_args(CAs, gd, tau, evidence=Es, skip=sk, producer_version=version)
    gs.gs_admission_gate(RBs, Ds, args, n, res, ws)
    torch.cuda.synchronize()
    return gs.gate_result_from(res), (host_u32(sk)[:n] if sk is not None else None)


def assert_gate_equal(r, ref, what=""):
    assert (r.admit, r.reason) == (ref.admit, ref.reason), (what, r.reason, ref.reason)
    assert (r.n_read, r.n_delayed, r.n_active, r.n_missing, r.n_second) == \
        (ref.n_read, ref.n_delayed, ref.n_active, ref.n_missing, ref.n_second), what
    assert r.rho == ref.rho, what                         # both: one correctly rounded fp64 division
    assert r.max_g == ref.max_g, what                     # a max of the same fp32 values
    # the mean: an fp64 sum in another order than the oracle's exact sum
    assert abs(r.mean_g - ref.mean_g) <= 1e-12 * abs(ref.mean_g), what
    assert abs(r.threshold - ref.threshold) <= 1e-12 * abs(ref.threshold), what


def gate_cases(rng, n):
    """Scopes and magnitudes that exercise every reason code."""
    RB = np.flatnonzero(rng.random(n) < 0.5)
    CA = np.flatnonzero(rng.random(n) < 0.3)
    g = (rng.random(n) * 2.0).astype(np.float32)
    cases = []
    small = CA[:max(1, CA.size // 100)]
    g_small = g.copy()
    g_small[small] = 1e-3
    D_ok = np.intersect1d(small, RB) if np.intersect1d(small, RB).size else small[:1]
    cases.append(("admit", RB, D_ok, CA, g_small, 0.2, None))
    cases.append(("no-delay", RB, np.zeros(0, np.int64), CA, g, 0.2, None))
    cases.append(("rho", RB, RB[: max(1, RB.size // 2)], CA, g, 0.2, None))
    cases.append(("no-active", RB, RB[:3], np.zeros(0, np.int64), g, 0.9, None))
    off = np.setdiff1d(np.arange(n), CA)[:2]
    cases.append(("missing", RB, np.concatenate([CA[:2], off]), CA, g, 0.9, None))
    cases.append(("evidence", RB, np.concatenate([CA[:2], off]), CA, g_small, 0.9, np.concatenate([CA, off])))
    cases.append(("gradient", RB, CA[: max(1, CA.size // 50)], CA, g, 0.2, None))
    return [c for c in cases if n >= 64 or c[0] in ("no-delay",)]


@pytest.mark.parametrize("n", [64, 100003, 1 << 20])
def test_admission_gate(n, torch_gpu, gs, orc):
    torch = torch_gpu
    rng = np.random.default_rng(2000 + n)
    seen = set()
    for name, RB, D, CA, g, tau, ev in gate_cases(rng, n):
        r, _ = gate_on_gpu(torch, gs, n, RB, D, CA, g, tau, evidence=ev)
        ref, _ = orc.admission_gate(RB, D, CA, g, tau, evidence=ev)
        assert_gate_equal(r, ref, name)
        seen.add(ref.reason)
    assert seen >= {orc.GATE_ADMIT, orc.GATE_NO_DELAY, orc.GATE_WAIT_RHO, orc.GATE_WAIT_NO_ACTIVE,
                    orc.GATE_WAIT_MISSING, orc.GATE_WAIT_GRADIENT}


def test_admission_gate_metadata(torch_gpu, gs, orc):
    """Publication metadata: an admitted delayed set records the producer
    version; a second producer on a marked primitive waits; a refused gate
    leaves the metadata unchanged."""
    torch = torch_gpu
    n = 70001
    rng = np.random.default_rng(9)
    RB = np.flatnonzero(rng.random(n) < 0.5)
    CA = np.flatnonzero(rng.random(n) < 0.3)
    g = (rng.random(n) + 1.0).astype(np.float32)
    D = np.intersect1d(RB, CA)[:50]
    g[D] = 0.01
    skip = np.zeros(n, np.uint32)
    skip[rng.integers(0, n, 500)] = 3       # another producer's skipped updates elsewhere
    skip[D] = 0
    skip[D[:5]] = 7                         # this producer's own, skipped by another reader
    r, s1 = gate_on_gpu(torch, gs, n, RB, D, CA, g, 0.2, skip=skip, version=7)
    ref, s1_ref = orc.admission_gate(RB, D, CA, g, 0.2, skip=skip, producer_version=7)
    assert_gate_equal(r, ref, "first")
    assert ref.reason == orc.GATE_ADMIT
    np.testing.assert_array_equal(s1, s1_ref)
    r, s2 = gate_on_gpu(torch, gs, n, RB, D[10:20], CA, g, 0.2, skip=s1, version=9)
    ref, s2_ref = orc.admission_gate(RB, D[10:20], CA, g, 0.2, skip=s1, producer_version=9)
    assert_gate_equal(r, ref, "second")
    assert ref.reason == orc.GATE_WAIT_SECOND
    np.testing.assert_array_equal(s2, s2_ref)


def test_scopes_of_consecutive_room_views(torch_gpu, gs, orc):
    """Two consecutive views of the room workload (1M primitives, 1080p): read
    scope = projection-visible set, update scope = realized active set, the
    gradient evidence = the backward's per-primitive |dL/d(u,v)|."""
    torch = torch_gpu
    from paper_2607_19893_amd import scenes
    from paper_2607_19893_amd.pipeline import ViewTrainer
    w = scenes.workload("room")
    cams = w.cameras[:2]
    tr = ViewTrainer(w.scene, capacity=1, max_width=cams[0].width, max_height=cams[0].height, lr=w.lr)
    tr.ensure_capacity(cams)
    n = w.scene.n
    words = gs.scope_words(n)
    sc = {k: torch.zeros(words, dtype=torch.int32, device="cuda") for k in ("RA", "WA", "RB", "WB")}
    vis, act = {}, {}
    for k, cam in zip("AB", cams):
        tr.project(cam); tr.visible(); tr.bin_sort(); tr.raster_fwd(active=True)
        tr.loss_l1(target=torch.from_numpy(target_of(w, 0 if k == "A" else 1).reshape(-1)).cuda())
        gs.gs_scope_from_pred(gs.GS_PRED_U32_NONZERO, tr.tiles, n, 0, sc["R" + k])
        gs.gs_scope_from_pred(gs.GS_PRED_U8_NONZERO, tr.active, n, 0, sc["W" + k])
        torch.cuda.synchronize()
        V = int(host_u32(tr.counts[0:1])[0])
        vis[k] = host_u32(tr.vis_idx, V).copy()
        act[k] = np.flatnonzero(tr.active.cpu().numpy()).astype(np.uint32)
        if k == "A":
            tr.raster_bwd(grad2d=False)
            torch.cuda.synchronize()
            gA = tr.grad_norm.cpu().numpy().copy()
    _say("room views: |R_A| %d |W_A| %d |R_B| %d |W_B| %d" % (vis["A"].size, act["A"].size, vis["B"].size,
                                                                act["B"].size))
    waw = torch.zeros(words, dtype=torch.int32, device="cuda")
    raw = torch.zeros(words, dtype=torch.int32, device="cuda")
    war = torch.zeros(words, dtype=torch.int32, device="cuda")
    il = [torch.zeros(n, dtype=torch.int32, device="cuda") for _ in range(3)]
    counts = torch.zeros(4, dtype=torch.int32, device="cuda")
    ws = torch.zeros(gs.gs_workspace_bytes(gs.GS_WS_SCOPE, n), dtype=torch.uint8, device="cuda")
    gs.gs_scope_conflicts(sc["RA"], sc["WA"], sc["RB"], sc["WB"], n, waw, raw, war, il[0], il[1], il[2], counts, ws)
    ref = orc.scope_conflicts(vis["A"], act["A"], vis["B"], act["B"])
    c = host_u32(counts)
    assert list(c) == [r.size for r in ref] + [vis["B"].size]
    for l, r in zip(il, ref):
        np.testing.assert_array_equal(host_u32(l, r.size), r)
    _say("hazards: WAW %d RAW %d WAR %d" % tuple(r.size for r in ref))
    g_dev = torch.from_numpy(gA).cuda()
    res = torch.zeros(16, dtype=torch.int32, device="cuda")
    for tau in (0.2, 1.0):
        args = gs.make_gate_args(sc["WA"], g_dev, tau, evidence=sc["RA"])
        gs.gs_admission_gate(sc["RB"], raw, args, n, res, ws)
        torch.cuda.synchronize()
        r = gs.gate_result_from(res)
        ref_g, _ = orc.admission_gate(vis["B"], ref[1], act["A"], gA, tau, evidence=vis["A"])
        assert_gate_equal(r, ref_g, "tau %g" % tau)
        _say("gate tau %g: reason %d rho %.4f mean %.4g max %.4g" % (tau, ref_g.reason, ref_g.rho, ref_g.mean_g,
                                                                      ref_g.max_g))
