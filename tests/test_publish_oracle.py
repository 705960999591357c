"""Pins of the oracle's versioned two-slot publication (Section 4.3, Shadow
Graph steps 3-4, and the per-primitive publication metadata that lets a read
skip at most one unpublished update):
  * the ring's life cycle with hand-computed replica values;
  * refusals (wrong slot, out-of-order and repeated commits) leave everything
    unchanged;
  * rows whose published version is already newer are left alone;
  * a simulation of overlapped task units, driving the oracle's hazards,
    admission gate and commit from an independent record of which updates
    are still unpublished, checks that no read ever skips two of them.
"""
import numpy as np
import pytest


def ids(*a):
    return np.array(a, dtype=np.uint32)


def msg_for(o, idx, rows, version):
    rows = np.asarray(rows, np.float32).reshape(len(idx), 1) if len(idx) == 0 else \
        np.asarray(rows, np.float32).reshape(len(idx), -1)
    return o.delta_message(ids(*idx), [rows], version)


def check_ring_cycle(o):
    base = [np.zeros((6, 1), np.float32)]
    ver = np.zeros(6, np.uint32)
    ring = np.zeros(4, np.uint32)
    slots = [None, None]
    # version 1 in slot 1, version 2 in slot 0 (both staged before either commits)
    slots[1] = msg_for(o, [1, 3], [[0.5], [1.0]], 1)
    slots[0] = msg_for(o, [3, 4], [[2.0], [-1.0]], 2)
    g, ver1, _, ring1, f = o.publish_commit(ring, slots, 1, base, "add", ver)
    assert f == o.COMMIT_OK
    assert list(g[0][:, 0]) == [0.0, 0.5, 0.0, 1.0, 0.0, 0.0]
    assert list(ver1) == [0, 1, 0, 1, 0, 0] and list(ring1[:3]) == [1, 2, 0]
    g, ver2, _, ring2, f = o.publish_commit(ring1, slots, 2, g, "add", ver1)
    assert f == o.COMMIT_OK
    assert list(g[0][:, 0]) == [0.0, 0.5, 0.0, 3.0, -1.0, 0.0]
    assert list(ver2) == [0, 1, 0, 2, 2, 0] and list(ring2[:3]) == [2, 2, 0]
    # overwrite mode copies
    slots[1] = msg_for(o, [0], [[7.0]], 3)
    g3, _, _, _, f = o.publish_commit(ring2, slots, 3, g, "overwrite", ver2)
    assert f == o.COMMIT_OK and g3[0][0, 0] == 7.0


def check_refusals(o):
    base = [np.arange(4, dtype=np.float32).reshape(4, 1)]
    ver = np.zeros(4, np.uint32)
    ring = np.zeros(4, np.uint32)
    slots = [msg_for(o, [0], [[1.0]], 2), msg_for(o, [1], [[1.0]], 1)]
    # version 2 before version 1: out of order
    g, v, _, r, f = o.publish_commit(ring, slots, 2, base, "add", ver)
    assert f == o.COMMIT_ORDER and np.array_equal(g[0], base[0]) and np.array_equal(v, ver) and r[0] == 0
    # version 3 is not in its slot (slot 1 holds version 1)
    _, _, _, _, f = o.publish_commit(ring, slots, 3, base, "add", ver)
    assert f == o.COMMIT_MISMATCH
    # version 1 commits once; a second commit of it is out of order
    g, v, _, r, f = o.publish_commit(ring, slots, 1, base, "add", ver)
    assert f == o.COMMIT_OK
    g2, v2, _, r2, f = o.publish_commit(r, slots, 1, g, "add", v)
    assert f == o.COMMIT_ORDER and np.array_equal(g2[0], g[0])
    # an id beyond the replica, or other group widths: mismatch
    slots[0] = msg_for(o, [9], [[1.0]], 2)
    assert o.publish_commit(r, slots, 2, g, "add", v)[4] == o.COMMIT_MISMATCH
    slots[0] = o.delta_message(ids(0), [np.ones((1, 2), np.float32)], 2)
    assert o.publish_commit(r, slots, 2, g, "add", v)[4] == o.COMMIT_MISMATCH


def check_newer_rows_left(o):
    base = [np.zeros((4, 1), np.float32)]
    ver = ids(0, 5, 0, 0)                 # primitive 1 already carries a later publication
    ring = ids(2, 0, 0, 0)
    slots = [None, msg_for(o, [0, 1, 2], [[1.0], [1.0], [1.0]], 3)]
    g, v, _, r, f = o.publish_commit(ring, slots, 3, base, "add", ver)
    assert f == o.COMMIT_OK
    assert list(g[0][:, 0]) == [1.0, 0.0, 1.0, 0.0]
    assert list(v) == [3, 5, 3, 0] and list(r[:3]) == [3, 2, 1]


def check_skip_cleared(o):
    base = [np.zeros((5, 1), np.float32)]
    ver = np.zeros(5, np.uint32)
    skip = ids(0, 1, 1, 4, 1)             # readers skipped version 1 at 1, 2, 4 and version 4 at 3
    slots = [None, msg_for(o, [1, 2, 3], [[1.0]] * 3, 1)]
    _, _, s, _, f = o.publish_commit(np.zeros(4, np.uint32), slots, 1, base, "add", ver, skip=skip)
    assert f == o.COMMIT_OK
    # 1, 2: published now; 3 names another version; 4 is not in this message
    assert list(s) == [0, 0, 0, 4, 1]
    # once version 1 is published a new delayed producer may be admitted on primitive 1
    g = np.zeros(5, np.float32)
    r, _ = o.admission_gate(RB=ids(0, 1, 2, 3, 4), D=ids(1), CA=ids(1), g=g, tau=1.0, skip=s, producer_version=2)
    assert r.reason == o.GATE_ADMIT


def simulate(o, seed, n=48, units=40):
    """Overlapped task units over n primitives, one scalar each.  Unit j stages
    its update as version j; publication is in version order; before unit B
    observes state, every pending producer P is checked: WAW or WAR hazards
    make B wait for P's publication, RAW hazards go through the admission gate
    and, if refused, wait too.  Returns the largest number of unpublished
    updates any read skipped and the number of admitted delayed reads."""
    rng = np.random.default_rng(seed)
    state = [np.zeros((n, 1), np.float32)]
    ver = np.zeros(n, np.uint32)
    skip = np.zeros(n, np.uint32)
    ring = np.zeros(4, np.uint32)
    slots = [None, None]
    pending = {}                                   # version -> set of ids it updates (unpublished)
    scopes = {}
    worst, admitted = 0, 0
    allowed = set()                                # (version, id) pairs this reader was admitted to skip

    def commit_next():
        nonlocal state, ver, skip, ring
        v = int(ring[0]) + 1
        state, ver, skip, ring, f = o.publish_commit(ring, slots, v, state, "add", ver, skip=skip)
        assert f == o.COMMIT_OK
        del pending[v]

    for j in range(1, units + 1):
        # a ring of two slots: version j reuses the slot of version j - 2
        while pending and min(pending) <= j - 2:
            commit_next()
        R = np.flatnonzero(rng.random(n) < 0.3)
        W = rng.choice(R, size=min(R.size, int(rng.integers(1, 4))), replace=False) if R.size else R
        g = rng.random(n).astype(np.float32)
        allowed.clear()
        for P in sorted(pending):
            if P not in pending:
                continue
            RP, WP, CP, gP = scopes[P]
            waw, raw, war = o.scope_conflicts(RP, WP, R, W)
            if waw.size or war.size:
                while P in pending:
                    commit_next()
                continue
            r, skip_new = o.admission_gate(R, raw, CP, gP, float(rng.choice([0.2, 0.5, 1.0])), skip=skip,
                                           producer_version=P)
            if r.reason == o.GATE_ADMIT:
                skip = skip_new
                admitted += 1
                allowed.update((P, int(p)) for p in raw)
            elif r.reason != o.GATE_NO_DELAY:
                while P in pending:
                    commit_next()
        # B observes state: count the unpublished updates each read skips; every
        # one of them must have been admitted for this reader
        for p in R:
            skipped = [v for v, s in pending.items() if p in s]
            worst = max(worst, len(skipped))
            assert all((v, int(p)) in allowed for v in skipped), (j, int(p), skipped)
        # B executes and stages its update
        active = W[rng.random(W.size) < 0.8]
        scopes[j] = (R, W, active, g)
        slots[j & 1] = msg_for(o, list(W), rng.standard_normal((W.size, 1)), j)
        pending[j] = set(int(x) for x in W)
    return worst, admitted


def check_skip_at_most_one(o):
    total = 0
    for seed in range(30):
        worst, admitted = simulate(o, seed)
        assert worst <= 1, (seed, worst)
        total += admitted
    assert total > 20                                # the throughput-first path was taken


CHECKS = [check_ring_cycle, check_refusals, check_newer_rows_left, check_skip_cleared, check_skip_at_most_one]


@pytest.mark.parametrize("check", CHECKS, ids=lambda f: f.__name__)
def test_publication(orc, check):
    check(orc)


PUBLISH_MUTATIONS = {
    13: check_skip_cleared,       # commit leaves the skip markers of the published version
    14: check_newer_rows_left,    # commit applies rows whose published version is newer
}


@pytest.mark.parametrize("k", sorted(PUBLISH_MUTATIONS))
def test_publish_planted_mistake_is_caught(orc, k):
    orc.set_mutation(k)
    try:
        with pytest.raises(AssertionError):
            PUBLISH_MUTATIONS[k](orc)
    finally:
        orc.set_mutation(0)
