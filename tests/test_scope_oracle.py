"""Pins of the oracle's primitive-scope hazards and throughput-first admission
(Section 4.3) against facts that do not come from the oracle itself:
  * scenarios read off the paper's wait rules (a read of something another
    unit updates waits for its publication, and so on), each a hand-derived
    expected result;
  * a worked example with hand-computed sets;
  * brute force over every primitive of tiny random scopes, classifying each
    id by who reads and who updates it;
  * identities the definitions imply (WAR(A,B) = RAW(B,A), WAW symmetric,
    equal read and update scopes give no RAW or WAR);
  * the admission tests at exactly representable boundaries.
"""
import itertools

import numpy as np
import pytest


def ids(*a):
    return np.array(a, dtype=np.uint32)


# ---------------------------------------------------------------------------
# hazard sets
# ---------------------------------------------------------------------------

def check_scenarios(o):
    E = ids()
    # B reads a primitive that A updates, without updating it: read-after-write
    waw, raw, war = o.scope_conflicts(RA=ids(7), WA=ids(7), RB=ids(7), WB=E)
    assert list(raw) == [7] and waw.size == 0 and war.size == 0
    # both update it: write-after-write only (RAW leaves out B's own updates)
    waw, raw, war = o.scope_conflicts(RA=ids(7), WA=ids(7), RB=ids(7), WB=ids(7))
    assert list(waw) == [7] and raw.size == 0 and war.size == 0
    # A only reads it, B updates it: write-after-read only
    waw, raw, war = o.scope_conflicts(RA=ids(7), WA=E, RB=ids(7), WB=ids(7))
    assert list(war) == [7] and waw.size == 0 and raw.size == 0
    # both only read it: no hazard
    waw, raw, war = o.scope_conflicts(RA=ids(7), WA=E, RB=ids(7), WB=E)
    assert waw.size == 0 and raw.size == 0 and war.size == 0
    # disjoint scopes: no hazard, B may proceed
    waw, raw, war = o.scope_conflicts(RA=ids(1, 2), WA=ids(1), RB=ids(3, 4), WB=ids(4))
    assert waw.size == 0 and raw.size == 0 and war.size == 0


def check_worked_example(o):
    # R+(A) = {0..5}, W+(A) = {1,2,3}, R+(B) = {2,...,7}, W+(B) = {3,5,6}
    #   WAW = {3,5,6} & {1,2,3}                 = {3}
    #   RAW = ({2,...,7} - {3,5,6}) & {1,2,3}   = {2,4,7} & {1,2,3} = {2}
    #   WAR = {3,5,6} & ({0..5} - {1,2,3})      = {3,5,6} & {0,4,5} = {5}
    waw, raw, war = o.scope_conflicts(RA=ids(0, 1, 2, 3, 4, 5), WA=ids(1, 2, 3), RB=ids(2, 3, 4, 5, 6, 7),
                                      WB=ids(3, 5, 6))
    assert list(waw) == [3] and list(raw) == [2] and list(war) == [5]


def _random_scope(rng, n, p):
    return np.flatnonzero(rng.random(n) < p).astype(np.uint32)


def check_brute_force(o):
    rng = np.random.default_rng(11)
    for trial in range(200):
        n = int(rng.integers(1, 24))
        RA, WA, RB, WB = (_random_scope(rng, n, rng.random()) for _ in range(4))
        waw, raw, war = o.scope_conflicts(RA, WA, RB, WB)
        for p in range(n):
            a_reads, a_writes = p in RA, p in WA
            b_reads, b_writes = p in RB, p in WB
            # who has to wait for what, per primitive
            assert (p in waw) == (a_writes and b_writes)
            assert (p in raw) == (a_writes and b_reads and not b_writes)
            assert (p in war) == (b_writes and a_reads and not a_writes)
        for s in (waw, raw, war):
            assert np.all(np.diff(s.astype(np.int64)) > 0)


def check_identities(o):
    rng = np.random.default_rng(12)
    for trial in range(100):
        n = 40
        RA, WA, RB, WB = (_random_scope(rng, n, 0.4) for _ in range(4))
        waw, raw, war = o.scope_conflicts(RA, WA, RB, WB)
        waw2, raw2, war2 = o.scope_conflicts(RB, WB, RA, WA)
        np.testing.assert_array_equal(war, raw2)          # WAR(A,B) = RAW(B,A)
        np.testing.assert_array_equal(waw, waw2)          # WAW is symmetric
        assert np.intersect1d(raw, WB).size == 0           # RAW leaves out B's updates
        assert np.intersect1d(raw, waw).size == 0
        # with R+ = W+ for both units only WAW remains
        w0, r0, x0 = o.scope_conflicts(WA, WA, WB, WB)
        assert r0.size == 0 and x0.size == 0
        np.testing.assert_array_equal(w0, np.intersect1d(WA, WB))


def test_scope_scenarios(orc):
    check_scenarios(orc)


def test_scope_worked_example(orc):
    check_worked_example(orc)


def test_scope_brute_force(orc):
    check_brute_force(orc)


def test_scope_identities(orc):
    check_identities(orc)


# ---------------------------------------------------------------------------
# throughput-first admission
# ---------------------------------------------------------------------------

def check_gate_no_delay(o):
    g = np.ones(16, np.float32)
    r, _ = o.admission_gate(RB=ids(1, 2, 3), D=ids(), CA=ids(1), g=g, tau=0.0)
    assert r.reason == o.GATE_NO_DELAY and r.admit == 1
    # an empty consumer read scope has no delayed read to admit
    r, _ = o.admission_gate(RB=ids(), D=ids(), CA=ids(), g=g, tau=0.2)
    assert r.reason == o.GATE_NO_DELAY and r.admit == 1 and r.rho == 0.0


def check_gate_rho(o):
    g = np.zeros(16, np.float32)
    RB = ids(0, 1, 2, 3, 4, 5, 6, 7)
    # rho = 2/8 = 0.25 <= tau = 0.25: the scope test passes (and g = 0 passes the gradient gate)
    r, _ = o.admission_gate(RB=RB, D=ids(1, 2), CA=ids(1, 2, 9), g=g, tau=0.25)
    assert r.reason == o.GATE_ADMIT and r.rho == 0.25
    # rho = 3/8 > 0.25: wait
    r, _ = o.admission_gate(RB=RB, D=ids(1, 2, 3), CA=ids(1, 2, 3), g=g, tau=0.25)
    assert r.reason == o.GATE_WAIT_RHO and r.admit == 0
    # tau = 0: any delayed read waits
    r, _ = o.admission_gate(RB=RB, D=ids(1), CA=ids(1), g=g, tau=0.0)
    assert r.reason == o.GATE_WAIT_RHO


def check_gate_evidence(o):
    g = np.zeros(16, np.float32)
    RB = ids(*range(10))
    r, _ = o.admission_gate(RB=RB, D=ids(1), CA=ids(), g=g, tau=0.5)
    assert r.reason == o.GATE_WAIT_NO_ACTIVE
    # primitive 2 is delayed but the producer reported nothing for it
    r, _ = o.admission_gate(RB=RB, D=ids(1, 2), CA=ids(1, 5), g=g, tau=0.5)
    assert r.reason == o.GATE_WAIT_MISSING and r.n_missing == 1
    # evidence may cover more than the active set
    r, _ = o.admission_gate(RB=RB, D=ids(1, 2), CA=ids(1, 5), g=g, tau=0.5, evidence=ids(1, 2, 5))
    assert r.reason == o.GATE_ADMIT


def check_gate_gradient(o):
    # active set {0..9} with ||g|| = 1..10: mean 5.5, tau = 0.5 -> threshold 2.75
    g = np.zeros(32, np.float32)
    g[:10] = np.arange(1, 11)
    g[20] = 2.5
    g[21] = 3.0
    RB = ids(*range(10, 30))
    CA = ids(*range(10))
    ev = ids(*range(10), 20, 21)
    r, _ = o.admission_gate(RB=RB, D=ids(20), CA=CA, g=g, tau=0.5, evidence=ev)
    assert r.reason == o.GATE_ADMIT and r.mean_g == 5.5 and r.threshold == 2.75 and r.max_g == 2.5
    r, _ = o.admission_gate(RB=RB, D=ids(20, 21), CA=CA, g=g, tau=0.5, evidence=ev)
    assert r.reason == o.GATE_WAIT_GRADIENT and r.max_g == 3.0
    # equality passes: mean of {1, 3} is 2, tau 0.5 -> threshold 1, delayed ||g|| = 1
    g2 = np.array([1.0, 3.0, 1.0, 0.0], np.float32)
    r, _ = o.admission_gate(RB=ids(2, 3), D=ids(2), CA=ids(0, 1), g=g2, tau=0.5, evidence=ids(0, 1, 2))
    assert r.reason == o.GATE_ADMIT and r.threshold == 1.0


def check_gate_skip(o):
    g = np.zeros(8, np.float32)
    RB = ids(*range(8))
    skip = np.zeros(8, np.uint32)
    # admitted: the delayed primitives now record the skipped producer version
    r, s1 = o.admission_gate(RB=RB, D=ids(2, 3), CA=ids(2, 3), g=g, tau=0.5, skip=skip, producer_version=7)
    assert r.reason == o.GATE_ADMIT
    assert list(s1) == [0, 0, 7, 7, 0, 0, 0, 0]
    # a second delayed producer on primitive 3 while version 7 is still unpublished: wait
    r, s2 = o.admission_gate(RB=RB, D=ids(3), CA=ids(3), g=g, tau=0.5, skip=s1, producer_version=8)
    assert r.reason == o.GATE_WAIT_SECOND and r.n_second == 1
    np.testing.assert_array_equal(s2, s1)
    # the same producer skipped by another reader is still one skipped update
    r, s3 = o.admission_gate(RB=RB, D=ids(3), CA=ids(3), g=g, tau=0.5, skip=s1, producer_version=7)
    assert r.reason == o.GATE_ADMIT
    np.testing.assert_array_equal(s3, s1)


def check_gate_precedence(o):
    g = np.full(8, 100.0, np.float32)
    g[0] = 1.0
    # both the scope test and the gradient test fail: the scope test is reported
    r, _ = o.admission_gate(RB=ids(1, 2), D=ids(1, 2), CA=ids(0), g=g, tau=0.5)
    assert r.reason == o.GATE_WAIT_RHO


GATE_CHECKS = [check_gate_no_delay, check_gate_rho, check_gate_evidence, check_gate_gradient, check_gate_skip,
               check_gate_precedence]


@pytest.mark.parametrize("check", GATE_CHECKS, ids=lambda f: f.__name__)
def test_gate(orc, check):
    check(orc)


# the pins above catch plausible mistakes planted in the oracle
SCOPE_MUTATIONS = {
    8: check_scenarios,          # RAW without leaving out B's own updates
    9: check_worked_example,     # WAR with A and B swapped
    10: check_gate_gradient,     # mean taken over the delayed set instead of C_A
    11: check_gate_rho,          # rho == tau treated as a failure
    12: check_gate_skip,         # second delayed producer not refused
}


@pytest.mark.parametrize("k", sorted(SCOPE_MUTATIONS))
def test_scope_planted_mistake_is_caught(orc, k):
    orc.set_mutation(k)
    try:
        with pytest.raises(AssertionError):
            SCOPE_MUTATIONS[k](orc)
    finally:
        orc.set_mutation(0)


def test_bitmap_layout_round_trip(orc):
    # bit i & 31 of word i >> 5: id 0 is the lowest bit of word 0, id 33 bit 1 of word 1
    w = orc.scope_bitmap([0, 33, 63, 64], 70)
    assert list(w) == [1, (1 << 1) | (1 << 31), 1]
    rng = np.random.default_rng(3)
    for n in (1, 31, 32, 33, 1000):
        s = np.flatnonzero(rng.random(n) < 0.3)
        np.testing.assert_array_equal(orc.scope_ids(orc.scope_bitmap(s, n), n), s)
