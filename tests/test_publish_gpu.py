"""GPU parity of the versioned two-slot publication (gs_publish_commit)
against the oracle, through the C ABI: versions staged with gs_delta_pack in
ring slot v & 1, committed in order into a replica with per-primitive
versions and skip markers; refused commits leave everything unchanged."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

COLS = [3, 3, 4, 1, 48]


@pytest.fixture(scope="module")
def env():
    import torch
    from paper_2607_19893_amd import gsmi
    assert torch.cuda.is_available(), "GPU parity tests need an MI355X"
    return torch, gsmi


def u32(t):
    return t.detach().cpu().numpy().view(np.uint32)


class Ring:
    def __init__(self, torch, gs, n, rng, background=False):
        self.torch, self.gs, self.n = torch, gs, n
        dev = torch.device("cuda")
        self.base = [rng.standard_normal((n, c)).astype(np.float32) for c in COLS]
        self.rep = [torch.from_numpy(a.copy()).to(dev) for a in self.base]
        nbytes = gs.gs_delta_msg_bytes(n, sum(COLS), len(COLS))
        self.slots = [torch.zeros((nbytes + 15) // 4, dtype=torch.int32, device=dev) for _ in range(2)]
        self.state = torch.zeros(8, dtype=torch.int32, device=dev)
        self.ring = gs.make_ring(self.slots, self.state, background=background)
        self.ver = torch.zeros(n, dtype=torch.int32, device=dev)
        self.skip = torch.zeros(n, dtype=torch.int32, device=dev)
        self.status = torch.zeros(4, dtype=torch.int32, device=dev)
        self.host_slots = [np.zeros(1, np.uint32), np.zeros(1, np.uint32)]

    def stage(self, orc, idx, rows, version):
        torch, gs = self.torch, self.gs
        src = [torch.from_numpy(np.ascontiguousarray(r)).cuda() for r in rows]
        full = [torch.zeros((self.n, c), device="cuda") for c in COLS]
        I = torch.from_numpy(idx.astype(np.int64)).cuda()
        for f, s in zip(full, src):
            if idx.size:
                f[I] = s
        idx_d = torch.from_numpy(idx.view(np.int32).copy() if idx.size else np.zeros(1, np.int32)).cuda()
        cnt = torch.tensor([idx.size], dtype=torch.int32, device="cuda")
        gs.gs_delta_pack(idx_d, cnt, self.n, gs.make_groups(full), len(COLS), version, self.slots[version & 1],
                         self.status)
        torch.cuda.synchronize()
        assert u32(self.status)[0] == 0
        self.host_slots[version & 1] = orc.delta_message(idx, rows, version)

    def commit(self, version, mode, groups=None, use_skip=True):
        gs = self.gs
        arr = gs.make_groups(groups if groups is not None else self.rep)
        gs.gs_publish_commit(self.ring, version, arr, len(COLS), self.n, self.n,
                             gs.GS_APPLY_ADD if mode == "add" else gs.GS_APPLY_OVERWRITE, self.ver,
                             self.skip if use_skip else None, self.status)
        self.torch.cuda.synchronize()


def check_equal(r, groups, ver, skip, state):
    for a, b in zip(r.rep, groups):
        np.testing.assert_array_equal(a.cpu().numpy().view(np.uint32), np.asarray(b, np.float32).view(np.uint32))
    np.testing.assert_array_equal(u32(r.ver), ver)
    np.testing.assert_array_equal(u32(r.skip), skip)
    np.testing.assert_array_equal(u32(r.state)[:3], np.asarray(state, np.uint32)[:3])


@pytest.mark.parametrize("n", [64, 70001])
@pytest.mark.parametrize("mode", ["add", "overwrite"])
@pytest.mark.parametrize("background", [False, True])
def test_publish_commit_in_order(n, mode, background, env, orc):
    """background: the narrow launch meant to run beside compute gives the same result."""
    torch, gs = env
    rng = np.random.default_rng(n + (mode == "add"))
    r = Ring(torch, gs, n, rng, background=background)
    groups = [a.copy() for a in r.base]
    ver = np.zeros(n, np.uint32)
    ver[rng.integers(0, n, max(1, n // 50))] = 100          # rows already carrying a later publication
    skip = np.zeros(n, np.uint32)
    skip[rng.integers(0, n, max(1, n // 10))] = rng.integers(1, 5, max(1, n // 10))
    r.ver.copy_(torch.from_numpy(ver.view(np.int32)))
    r.skip.copy_(torch.from_numpy(skip.view(np.int32)))
    state = np.zeros(4, np.uint32)
    slots = [None, None]
    for v in (1, 2, 3, 4):
        K = [n // 3, 0, n, n // 7][v - 1]
        idx = np.sort(rng.choice(n, K, replace=False)).astype(np.uint32)
        rows = [rng.standard_normal((K, c)).astype(np.float32) for c in COLS]
        r.stage(orc, idx, rows, v)
        slots[v & 1] = r.host_slots[v & 1]
        r.commit(v, mode)
        assert u32(r.status)[0] == 0
        groups, ver, skip, state, f = orc.publish_commit(state, slots, v, groups, mode, ver, skip=skip)
        assert f == orc.COMMIT_OK
        check_equal(r, groups, ver, skip, state)


def test_publish_commit_refusals(env, orc):
    torch, gs = env
    n = 5000
    rng = np.random.default_rng(7)
    r = Ring(torch, gs, n, rng)
    idx = np.sort(rng.choice(n, 900, replace=False)).astype(np.uint32)
    rows = [rng.standard_normal((900, c)).astype(np.float32) for c in COLS]
    r.stage(orc, idx, rows, 1)
    r.stage(orc, idx[:100], [a[:100] for a in rows], 2)
    snap = [t.clone() for t in r.rep] + [r.ver.clone(), r.skip.clone(), r.state.clone()]

    def unchanged():
        for a, b in zip([*r.rep, r.ver, r.skip, r.state], snap):
            assert torch.equal(a, b)

    # version 2 before version 1: out of order
    r.commit(2, "add")
    assert u32(r.status)[0] & gs.GS_DEV_MSG_ORDER
    unchanged()
    # version 3's slot holds version 1: mismatch
    r.status.zero_()
    r.commit(3, "add")
    assert u32(r.status)[0] & gs.GS_DEV_MSG_MISMATCH
    unchanged()
    # a replica with other group widths: mismatch
    r.status.zero_()
    wrong = [torch.zeros((n, c), device="cuda") for c in (3, 3, 4, 1, 45)]
    gs.gs_publish_commit(r.ring, 1, gs.make_groups(wrong), 5, n, n, gs.GS_APPLY_ADD, r.ver, r.skip, r.status)
    torch.cuda.synchronize()
    assert u32(r.status)[0] & gs.GS_DEV_MSG_MISMATCH
    assert all(float(t.abs().sum()) == 0.0 for t in wrong)
    unchanged()
    # a replica shorter than the message's ids: mismatch
    r.status.zero_()
    gs.gs_publish_commit(r.ring, 1, gs.make_groups(r.rep), 5, int(idx.max()), n, gs.GS_APPLY_ADD, r.ver, r.skip,
                         r.status)
    torch.cuda.synchronize()
    assert u32(r.status)[0] & gs.GS_DEV_MSG_MISMATCH
    unchanged()
    # version 1 commits; committing it again is out of order
    r.status.zero_()
    r.commit(1, "add")
    assert u32(r.status)[0] == 0 and u32(r.state)[0] == 1
    snap = [t.clone() for t in r.rep] + [r.ver.clone(), r.skip.clone(), r.state.clone()]
    r.commit(1, "add")
    assert u32(r.status)[0] & gs.GS_DEV_MSG_ORDER
    unchanged()
