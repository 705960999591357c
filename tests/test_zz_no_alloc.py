"""The no-allocation visible-set entry point (gs_visible_set_noalloc) against
gs_visible_set, through the C ABI: two calls in a row on the same GPU, the
second with a smaller input, for each predicate kind.  Ids are compared bit for
bit, and both against the ascending non-zero positions computed on the host."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    return torch


@pytest.fixture(scope="module")
def gs():
    from paper_2607_19893_amd import gsmi
    return gsmi


def _pred(torch, gs, kind, n, rng, density):
    """A seeded predicate array of `kind` on the GPU, plus its set ids (host)."""
    on = rng.random(n) < density
    if kind == gs.GS_PRED_U32_NONZERO:
        vals = np.where(on, rng.integers(1, 1 << 20, n), 0).astype(np.uint32)
        dev = torch.from_numpy(vals.view(np.int32).copy() if n else np.zeros(4, np.int32)).cuda()
    elif kind == gs.GS_PRED_U8_NONZERO:
        vals = np.where(on, rng.integers(1, 256, n), 0).astype(np.uint8)
        dev = torch.from_numpy(vals.copy() if n else np.zeros(8, np.uint8)).cuda()
    else:
        words = np.zeros(max(1, gs.scope_words(n)), np.uint32)
        ids = np.flatnonzero(on)
        np.bitwise_or.at(words, ids >> 5, (np.uint32(1) << (ids & 31).astype(np.uint32)))
        dev = torch.from_numpy(words.view(np.int32).copy()).cuda()
    return dev, np.flatnonzero(on).astype(np.uint32)


def _run_both(torch, gs, kind, dev, n):
    out_a = torch.full((max(1, n),), -1, dtype=torch.int32, device="cuda")
    out_b = torch.full((max(1, n),), -1, dtype=torch.int32, device="cuda")
    cnt_a = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    cnt_b = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    ws = torch.empty(max(1, gs.gs_workspace_bytes(gs.GS_WS_VISIBLE_SET, n)), dtype=torch.uint8, device="cuda")
    gs.gs_visible_set(kind, dev, n, out_a, cnt_a, ws)
    gs.gs_visible_set_noalloc(kind, dev, n, out_b, cnt_b)
    torch.cuda.synchronize()
    ca = int(cnt_a.cpu().numpy().view(np.uint32)[0])
    cb = int(cnt_b.cpu().numpy().view(np.uint32)[0])
    return (out_a.cpu().numpy().view(np.uint32)[:ca], ca, out_b.cpu().numpy().view(np.uint32)[:cb], cb,
            out_b.cpu().numpy().view(np.uint32)[cb:])


# (first n, second n): the second call is smaller and reuses the buffer the first filled
SIZES = [(3_000_017, 70_001), (200_000, 2049), (4097, 0)]


@pytest.mark.parametrize("kind_name", ["u32", "u8", "bitmap"])
def test_noalloc_matches_workspace_entry_point(torch_gpu, gs, kind_name):
    torch = torch_gpu
    kind = {"u32": gs.GS_PRED_U32_NONZERO, "u8": gs.GS_PRED_U8_NONZERO, "bitmap": gs.GS_PRED_BITMAP}[kind_name]
    rng = np.random.default_rng(97)
    for first, second in SIZES:
        for n, density in ((first, 0.3), (second, 0.55)):
            _say("noalloc visible set: kind %s n %d density %.2f" % (kind_name, n, density))
            dev, ref = _pred(torch, gs, kind, n, rng, density)
            ids_a, ca, ids_b, cb, tail = _run_both(torch, gs, kind, dev, n)
            assert ca == cb == ref.size
            assert np.array_equal(ids_a, ref)
            assert np.array_equal(ids_b, ids_a)
            assert np.all(tail == 0xFFFFFFFF)          # nothing written past the count


def test_noalloc_refuses_oversize(torch_gpu, gs):
    torch = torch_gpu
    out = torch.zeros(4, dtype=torch.int32, device="cuda")
    cnt = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    with pytest.raises(gs.GsmiError):
        gs.gs_visible_set_noalloc(gs.GS_PRED_U32_NONZERO, out, gs.GS_NOALLOC_MAX_N + 1, out, cnt)
    torch.cuda.synchronize()
    assert int(cnt.cpu()[0]) == 7                      # nothing enqueued
