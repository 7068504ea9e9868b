"""c3_localize_noalloc through the C ABI against c3_localize: identical
lists and counts on two calls in a row (the second smaller, so the fixed
scratch array still holds the first call's segment counts), at sizes that
take the three-pass path whose counts live in that array, with one-word and
multi-word bitmaps and truncated lists."""
import ctypes

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

c3 = pytest.importorskip("paper_2608_11034_amd.c3")
DEV = "cuda"


def _inputs(U, R, seed):
    rng = np.random.default_rng(seed)
    ev = rng.integers(0, 2, size=(U, R)).astype(np.int64)
    ev[rng.random(U) < 0.8] = 0            # most units agree
    ev[rng.random(U) < 0.05, : R // 2] = 5  # some have no strict majority
    return c3.consensus(torch.from_numpy(ev).to(DEV), c3.EXACT)


def _alloc(U, R, cap):
    out = torch.full((max(cap, 1), 80), 0x5A, dtype=torch.uint8, device=DEV)
    und = torch.full((max(cap, 1),), -7, dtype=torch.int64, device=DEV)
    cnt = torch.full((3,), -7, dtype=torch.int64, device=DEV)
    return out, und, cnt


def _call_noalloc(st, bm, mj, R, U, cap, bufs):
    out, und, cnt = bufs
    L = c3.lib()
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return L.c3_localize_noalloc(p(st), p(bm), p(mj), None, R, U, p(out), cap, p(und), cap,
                                 p(cnt), s)


def _call_ws(st, bm, mj, R, U, cap, bufs):
    out, und, cnt = bufs
    L = c3.lib()
    ws = torch.empty(int(L.c3_localize_workspace_size(U)), dtype=torch.uint8, device=DEV)
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return L.c3_localize(p(st), p(bm), p(mj), None, R, U, p(out), cap, p(und), cap, p(cnt),
                         p(ws), ws.numel(), s), ws


@pytest.mark.parametrize("R", [8, 130])
def test_noalloc_equals_workspace_localize_on_two_calls(R):
    sizes = [(1_000_003, 7), (70_001, 8)] if R == 8 else [(300_001, 9), (40_000, 10)]
    for U, seed in sizes:
        print("CASE localize_noalloc", R, U, flush=True)
        st, bm, mj = _inputs(U, R, seed)
        for cap in (U * R, 1000):
            a, b = _alloc(U, R, cap), _alloc(U, R, cap)
            assert _call_noalloc(st, bm, mj, R, U, cap, a) == 0
            rc, ws = _call_ws(st, bm, mj, R, U, cap, b)
            assert rc == 0
            torch.cuda.synchronize()
            assert torch.equal(a[2], b[2]), (U, cap)
            n_o = min(int(a[2][0]), cap)
            n_u = min(int(a[2][1]), cap)
            assert n_o > 0 and n_u > 0
            assert torch.equal(a[0][:n_o], b[0][:n_o])
            assert torch.equal(a[1][:n_u], b[1][:n_u])
            assert (a[0][n_o:] == 0x5A).all() and (a[1][n_u:] == -7).all()


def test_noalloc_rejects_more_than_its_maximum():
    st = torch.zeros(8, dtype=torch.uint8, device=DEV)
    bm = torch.zeros(8, dtype=torch.int64, device=DEV)
    mj = torch.zeros(8, dtype=torch.int32, device=DEV)
    bufs = _alloc(8, 8, 8)
    assert _call_noalloc(st, bm, mj, 8, c3.LOCALIZE_NOALLOC_MAX_UNITS + 1, 8, bufs) == -1
    torch.cuda.synchronize()
    assert (bufs[2] == -7).all()
