"""Large peer groups through the C ABI against the oracle.

The paper's table of published configurations lists data-parallel peer
degrees up to 192 (Table 2).  Above 64 replicas a unit's outlier bitmap is
ceil(R / 64) words; c3_consensus decides one unit per wave (exact votes from
17 replicas, statistical ones from 33) and c3_localize walks every word.
Checked element by element: status, every bitmap word, majority index, and
the outlier and undecided lists (single-workgroup and multi-pass
localization, with and without truncation).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from parity import compare_all_records

pytestmark = pytest.mark.gpu

c3 = pytest.importorskip("paper_2608_11034_amd.c3")
DEV = "cuda"


def _case(*a):
    print("CASE", *a, flush=True)


def _labels(R, U, rng):
    """[U, R] labels mixing the vote's cases: all equal, a planted majority
    with replica 0 inside or outside it, a bare majority, two halves, many
    small classes, all values distinct (every candidate tried), and the
    upper ceil(R / 2) replicas equal with the others distinct (a majority for
    odd R, first held by the last candidate, replica floor(R / 2))."""
    ev = np.empty((U, R), np.int64)
    kinds = rng.integers(0, 8, size=U)
    for u in range(U):
        k = kinds[u]
        if k == 0:
            row = np.zeros(R, np.int64)
        elif k == 1:
            row = rng.integers(1, 4, size=R)
            row[rng.choice(R, size=int(rng.integers(R // 2 + 1, R + 1)), replace=False)] = 0
        elif k == 2:
            row = np.full(R, 5, np.int64)
            row[rng.choice(np.arange(1, R), size=R // 2 + 1, replace=False)] = 6
        elif k == 3:
            row = np.where(rng.permutation(R) < R // 2, 1, 2).astype(np.int64)
        elif k == 4:
            row = rng.integers(0, 6, size=R)
        elif k == 5:
            row = np.zeros(R, np.int64)
            row[rng.integers(0, R)] = 9
        elif k == 6:
            row = 100 + rng.permutation(R)
        else:
            row = 100 + np.arange(R)
            row[R // 2:] = 7
        ev[u] = row
    return ev


def _check_votes(st, bm, mj, ost, obm, omj, R, where):
    U = ost.shape[0]
    assert np.array_equal(st.cpu().numpy(), ost), where
    g = bm.cpu().numpy().view(np.uint64).reshape(U, c3.bitmap_words(R))
    assert np.array_equal(g, obm.reshape(U, c3.bitmap_words(R))), where
    assert np.array_equal(mj.cpu().numpy(), omj), where


@pytest.mark.parametrize("R", [17, 24, 31, 32, 33, 64, 65, 100, 127, 128, 129, 192, 255, 256])
def test_exact_consensus_wide_matches_oracle(R):
    """R = 17-32 takes the 32-slot thread-per-unit kernel (128-bit row loads
    where a unit-major row is a whole number of 16-byte words, R = 24 and
    32; strided loads otherwise and replica-major), every R above 32 the
    wave-per-unit kernel."""
    _case("exact wide", R)
    rng = np.random.default_rng(R)
    U = 3001                                   # ragged against 4 units per workgroup
    lab = _labels(R, U, rng)
    ev = lab * (2 ** 40 + 12345) - 7           # values differ in both halves of the word
    ost, obm, omj = oracle.vote_exact(ev.view(np.uint64), replica_axis=1)
    assert obm.shape == ((U,) if R <= 64 else (U, c3.bitmap_words(R)))
    # unit-major [U, R]
    st, bm, mj = c3.consensus(torch.from_numpy(ev).to(DEV), c3.EXACT)
    assert tuple(bm.shape) == ((U,) if R <= 64 else (U, c3.bitmap_words(R)))
    _check_votes(st, bm, mj, ost, obm, omj, R, "unit-major")
    # replica-major [R, U]
    evr = torch.from_numpy(np.ascontiguousarray(ev.T)).to(DEV)
    st, bm, mj = c3.consensus(evr, c3.EXACT, R=R, replica_stride=U * 8, unit_stride=8, n_units=U)
    _check_votes(st, bm, mj, ost, obm, omj, R, "replica-major")
    # 32-bit evidence
    ev32 = (lab * 1000003 + 11).astype(np.int32)
    ost, obm, omj = oracle.vote_exact(ev32.view(np.uint32), replica_axis=1)
    st, bm, mj = c3.consensus(torch.from_numpy(ev32).to(DEV), c3.EXACT)
    _check_votes(st, bm, mj, ost, obm, omj, R, "u32")
    torch.cuda.synchronize()


@pytest.mark.parametrize("R", [17, 20, 31, 32, 33, 48, 64, 65, 97, 128, 129, 192, 255, 256])
@pytest.mark.parametrize("dt", [np.float32, np.float64])
def test_statistical_consensus_wide_matches_oracle(R, dt):
    """R = 17-32 takes the 32-slot thread-per-unit kernel (padding slots
    past R, so the sort runs over the finite values and +inf), every R above
    32 the wave kernel: one sort of the finite values."""
    _case("statistical wide", R, dt)
    rng = np.random.default_rng(1000 + R)
    U = 1201
    tau = np.exp(rng.standard_normal((U, R)) * 0.02)
    tau[::5, 70 % R] *= 1.4                      # a slow replica in the second word
    tau[::7, R - 1] *= 0.6                       # a fast one in the last
    tau[::11, R // 3] = tau[::11, 0]             # ties
    tau[3::13, : R // 2 + 1] = 1.0               # majority equal: MAD 0, IQR path
    tau[6::17] = 1.0
    tau[6::17, R - 2] = 1.5                      # all equal but one: range path
    tau[8::19] = 2.0                             # all equal: Agree
    tau[9::23, 64 % R] = np.nan
    tau[10::29, : R // 2] = np.inf               # finite majority only for odd R
    tau[12::31, 1::2] = -np.inf
    tau[14::37] = np.round(tau[14::37] * 16) / 16  # few distinct values, long runs of ties
    tau[15::41] = rng.integers(-3, 4, size=R) * 0.25  # negatives and zeros
    tau[16::43, ::3] = -0.0                       # signed zeros among the zeros
    tau[18::47, : (R + 1) // 2] = 3.0             # half equal: MAD 0 (odd R), median between runs (even R)
    t = tau.astype(dt)
    st, bm, mj = c3.consensus(torch.from_numpy(t).to(DEV), c3.STATISTICAL)
    ost, obm, omj = oracle.vote_statistical(t, oracle.KAPPA_DEFAULT, replica_axis=1)
    _check_votes(st, bm, mj, ost, obm, omj, R, "statistical")
    for kappa in (0.5, 10.0):
        st, bm, mj = c3.consensus(torch.from_numpy(t).to(DEV), c3.STATISTICAL, kappa=kappa)
        ost, obm, omj = oracle.vote_statistical(t, kappa, replica_axis=1)
        _check_votes(st, bm, mj, ost, obm, omj, R, ("kappa", kappa))


@pytest.mark.parametrize("R,U", [(65, 40000), (130, 32769), (192, 32768), (192, 2049),
                                 (256, 1), (256, 3000)])
def test_localize_wide_matches_oracle(R, U):
    """U <= 32,768 takes the single-workgroup kernel, larger U the
    count / scan / emit passes."""
    _case("localize wide", R, U)
    rng = np.random.default_rng(R * 7 + U)
    ev = rng.integers(0, 2, size=(U, R)).astype(np.int64)
    ev[rng.random(U) < 0.6] = 0
    ev[::9, R - 3:] = 5                          # outliers in the last word
    st, bm, mj = c3.consensus(torch.from_numpy(ev).to(DEV), c3.EXACT)
    ost, obm, omj = oracle.vote_exact(ev.view(np.uint64), replica_axis=1)
    _check_votes(st, bm, mj, ost, obm, omj, R, "vote")
    for cap in (None, 7):
        outl, und, cnt = c3.localize(st, bm, mj, None, R=R, out_cap=cap, und_cap=cap)
        torch.cuda.synchronize()
        loc = oracle.localize(ost, obm, omj, R, out_cap=cap, und_cap=cap)
        assert cnt.cpu().tolist() == loc["counts"].tolist(), cap
        o = c3.outliers_numpy(outl, cnt)
        assert o["chunk"].tolist() == loc["unit"].tolist(), cap
        assert o["replica"].tolist() == loc["replica"].tolist(), cap
        assert o["majority_replica"].tolist() == loc["majority"].tolist(), cap
        n_u = min(int(cnt[1]), und.numel())
        assert und.cpu().numpy()[:n_u].tolist() == loc["undecided"].tolist(), cap


@pytest.mark.parametrize("R", [65, 130, 256])
def test_wide_group_sign_vote_localize(R):
    """R replicas signed on one GPU, voted and localized: records, votes and
    lists against the oracle, faults planted in different bitmap words."""
    _case("wide end to end", R)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(R)
    base = [torch.randn(3000, generator=gen, device=DEV).to(torch.bfloat16),
            torch.randn(777, generator=gen, device=DEV)]
    reps = [[t.clone() for t in base] for _ in range(R)]
    bad = sorted({1, 63, 64, R - 1, R // 2 + 3})
    for r in bad:
        reps[r][r % 2].view(torch.uint8)[(r * 37) % 1500] ^= 0x10
    w = workloads.ReplicaWorkload("wide", R, [(workloads.BF16, (3000,)), (workloads.F32, (777,))],
                                  2048, reps)
    plan = c3.SignaturePlan(w.replicas, w.chunk_bytes)
    rec = plan.new_records()
    plan.run(rec, plan.new_workspace())
    st, bm, mj = c3.consensus(rec, c3.EXACT)
    outl, und, cnt = c3.localize(st, bm, mj, rec)
    torch.cuda.synchronize()
    host = [[workloads.host_bytes(t) for t in rep] for rep in w.replicas]
    ref = oracle.signature(host, w.metas, w.chunk_bytes)
    compare_all_records(c3.records_numpy(rec), ref)
    ost, obm, omj = oracle.vote_exact(ref["sig"])
    _check_votes(st, bm, mj, ost, obm, omj, R, "records")
    o = c3.outliers_numpy(outl, cnt)
    assert sorted(set(o["replica"].tolist())) == bad
    loc = oracle.localize(ost, obm, omj, R)
    assert list(zip(o["chunk"].tolist(), o["replica"].tolist())) == \
        list(zip(loc["unit"].tolist(), loc["replica"].tolist()))
    recs = c3.records_numpy(rec)
    for e in o:
        for z, r in enumerate((e["replica"], e["majority_replica"])):
            assert e["sum"][z] == recs[r, e["chunk"]]["sum"]
    # votes on the byte-equality definition agree as well
    vst, vbm, vmj = oracle.vote_bytes(oracle.chunk_views(host, w.metas, w.chunk_bytes))
    assert np.array_equal(vst, ost) and np.array_equal(vbm, obm) and np.array_equal(vmj, omj)


def test_wide_bitmap_outputs_are_checked():
    _case("wide output checks")
    ev = torch.zeros((10, 130), dtype=torch.int64, device=DEV)
    small = (torch.empty(10, dtype=torch.uint8, device=DEV), torch.empty(10, dtype=torch.int64,
             device=DEV), torch.empty(10, dtype=torch.int32, device=DEV))
    with pytest.raises(c3.C3Error):
        c3.consensus(ev, c3.EXACT, out=small)      # one word per unit, three needed
    st, bm, mj = c3.consensus(ev, c3.EXACT)
    with pytest.raises(c3.C3Error):
        c3.localize(st, bm[:, 0].contiguous(), mj, None, R=130)
    with pytest.raises(c3.C3Error):
        c3.consensus(torch.zeros((4, 257), dtype=torch.int64, device=DEV), c3.EXACT)
    torch.cuda.synchronize()
