"""GPU parity of the fused timing consensus (c3_timing_consensus): exact vote
on collective fingerprints, statistical vote on step times and temporal
confirmation, against the oracle's vote_exact, vote_statistical and confirm,
bit for bit, through the C ABI.

Inputs: seeded [T][G][R] fingerprints with ranks that diverge from a seeded
iteration on and occasional splits; lognormal step times with persistent and
intermittent stragglers, exact ties (so the IQR and range fallbacks of the
scale are reached) and non-finite values.  Sizes cover ragged workgroup
tiles (G around 64, T around the 32-iteration mask segments), R from 1 to 16
on the fused kernels and above 16 or W above 64 on the separate steps, and
the single-pass kernel's shapes (G of 4096 and more, ragged 16-group
workgroups, T up to its LDS limit).
"""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

c3 = pytest.importorskip("paper_2608_11034_amd.c3")
DEV = "cuda"


def _case(*a):
    print("CASE", *a, flush=True)


def _inputs(R, G, T, seed, f64=False):
    rng = np.random.default_rng(seed)
    base = rng.integers(-(2 ** 63), 2 ** 63 - 1, size=(T, G, 1), dtype=np.int64)
    fp = np.repeat(base, R, axis=2)
    for _ in range(max(1, R * G // 20)):                   # divergent ranks
        g, r, t0 = rng.integers(0, G), rng.integers(0, R), rng.integers(0, T)
        fp[t0:, g, r] ^= np.int64(rng.integers(1, 2 ** 62))
    for _ in range(max(1, T * G // 30)):                   # splits in single units
        t, g = rng.integers(0, T), rng.integers(0, G)
        k = int(rng.integers(1, R + 1))
        fp[t, g, :k] ^= np.int64(12345)
    tau = np.exp(rng.normal(0.0, 0.02, size=(T, G, R)))
    for _ in range(max(1, R * G // 25)):                   # persistent stragglers
        g, r = rng.integers(0, G), rng.integers(0, R)
        tau[:, g, r] *= 1.3
    mask = rng.random((T, G, R)) < 0.03                      # intermittent slowness
    tau[mask] *= 1.5
    ties = rng.random((T, G)) < 0.05                          # all equal: d falls back
    tau[ties] = 1.0
    half = rng.random((T, G)) < 0.05                          # two values only
    tau[half, : R // 2 + 1] = 0.5
    bad = rng.random((T, G, R)) < 0.01
    tau[bad] = rng.choice([np.nan, np.inf, -np.inf], size=int(bad.sum()))
    tau = tau.astype(np.float64 if f64 else np.float32)
    return fp, tau


def _oracle(fp, tau, W):
    T, G, R = fp.shape
    ost, obm, omj = oracle.vote_exact(fp.reshape(T * G, R).view(np.uint64), replica_axis=1)
    sst, sbm, smj = oracle.vote_statistical(tau.reshape(T * G, R), oracle.KAPPA_DEFAULT,
                                            replica_axis=1)
    ver = oracle.confirm(obm.reshape(T, G), sbm.reshape(T, G), R, W)
    return (ost, obm, omj), (sst, sbm, smj), ver


def _check(fp, tau, W, per_unit=True):
    T, G, R = fp.shape
    ver, fo, to = c3.timing_consensus(torch.from_numpy(fp).to(DEV), torch.from_numpy(tau).to(DEV),
                                      window=W, per_unit=per_unit)
    torch.cuda.synchronize()
    (ost, obm, omj), (sst, sbm, smj), ref = _oracle(fp, tau, W)
    if per_unit:
        assert np.array_equal(fo[0].cpu().numpy(), ost)
        assert np.array_equal(fo[1].cpu().numpy().view(np.uint64), obm)
        assert np.array_equal(fo[2].cpu().numpy(), omj)
        assert np.array_equal(to[0].cpu().numpy(), sst)
        assert np.array_equal(to[1].cpu().numpy().view(np.uint64), sbm)
        assert np.array_equal(to[2].cpu().numpy(), smj)
    else:
        assert fo is None and to is None
    v = c3.verdicts_numpy(ver)
    assert np.array_equal(v["flags"], ref["flags"])
    assert np.array_equal(v["first_divergent_iter"], ref["first_div"])
    assert np.array_equal(v["divergent_count"], ref["div_count"])
    assert np.array_equal(v["slow_count"], ref["slow_count"])
    assert np.array_equal(v["max_window_slow"], ref["max_window"])
    assert np.array_equal(v["first_straggler_window"], ref["first_window"])
    return v


CASES = [
    # R, G, T, W, f64
    (8, 64, 16, 16, False), (8, 65, 17, 16, False), (8, 130, 100, 16, True),
    (3, 63, 40, 5, False), (4, 1, 1, 16, False), (2, 7, 33, 3, False), (2, 70, 31, 1, True),
    (5, 64, 64, 64, False), (7, 66, 90, 64, True), (8, 20, 129, 63, False),
    (9, 64, 16, 16, False), (13, 33, 41, 16, True), (16, 64, 24, 8, False), (16, 3, 9, 64, False),
    (4, 66, 300, 1, False), (6, 9, 700, 2, True),   # several lanes per rank, short windows
    (4, 50, 37, 4, True), (16, 40, 30, 16, True), (8, 1, 70, 16, True),   # fp64 times, R = 4, 16
    (20, 40, 50, 16, False),                 # R > 16: separate steps
    (8, 50, 120, 80, False),                 # W > 64: separate steps
]


# Shapes of the single-pass kernel (with the per-unit results of either
# kind, both or neither): R a group bound (4, 8, 16), at least one
# 16-group workgroup per
# compute unit (G >= 4081 on 256 CUs), masks within the LDS budget (T <= 2048
# at R = 8).  Ragged G leaves the last workgroup 1-15 groups; ragged T leaves
# a partial 4-iteration step and a partial 32-iteration mask segment.
PASS_CASES = [
    (8, 4096, 40, 16, False), (8, 4100, 37, 16, False), (8, 4100, 129, 33, True),
    (4, 4100, 70, 5, False), (4, 4097, 33, 64, True), (16, 4100, 45, 16, False),
    (16, 4096, 20, 1, True), (8, 4096, 1, 16, False), (8, 4111, 2048, 16, False),
]


@pytest.mark.parametrize("R,G,T,W,f64", CASES)
def test_timing_consensus_matches_oracle(R, G, T, W, f64):
    _case("timing", R, G, T, W, f64)
    fp, tau = _inputs(R, G, T, seed=R * 1000 + G * 7 + T, f64=f64)
    _check(fp, tau, W)


@pytest.mark.parametrize("per_unit", [False, True])
@pytest.mark.parametrize("R,G,T,W,f64", PASS_CASES)
def test_timing_consensus_single_pass_matches_oracle(R, G, T, W, f64, per_unit):
    _case("timing single pass", R, G, T, W, f64, per_unit)
    fp, tau = _inputs(R, G, T, seed=R * 1000 + G * 7 + T, f64=f64)
    _check(fp, tau, W, per_unit=per_unit)


@pytest.mark.parametrize("R,G,T,W,f64", [
    (8, 4100, 37, 16, False),     # the single pass: ragged G and T
    (16, 4096, 20, 1, True),      # the single pass: fp64 times, W = 1
    (4, 4097, 33, 64, False),     # the single pass: a window over 32
    (8, 100, 40, 16, False),      # too few groups for the pass: the workspace path
])
@pytest.mark.parametrize("kind", ["fp", "time"])
def test_timing_consensus_per_unit_results_of_one_kind(kind, R, G, T, W, f64):
    """Per-unit results of one kind only: the single pass where its shape
    conditions hold, the workspace path otherwise; every per-unit result of
    that kind and every verdict field against the oracle."""
    import ctypes
    _case("timing one kind", kind, R, G, T, W, f64)
    fp, tau = _inputs(R, G, T, seed=77 + R + T, f64=f64)
    (ost, obm, omj), (sst, sbm, smj), ref = _oracle(fp, tau, W)
    dfp, dtau = torch.from_numpy(fp).to(DEV), torch.from_numpy(tau).to(DEV)
    outs = (torch.full((T * G,), 0xEE, dtype=torch.uint8, device=DEV),
            torch.full((T * G,), -5, dtype=torch.int64, device=DEV),
            torch.full((T * G,), -7, dtype=torch.int32, device=DEV))
    ver = torch.empty((R * G, 24), dtype=torch.uint8, device=DEV)
    ws = torch.empty(c3.timing_consensus_workspace_size(R, G, T, W), dtype=torch.uint8, device=DEV)
    p = lambda x: ctypes.c_void_p(x.data_ptr())
    null = ctypes.c_void_p(0)
    fo = tuple(p(x) for x in outs) if kind == "fp" else (null, null, null)
    to = tuple(p(x) for x in outs) if kind == "time" else (null, null, null)
    rc = c3.lib().c3_timing_consensus(p(dfp), p(dtau), c3.EV_F64 if f64 else c3.EV_F32, R, G, T,
                                      c3.KAPPA_DEFAULT, W, *fo, *to, p(ver), p(ws), ws.numel(), null)
    assert rc == 0
    torch.cuda.synchronize()
    st, bm, mj = (ost, obm, omj) if kind == "fp" else (sst, sbm, smj)
    assert np.array_equal(outs[0].cpu().numpy(), st)
    assert np.array_equal(outs[1].cpu().numpy().view(np.uint64), bm)
    assert np.array_equal(outs[2].cpu().numpy(), mj)
    v = c3.verdicts_numpy(ver)
    assert np.array_equal(v["flags"], ref["flags"])
    assert np.array_equal(v["first_divergent_iter"], ref["first_div"])
    assert np.array_equal(v["divergent_count"], ref["div_count"])
    assert np.array_equal(v["slow_count"], ref["slow_count"])
    assert np.array_equal(v["max_window_slow"], ref["max_window"])
    assert np.array_equal(v["first_straggler_window"], ref["first_window"])


@pytest.mark.parametrize("R,G,T,W", [(8, 100, 70, 16), (12, 70, 50, 16), (20, 10, 30, 16)])
def test_timing_consensus_without_per_unit_outputs(R, G, T, W):
    _case("timing verdicts only", R, G, T, W)
    fp, tau = _inputs(R, G, T, seed=R + G + T)
    _check(fp, tau, W, per_unit=False)


@pytest.mark.parametrize("G,per_unit", [(3, True), (4096, False)])
@pytest.mark.parametrize("W", [1, 2, 16])
@pytest.mark.parametrize("t0", [31, 63, 64, 127, 255])
def test_timing_consensus_pair_across_lane_boundary(W, t0, G, per_unit):
    # T = 300 splits into lanes of 64 iterations: slowness at t0 and t0 + 1
    # straddles a lane boundary when t0 + 1 is a multiple of 64.  G = 4096
    # without per-unit results takes the single-pass kernel, G = 3 the three
    # launches.
    _case("timing pair", W, t0, G, per_unit)
    R, T = 8, 300
    rng = np.random.default_rng(t0 * 10 + W)
    fp = np.repeat(rng.integers(-(2 ** 63), 2 ** 63 - 1, size=(T, G, 1), dtype=np.int64), R,
                   axis=2)
    tau = np.exp(rng.normal(0.0, 0.01, size=(T, G, R))).astype(np.float32)
    tau[t0:t0 + 2, 1, 5] = 4.0
    v = _check(fp, tau, W, per_unit=per_unit)
    rank = 5 * G + 1
    assert v["flags"][rank] & c3.RANK_CONSEC2
    assert v["slow_count"][rank] >= 2


def test_timing_consensus_argument_errors():
    _case("timing errors")
    fp = torch.zeros((4, 4, 8), dtype=torch.int64, device=DEV)
    tau = torch.ones((4, 4, 8), dtype=torch.float32, device=DEV)
    with pytest.raises(c3.C3Error):
        c3.timing_consensus(fp, tau, window=0)
    with pytest.raises(c3.C3Error):
        c3.timing_consensus(fp, tau, kappa=0.0)
    with pytest.raises(c3.C3Error):
        c3.timing_consensus(fp, tau.to(torch.float16))
    L = c3.lib()
    import ctypes
    ver = torch.empty((32, 24), dtype=torch.uint8, device=DEV)
    ws = torch.empty((c3.timing_consensus_workspace_size(8, 4, 4, 16),), dtype=torch.uint8,
                     device=DEV)
    st = torch.empty((16,), dtype=torch.uint8, device=DEV)
    null = ctypes.c_void_p(0)
    p = c3._ptr
    # one kind's outputs given only in part
    rc = L.c3_timing_consensus(p(fp), p(tau), c3.EV_F32, 8, 4, 4, c3.KAPPA_DEFAULT, 16, p(st),
                               null, null, null, null, null, p(ver), p(ws), ws.numel(), null)
    assert rc == -1
    rc = L.c3_timing_consensus(p(fp), p(tau), c3.EV_F32, 8, 4, 4, c3.KAPPA_DEFAULT, 16, null,
                               null, null, null, null, null, p(ver), p(ws), 16, null)
    assert rc == -4


def test_full_config5_fused_equals_oracle_and_ground_truth():
    import workloads
    _case("full config 5 fused")
    torch.cuda.empty_cache()
    w = workloads.make(5, device=DEV, scale="full")
    T, G, R = w.T, w.G, w.R
    ver, fo, to = c3.timing_consensus(w.fingerprints, w.times, window=16)
    torch.cuda.synchronize()
    fp = w.fingerprints.cpu().numpy()
    tau = w.times.cpu().numpy()
    (ost, obm, omj), (sst, sbm, smj), ref = _oracle(fp, tau, 16)
    assert np.array_equal(fo[0].cpu().numpy(), ost)
    assert np.array_equal(fo[1].cpu().numpy().view(np.uint64), obm)
    assert np.array_equal(to[1].cpu().numpy().view(np.uint64), sbm)
    assert np.array_equal(to[2].cpu().numpy(), smj)
    v = c3.verdicts_numpy(ver)
    for k, rk in (("flags", "flags"), ("first_divergent_iter", "first_div"),
                  ("max_window_slow", "max_window"), ("first_straggler_window", "first_window"),
                  ("slow_count", "slow_count"), ("divergent_count", "div_count")):
        assert np.array_equal(v[k], ref[rk]), k
    strag = set(np.nonzero(v["flags"] & c3.RANK_STRAGGLER)[0].tolist())
    proto = {int(r): int(v["first_divergent_iter"][r])
             for r in np.nonzero(v["flags"] & c3.RANK_PROTOCOL)[0]}
    assert strag == set(w.stragglers)
    assert proto == w.divergent
    # verdicts only: the same ranks
    ver2, _, _ = c3.timing_consensus(w.fingerprints, w.times, window=16, per_unit=False)
    assert torch.equal(ver2, ver)
