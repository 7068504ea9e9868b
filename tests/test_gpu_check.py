"""c3_check (signature, exact vote and localization in one call) against the
three separate calls it replaces and against the oracle, through the C ABI:
every record, status, bitmap word, majority index, list entry and count bit
for bit.  Covers the fused tail (R <= 32: a vote kernel that stages the
lists per segment and a one-workgroup kernel that places them, up to 8,192
chunks; a separate localization above; one workgroup for records, votes
and lists on plans of up to 256 chunks and 1,024 records), the separate
steps of larger groups, repeated calls on a staged plan, truncated lists
and graph replay."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from parity import compare_all_records

pytestmark = pytest.mark.gpu

c3 = pytest.importorskip("paper_2608_11034_amd.c3")
DEV = "cuda"
CODE = {torch.float32: workloads.F32, torch.bfloat16: workloads.BF16,
        torch.float16: workloads.F16, torch.uint8: workloads.RAW}


def _case(*a):
    print("CASE", *a, flush=True)


def _host(outs, out_cap=None, und_cap=None):
    rec, st, bm, mj, outl, und, cnt = outs
    torch.cuda.synchronize()
    c = cnt.cpu().numpy()
    oc = outl.shape[0] if out_cap is None else min(out_cap, outl.shape[0])
    uc = und.numel() if und_cap is None else min(und_cap, und.numel())
    return dict(records=c3.records_numpy(rec), status=st.cpu().numpy(),
                bitmap=bm.cpu().numpy().view(np.uint64), maj=mj.cpu().numpy(),
                outliers=outl[:min(int(c[0]), oc)].cpu().numpy(),
                undecided=und.cpu().numpy()[:min(int(c[1]), uc)], counts=c)


def _three_calls(reps, chunk, tile=0, out_cap=None, und_cap=None):
    plan = c3.SignaturePlan(reps, chunk, tile)
    rec = plan.new_records()
    plan.run(rec, plan.new_workspace())
    st, bm, mj = c3.consensus(rec, c3.EXACT)
    outl, und, cnt = c3.localize(st, bm, mj, rec, out_cap=out_cap, und_cap=und_cap)
    return _host((rec, st, bm, mj, outl, und, cnt), out_cap, und_cap)


def _check(reps, chunk, tile=0, out_cap=None, und_cap=None):
    plan = c3.SignaturePlan(reps, chunk, tile)
    outs = plan.new_check_outputs(out_cap, und_cap)
    ws = torch.empty(plan.check_workspace_size(), dtype=torch.uint8, device=DEV)
    plan.run_check(outs, ws, out_cap=out_cap, und_cap=und_cap)
    return _host(outs, out_cap, und_cap)


def _same(a, b):
    for f in a["records"].dtype.names:
        assert np.array_equal(a["records"][f], b["records"][f]), f
    for k in ("status", "bitmap", "maj", "undecided", "counts"):
        assert np.array_equal(a[k], b[k]), k
    assert a["outliers"].tobytes() == b["outliers"].tobytes()


def _vs_oracle(g, reps, chunk):
    metas = [(CODE[t.dtype], tuple(t.shape)) for t in reps[0]]
    ref = oracle.signature([[workloads.host_bytes(t) for t in rep] for rep in reps], metas, chunk)
    compare_all_records(g["records"], ref)
    ost, obm, omj = oracle.vote_exact(ref["sig"])
    assert np.array_equal(g["status"], ost) and np.array_equal(g["maj"], omj)
    assert np.array_equal(g["bitmap"].reshape(obm.shape), obm)
    loc = oracle.localize(ost, obm, omj, len(reps))
    assert g["counts"].tolist() == loc["counts"].tolist()
    o = g["outliers"].reshape(-1).view(c3.OUTLIER_DTYPE) if g["outliers"].size else \
        np.zeros(0, c3.OUTLIER_DTYPE)
    assert len(o) == len(loc["unit"])
    assert [int(x) for x in o["chunk"]] == loc["unit"].tolist()
    assert [int(x) for x in o["replica"]] == loc["replica"].tolist()
    assert g["undecided"].tolist() == loc["undecided"].tolist()


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_small_configs_equal_three_calls_and_oracle(k):
    _case("check small config", k)
    w = workloads.make(k, device=DEV, scale="small")
    g = _check(w.replicas, w.chunk_bytes)
    _same(g, _three_calls(w.replicas, w.chunk_bytes))
    _vs_oracle(g, w.replicas, w.chunk_bytes)
    assert g["counts"][0] + g["counts"][1] > 0


def _random_reps(seed, R, n_max=300_000, T_max=6, chunk=None):
    rng = np.random.default_rng(seed)
    chunk = chunk or int(1024 << rng.integers(0, 9))
    tile = int(1024 << rng.integers(0, int(np.log2(chunk // 1024)) + 1))
    gen = torch.Generator(device=DEV)
    gen.manual_seed(seed)
    dts = list(CODE)
    base = []
    for _ in range(int(rng.integers(1, T_max + 1))):
        dt = dts[int(rng.integers(0, 4))]
        n = int(rng.integers(0, n_max))
        base.append(torch.randint(0, 256, (n,), generator=gen, device=DEV, dtype=torch.uint8)
                    if dt == torch.uint8 else torch.randn(n, generator=gen, device=DEV).to(dt))
    reps = [[t.clone() for t in base] for _ in range(R)]
    for _ in range(max(3, R // 2)):                       # byte faults, some in shared chunks
        t = int(rng.integers(0, len(base)))
        if reps[0][t].numel():
            pos = int(rng.integers(0, reps[0][t].numel() * reps[0][t].element_size()))
            for r in rng.choice(R, size=int(rng.integers(1, max(2, R // 2 + 1))), replace=False):
                reps[int(r)][t].view(torch.uint8)[pos] ^= 0x5A
    return reps, chunk, tile


@pytest.mark.parametrize("seed,R", [(0, 2), (1, 3), (2, 4), (3, 5), (4, 8), (5, 13), (6, 16),
                                    (7, 17), (10, 24), (11, 32), (12, 33), (8, 40),
                                    (9, 130)])
def test_random_plans_equal_three_calls_and_oracle(seed, R):
    reps, chunk, tile = _random_reps(2000 + seed, R, n_max=200_000 if R < 40 else 40_000)
    _case("check random", seed, R, chunk, tile)
    g = _check(reps, chunk, tile)
    _same(g, _three_calls(reps, chunk, tile))
    _vs_oracle(g, reps, chunk)


def _small_reps(R, C, seed, two_tensors=False):
    """R replicas of C chunks of 4 KiB (the last one short), faults in about
    half of the chunks: a minority of replicas flipped (attributed), for
    even R also half against half (undecided), and one replica's NaN."""
    gen = torch.Generator(device=DEV)
    gen.manual_seed(seed)
    if two_tensors:
        c1 = C // 3
        base = [torch.randn(c1 * 2048 - 5, generator=gen, device=DEV).to(torch.bfloat16),
                torch.randn((C - c1) * 1024 - 7, generator=gen, device=DEV)]
    else:
        base = [torch.randn(C * 1024 - 7, generator=gen, device=DEV)]
    reps = [[t.clone() for t in base] for _ in range(R)]
    rng = np.random.default_rng(seed)
    for c in range(C):
        kind = int(rng.integers(0, 6))
        if c == 0:
            kind = 0                                    # the first chunk always has a fault
        if kind > 2:
            continue
        t = 0 if not two_tensors or c < C // 3 else 1
        c0 = c if t == 0 else c - C // 3
        nb = reps[0][t].numel() * reps[0][t].element_size()
        pos = min(c0 * 4096 + int(rng.integers(0, 4096)), nb - 1)
        if kind == 0 and R >= 3:                        # a minority flipped
            who = rng.choice(R, size=int(rng.integers(1, (R - 1) // 2 + 1)), replace=False)
        elif kind == 1 and R % 2 == 0:                  # half against half
            who = rng.choice(R, size=R // 2, replace=False)
        else:                                           # one replica's NaN
            who = [int(rng.integers(0, R))]
            if reps[0][t].dtype == torch.float32:
                pos -= pos % 4
                for r in who:
                    reps[int(r)][t].view(torch.int32)[pos // 4] = 0x7FC00001
                continue
        for r in who:
            reps[int(r)][t].view(torch.uint8)[pos] ^= 0x21
    return reps


# Plans of at most 256 chunks, 1,024 records and 64 replicas take the
# one-workgroup tail: records (from partials when chunks span several
# tiles), votes and lists in one launch after the streaming kernel.
@pytest.mark.parametrize("R,C,tile,caps,two", [
    (3, 256, 4096, None, False),        # the 1M fp32 shape: 768 records, one-tile chunks
    (2, 256, 1024, None, False),        # four partials per record combined in the workgroup
    (4, 256, 4096, (5, 2), False),      # truncated lists; half-against-half chunks undecided
    (8, 128, 2048, None, True),         # bf16 and fp32 tensors
    (16, 64, 4096, (0, 0), False),      # lists of capacity zero
    (32, 32, 4096, None, False),        # 1,024 records, the workgroup's limit
    (5, 1, 4096, None, False),          # one chunk
    (40, 25, 2048, None, False),        # above the 32-replica tail, partials combined
    (64, 16, 4096, (3, 1), False),      # 64 replicas: one bitmap word
])
def test_one_workgroup_tail_equals_three_calls_and_oracle(R, C, tile, caps, two):
    _case("check one-workgroup tail", R, C, tile, caps, two)
    reps = _small_reps(R, C, 100 + R + C, two)
    oc, uc = caps if caps else (None, None)
    g = _check(reps, 4096, tile, out_cap=oc, und_cap=uc)
    assert len(g["status"]) == C
    _same(g, _three_calls(reps, 4096, tile, out_cap=oc, und_cap=uc))
    if caps is None:
        _vs_oracle(g, reps, 4096)
        assert g["counts"][0] > 0 or R == 2           # two replicas never outvote one
    else:
        assert len(g["outliers"]) == min(oc, g["counts"][0])
        assert len(g["undecided"]) == min(uc, g["counts"][1])
    if R % 2 == 0 and C > 1:
        assert g["counts"][1] > 0


@pytest.mark.parametrize("n_chunks,R", [(8192, 8), (8193, 8), (40_000, 4), (9000, 16),
                                         (8192, 32), (8193, 20)])
def test_many_chunks_take_the_separate_localization(n_chunks, R):
    """Above 8,192 chunks the tail kernel votes and a separate localization
    lists; above 32,768 that localization is the three-pass one."""
    _case("check many chunks", n_chunks, R)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(n_chunks)
    base = torch.randint(0, 256, (n_chunks * 1024 - 100,), generator=gen, device=DEV,
                         dtype=torch.uint8)
    reps = [[base.clone()] for _ in range(R)]
    rng = np.random.default_rng(n_chunks)
    for pos in rng.integers(0, base.numel(), 50):
        reps[int(rng.integers(0, R))][0][int(pos)] ^= 1
    g = _check(reps, 1024)
    _same(g, _three_calls(reps, 1024))
    assert g["counts"][0] >= 40


def test_truncated_lists():
    w = workloads.make(3, device=DEV, scale="small")
    _case("check truncated")
    g = _check(w.replicas, w.chunk_bytes, out_cap=2, und_cap=0)
    _same(g, _three_calls(w.replicas, w.chunk_bytes, out_cap=2, und_cap=0))
    assert g["counts"][0] > 2 and len(g["outliers"]) == 2


def test_repeated_calls_on_a_staged_plan():
    """Five calls on one staged plan with the bytes changed between calls:
    every call must see the new bytes and leave nothing that changes the
    next."""
    _case("check repeated staged")
    w = workloads.make(3, device=DEV, scale="small")
    plan = c3.SignaturePlan(w.replicas, w.chunk_bytes)
    outs = plan.new_check_outputs()
    ws = torch.empty(plan.check_workspace_size(), dtype=torch.uint8, device=DEV)
    plan.run_check(outs, ws)
    for i in range(5):
        b = w.replicas[i % w.R][i % len(w.metas)].view(-1).view(torch.uint8)
        b[(i * 7919) % b.numel()] ^= 0x10
        plan.run_check(outs, ws, plan_staged=True)
        _same(_host(outs), _three_calls(w.replicas, w.chunk_bytes))


def test_graph_replay_equals_eager():
    _case("check graph")
    w = workloads.make(2, device=DEV, scale="small")
    plan = c3.SignaturePlan(w.replicas, w.chunk_bytes)
    outs = plan.new_check_outputs()
    ws = torch.empty(plan.check_workspace_size(), dtype=torch.uint8, device=DEV)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        plan.run_check(outs, ws, stream=s)
    s.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        plan.run_check(outs, ws, stream=s, plan_staged=True)
    for i in range(3):
        b = w.replicas[1][0].view(-1).view(torch.uint8)
        b[1000 * (i + 1)] ^= 0x04
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        _same(_host(outs), _three_calls(w.replicas, w.chunk_bytes))


def test_argument_errors():
    w = workloads.make(1, device=DEV, scale="small")
    plan = c3.SignaturePlan(w.replicas, w.chunk_bytes)
    outs = plan.new_check_outputs()
    ws = torch.empty(plan.check_workspace_size(), dtype=torch.uint8, device=DEV)
    with pytest.raises(c3.C3Error, match=r"\(-4\)"):
        plan.run_check(outs, ws[: plan.ws_bytes])              # room for the signature only
    one = c3.SignaturePlan([w.replicas[0]], w.chunk_bytes)
    with pytest.raises(c3.C3Error, match=r"\(-1\)"):
        one.run_check(one.new_check_outputs(), ws)             # a group of one
