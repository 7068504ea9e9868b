"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Element-by-element at sizes the oracle finishes in seconds (several tiles,
ragged tails, every dtype, edge cases), and at the benchmark's full sizes in
the benchmark's launch configuration on sampled chunks plus properties that
hold at any size (signature equality <=> byte equality; the planted faults are
exactly the outliers).
"""
import ctypes
import math

import numpy as np
import pytest
import torch

import oracle
import workloads
from parity import compare_all_records

pytestmark = pytest.mark.gpu

c3mod = pytest.importorskip("paper_2608_11034_amd.c3")
c3 = c3mod
DEV = "cuda"


def _host_reps(w):
    return [[workloads.host_bytes(t) for t in rep] for rep in w.replicas]


def _chunk_bases(metas, chunk_bytes):
    return np.cumsum([0] + [oracle.num_chunks([m], chunk_bytes) for m in metas])


def _expected(w):
    bases = _chunk_bases(w.metas, w.chunk_bytes)
    out = set()
    for f in w.faults:
        for b in range(f.byte_offset, f.byte_offset + f.byte_len):
            out.add((f.replica, int(bases[f.tensor]) + b // w.chunk_bytes))
    und = {int(bases[f.tensor]) + f.byte_offset // w.chunk_bytes for f in w.split_faults}
    return out, und


def _gpu_pipeline(w, grid_blocks=0, tile_bytes=0):
    plan = c3.SignaturePlan(w.replicas, w.chunk_bytes, tile_bytes)
    rec = plan.new_records()
    ws = plan.new_workspace()
    plan.run(rec, ws, grid_blocks=grid_blocks)
    st, bm, mj = c3.consensus(rec, c3.EXACT)
    outl, und, cnt = c3.localize(st, bm, mj, rec)
    torch.cuda.synchronize()
    return dict(rec=rec, records=c3.records_numpy(rec), status=st.cpu().numpy(),
                bitmap=bm.cpu().numpy().view(np.uint64), maj=mj.cpu().numpy(),
                outliers=c3.outliers_numpy(outl, cnt),
                undecided=und.cpu().numpy()[:min(int(cnt[1]), und.numel())],
                counts=cnt.cpu().numpy())


def _print_case(*a):
    print("CASE", *a, flush=True)


# ---------------------------------------------------------------------------
# small configs, every record
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_small_config_records_and_lists_match_oracle(k):
    _print_case("small config", k)
    w = workloads.make(k, device=DEV, scale="small")
    g = _gpu_pipeline(w)
    reps = _host_reps(w)
    ref = oracle.signature(reps, w.metas, w.chunk_bytes)
    compare_all_records(g["records"], ref)
    st, bm, mj = oracle.vote_exact(ref["sig"])
    assert np.array_equal(g["status"], st)
    assert np.array_equal(g["bitmap"], bm)
    assert np.array_equal(g["maj"], mj)
    loc = oracle.localize(st, bm, mj, w.R)
    assert g["counts"].tolist() == loc["counts"].tolist()
    assert g["outliers"]["chunk"].tolist() == loc["unit"].tolist()
    assert g["outliers"]["replica"].tolist() == loc["replica"].tolist()
    assert g["outliers"]["majority_replica"].tolist() == loc["majority"].tolist()
    assert g["undecided"].tolist() == loc["undecided"].tolist()
    # summaries carried by each outlier are the records of both replicas
    for e in g["outliers"]:
        for z, r in enumerate((e["replica"], e["majority_replica"])):
            row = g["records"][r, e["chunk"]]
            assert e["nan_count"][z] == row["nan_count"] and e["sum"][z] == row["sum"]
            assert e["absmax"][z] == row["absmax"] and e["sumsq"][z] == row["sumsq"]
    want_out, want_und = _expected(w)
    assert set(zip(g["outliers"]["replica"].tolist(), g["outliers"]["chunk"].tolist())) == want_out
    assert set(g["undecided"].tolist()) == want_und


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_tensor_signatures_match_oracle(k):
    _print_case("tensor signatures", k)
    w = workloads.make(k, device=DEV, scale="small")
    rec = c3.signature(w.replicas, w.chunk_bytes)
    T = len(w.metas)
    ts = c3.tensor_signature(rec, T)
    st, bm, mj = c3.consensus(ts, c3.EXACT, replica_stride=T * 8, unit_stride=8, n_units=T, R=w.R)
    torch.cuda.synchronize()
    ref = oracle.signature(_host_reps(w), w.metas, w.chunk_bytes)
    want = oracle.tensor_signature(ref, T)
    assert np.array_equal(ts.cpu().numpy().view(np.uint64), want)
    ost, obm, omj = oracle.vote_bytes(_host_reps(w))
    assert np.array_equal(st.cpu().numpy(), ost) and np.array_equal(bm.cpu().numpy().view(np.uint64), obm)
    assert np.array_equal(mj.cpu().numpy(), omj)


def test_tensor_signatures_of_many_ragged_tensors():
    """300 tensors per replica of 0 to 12 KB (empty tensors included, each
    one chunk): every tensor's chunk range, which the kernel finds by a
    64-way search over the records' tensor ids, and so every per-tensor
    signature equals the oracle's; the one changed tensor is the only
    outlier."""
    _print_case("tensor signatures, 300 ragged tensors")
    rng = np.random.default_rng(7)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(7)
    base = [torch.randn(int(rng.choice([0, 1, 5, 255, 256, 257, 1000, 3000])), generator=gen,
                        device=DEV) for _ in range(300)]
    R, chunk = 3, 1024
    reps = [[t.clone() for t in base] for _ in range(R)]
    hit = next(i for i in range(17, 300) if base[i].numel() > 0)
    reps[1][hit].view(torch.uint8)[0] ^= 1
    rec = c3.signature(reps, chunk)
    ts = c3.tensor_signature(rec, len(base))
    torch.cuda.synchronize()
    metas = [(workloads.F32, tuple(t.shape)) for t in base]
    ref = oracle.signature([[workloads.host_bytes(t) for t in rep] for rep in reps], metas, chunk)
    want = oracle.tensor_signature(ref, len(base))
    got = ts.cpu().numpy().view(np.uint64)
    assert np.array_equal(got, want)
    diff = {(r, t) for r in range(R) for t in range(len(base)) if got[r, t] != got[0 if r else 2, t]}
    assert {t for _, t in diff} == {hit}


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_three_step_protocol_on_gpu(k):
    """Fault-injection protocol of the paper's evaluation: clean replicas give
    no outlier and no undecided chunk, the planted faults give exactly their
    (replica, chunk) pairs and split chunks, and removing them gives nothing
    again."""
    _print_case("three-step protocol", k)
    w = workloads.make(k, device=DEV, scale="small")
    faulty = [list(rep) for rep in w.replicas]
    faulted = {f.replica for f in w.faults} | {f.replica for f in w.split_faults}
    src = next(r for r in range(w.R) if r not in faulted)
    clean = [[t.clone() for t in w.replicas[src]] for _ in range(w.R)]
    want_out, want_und = _expected(w)
    for step, reps in (("clean", clean), ("fault", faulty), ("clean-again", clean)):
        w.replicas = reps
        g = _gpu_pipeline(w)
        got = set(zip(g["outliers"]["replica"].tolist(), g["outliers"]["chunk"].tolist()))
        assert got == (want_out if step == "fault" else set()), step
        assert set(g["undecided"].tolist()) == (want_und if step == "fault" else set()), step


# ---------------------------------------------------------------------------
# edge cases: ragged tails, empty and scalar tensors, special values, R bounds
# ---------------------------------------------------------------------------
def _special_tensor(dtype, n, gen):
    x = torch.randn(n, generator=gen, device=DEV)
    if dtype == torch.uint8:
        return torch.randint(0, 256, (n,), generator=gen, device=DEV, dtype=torch.uint8)
    t = x.to(dtype)
    iv = {torch.float32: torch.int32, torch.bfloat16: torch.int16, torch.float16: torch.int16}[dtype]
    v = t.view(iv)
    pats = {torch.float32: [0, -2 ** 31, 1, 0x007FFFFF, 0x7F800000, -8388608, 0x7FC00000,
                            0x7F800001, -1, 0x00400000],
            torch.bfloat16: [0, -32768, 1, 0x007F, 0x7F80, -128, 0x7FC0, 0x7F81, -1, 0x0040],
            torch.float16: [0, -32768, 1, 0x03FF, 0x7C00, -1024, 0x7E00, 0x7C01, -1, 0x0200]}[dtype]
    for i, p in enumerate(pats):
        if 7 * i < n:
            v[7 * i] = p
    return t


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16, torch.float16, torch.uint8])
@pytest.mark.parametrize("chunk_bytes", [1024, 3072, 8192])
def test_edge_shapes_every_record(dtype, chunk_bytes):
    _print_case("edge shapes", dtype, chunk_bytes)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(chunk_bytes)
    sizes = [0, 1, 3, 7, 8, 9, 255, 256, 257, 511, 512, 513, 4097, 20000]
    base = [_special_tensor(dtype, n, gen) for n in sizes]
    base.append(_special_tensor(dtype, 1, gen).reshape(()))        # scalar
    base.append(_special_tensor(dtype, 96, gen).reshape(4, 3, 8))  # 3-D
    R = 3
    reps = [[t.clone() for t in base] for _ in range(R)]
    # a fault in the last (ragged) segment of one tensor and in the middle of another
    reps[1][8].view(torch.uint8)[-1] ^= 1
    reps[2][13].view(torch.uint8)[5000] ^= 0x80
    plan = c3.SignaturePlan(reps, chunk_bytes)
    rec = plan.new_records()
    plan.run(rec, plan.new_workspace())
    torch.cuda.synchronize()
    metas = [(workloads.F32 if dtype == torch.float32 else workloads.BF16 if dtype == torch.bfloat16
              else workloads.F16 if dtype == torch.float16 else workloads.RAW, tuple(t.shape))
             for t in base]
    ref = oracle.signature([[workloads.host_bytes(t) for t in rep] for rep in reps], metas, chunk_bytes)
    compare_all_records(c3.records_numpy(rec), ref)


def test_largest_tile_and_long_lanes():
    """The largest tile the ABI takes (16 MiB): each lane folds 64 KiB in one
    fp64 run and a wave walks 4,096 blocks; 64 MiB chunks, ragged tensors,
    one fault in the last block of a tile."""
    _print_case("largest tile")
    gen = torch.Generator(device=DEV)
    gen.manual_seed(16)
    base = [torch.randn(20 * (1 << 20) + 12345, generator=gen, device=DEV).to(torch.bfloat16),
            torch.randn(3 * (1 << 20) + 7, generator=gen, device=DEV) * 1e3]
    reps = [[t.clone() for t in base] for _ in range(3)]
    reps[1][0].view(torch.uint8)[(16 << 20) - 3] ^= 0x40
    plan = c3.SignaturePlan(reps, 64 << 20, 16 << 20)
    rec = plan.new_records()
    plan.run(rec, plan.new_workspace())
    torch.cuda.synchronize()
    metas = [(workloads.BF16, tuple(base[0].shape)), (workloads.F32, tuple(base[1].shape))]
    ref = oracle.signature([[workloads.host_bytes(t) for t in rep] for rep in reps], metas, 64 << 20)
    compare_all_records(c3.records_numpy(rec), ref)
    assert (ref["sig"][1] != ref["sig"][0]).sum() == 1


@pytest.mark.parametrize("seed", range(8))
def test_random_shapes_chunks_and_tiles(seed):
    """Seeded random tensor counts, lengths and types, chunk sizes and tile
    sizes: every record against the oracle.  Covers tiles whose blocks leave
    a wave a partial batch, ragged tensor ends and multi-tile chunks in
    combinations the fixed cases do not."""
    rng = np.random.default_rng(1000 + seed)
    chunk = int(1024 << rng.integers(0, 9))                # 1 KiB .. 256 KiB
    tile = int(1024 << rng.integers(0, int(np.log2(chunk // 1024)) + 1))
    dts = [torch.float32, torch.bfloat16, torch.float16, torch.uint8]
    T = int(rng.integers(1, 7))
    gen = torch.Generator(device=DEV)
    gen.manual_seed(seed)
    base = []
    for _ in range(T):
        dt = dts[int(rng.integers(0, 4))]
        n = int(rng.integers(0, 300_000))
        base.append(_special_tensor(dt, n, gen) if rng.random() < 0.3 else
                    (torch.randint(0, 256, (n,), generator=gen, device=DEV, dtype=torch.uint8)
                     if dt == torch.uint8 else torch.randn(n, generator=gen, device=DEV).to(dt)))
    R = int(rng.integers(2, 6))
    reps = [[t.clone() for t in base] for _ in range(R)]
    for _ in range(3):                                     # a few byte faults
        t = int(rng.integers(0, T))
        if reps[0][t].numel():
            r = int(rng.integers(0, R))
            b = reps[r][t].view(torch.uint8)
            b[int(rng.integers(0, b.numel()))] ^= int(rng.integers(1, 256))
    _print_case("random shapes", seed, "chunk", chunk, "tile", tile, "T", T, "R", R,
                [(str(t.dtype), t.numel()) for t in base])
    plan = c3.SignaturePlan(reps, chunk, tile)
    rec = plan.new_records()
    plan.run(rec, plan.new_workspace())
    torch.cuda.synchronize()
    code = {torch.float32: workloads.F32, torch.bfloat16: workloads.BF16,
            torch.float16: workloads.F16, torch.uint8: workloads.RAW}
    metas = [(code[t.dtype], tuple(t.shape)) for t in base]
    ref = oracle.signature([[workloads.host_bytes(t) for t in rep] for rep in reps], metas, chunk)
    compare_all_records(c3.records_numpy(rec), ref)


@pytest.mark.parametrize("chunk", [256 << 10, 1 << 20])
def test_xcd_tile_map_every_record(chunk):
    """Launches of at least 2,048 tiles of 256 KiB take their tiles through
    the XCD map (uneven rounds of 256 tiles, a proportional last round,
    workgroups without a tile).  Two ragged tensors of two dtypes over three
    replicas give launches of 5,283 fp32 and 2,163 bf16 tiles, both with a
    partial last round: every record against the oracle and against the
    same launches in plain order (an explicit grid), with faults in the
    first and the last chunk."""
    _print_case("xcd tile map", chunk)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(chunk)
    base = [torch.randn(110 * (1 << 20) + 4099, generator=gen, device=DEV) * 1e-2,
            torch.randn(90 * (1 << 20) + 77, generator=gen, device=DEV).to(torch.bfloat16)]
    reps = [[t.clone() for t in base] for _ in range(3)]
    reps[2][0].view(torch.uint8)[11] ^= 0x10
    reps[1][1].view(torch.uint8)[-1] ^= 0x01
    plan = c3.SignaturePlan(reps, chunk, 256 << 10)
    rec = plan.new_records()
    ws = plan.new_workspace()
    plan.run(rec, ws)
    rec_plain = plan.new_records()
    plan.run(rec_plain, ws, grid_blocks=997)
    torch.cuda.synchronize()
    g = c3.records_numpy(rec)
    assert g.tobytes() == c3.records_numpy(rec_plain).tobytes()
    metas = [(workloads.F32, tuple(base[0].shape)), (workloads.BF16, tuple(base[1].shape))]
    ref = oracle.signature([[workloads.host_bytes(t) for t in rep] for rep in reps], metas, chunk)
    compare_all_records(g, ref)
    diff = np.argwhere(ref["sig"] != ref["sig"][0:1])
    assert sorted(map(tuple, diff.tolist())) == [(1, int(ref["sig"].shape[1]) - 1), (2, 0)]


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16, torch.float16])
def test_absmax_finite_extremes_every_record(dtype):
    """Chunks without NaN or Inf (the kernel's unclassified path) whose largest
    magnitude is a signed zero, a subnormal, the largest finite value or a
    negative number, at random positions: absmax must be the exact magnitude."""
    _print_case("absmax finite extremes", dtype)
    iv, pos_max, sub_max = {torch.float32: (torch.int32, 0x7F7FFFFF, 0x007FFFFF),
                            torch.bfloat16: (torch.int16, 0x7F7F, 0x007F),
                            torch.float16: (torch.int16, 0x7BFF, 0x03FF)}[dtype]
    sign = -(2 ** 31) if dtype == torch.float32 else -(2 ** 15)
    chunk = 4096
    per = chunk // (4 if dtype == torch.float32 else 2)
    gen = torch.Generator(device="cpu")
    gen.manual_seed(17)
    pieces = []
    for kind in range(6):
        if kind == 0:    # zeros, some negative
            bits = torch.where(torch.rand(per, generator=gen) < 0.5, 0, sign)
        elif kind == 1:  # subnormals only, mixed signs
            bits = torch.randint(1, sub_max + 1, (per,), generator=gen)
            bits = torch.where(torch.rand(per, generator=gen) < 0.5, bits, bits + sign)
        elif kind == 2:  # subnormals and zeros, the largest one negative
            bits = torch.randint(0, sub_max // 2, (per,), generator=gen)
            bits[int(torch.randint(0, per, (1,), generator=gen))] = sub_max + sign
        elif kind == 3:  # the largest finite value, positive, once
            bits = torch.randint(0, pos_max // 2, (per,), generator=gen)
            bits[int(torch.randint(0, per, (1,), generator=gen))] = pos_max
        elif kind == 4:  # the largest finite value, negative, several times
            bits = torch.randint(0, pos_max, (per,), generator=gen)
            bits[torch.randint(0, per, (5,), generator=gen)] = pos_max + sign
        else:            # all values negative normals
            bits = torch.randint(0x00800000 if dtype == torch.float32 else 0x0080 if dtype ==
                                 torch.bfloat16 else 0x0400, pos_max, (per,), generator=gen) + sign
        pieces.append(bits)
    host = torch.cat(pieces).to(iv).view(dtype)
    t = host.to(DEV)
    assert not torch.isnan(host.float()).any() and not torch.isinf(host.float()).any()
    reps = [[t.clone()] for _ in range(3)]
    reps[2][0].view(torch.uint8)[3 * chunk + 1] ^= 0x01   # one differing chunk
    plan = c3.SignaturePlan(reps, chunk)
    rec = plan.new_records()
    plan.run(rec, plan.new_workspace())
    torch.cuda.synchronize()
    meta = workloads.F32 if dtype == torch.float32 else workloads.BF16 if dtype == torch.bfloat16 \
        else workloads.F16
    ref = oracle.signature([[workloads.host_bytes(r[0])] for r in reps], [(meta, tuple(t.shape))], chunk)
    compare_all_records(c3.records_numpy(rec), ref)
    assert (ref["absmax"][0] > 0).sum() == 5        # the zero chunk's absmax is +0


@pytest.mark.parametrize("k", [2, 3, 4])
def test_sharded_protocol_emulated(k):
    """The protocol with one replica per GPU, on one GPU: every replica is
    signed on its own (R = 1, what each rank does), the record tables are
    stacked (what the AllGather of Algorithm 1 delivers), and consensus and
    localize on the stacked table give exactly the joint call's bits."""
    _print_case("sharded protocol", k)
    w = workloads.make(k, device=DEV, scale="small")
    joint = _gpu_pipeline(w)
    parts = [c3.signature([rep], w.chunk_bytes) for rep in w.replicas]
    stacked = torch.cat(parts, dim=0)
    assert stacked.shape == joint["rec"].shape
    st, bm, mj = c3.consensus(stacked, c3.EXACT)
    outl, und, cnt = c3.localize(st, bm, mj, stacked)
    torch.cuda.synchronize()
    assert stacked.cpu().numpy().tobytes() == joint["rec"].cpu().numpy().tobytes()
    assert np.array_equal(st.cpu().numpy(), joint["status"])
    assert np.array_equal(bm.cpu().numpy().view(np.uint64), joint["bitmap"])
    assert np.array_equal(mj.cpu().numpy(), joint["maj"])
    assert cnt.cpu().numpy().tolist() == joint["counts"].tolist()
    o = c3.outliers_numpy(outl, cnt)
    assert o.tobytes() == joint["outliers"].tobytes()


@pytest.mark.parametrize("R", [2, 5, 64])
def test_replica_count_bounds(R):
    _print_case("replica count", R)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(R)
    base = [torch.randn(3000, generator=gen, device=DEV).to(torch.bfloat16),
            torch.randn(777, generator=gen, device=DEV)]
    reps = [[t.clone() for t in base] for _ in range(R)]
    for r in range(1, R, 3):
        reps[r][r % 2].view(torch.uint8)[r * 7 % 1000] ^= 4
    w = workloads.ReplicaWorkload("rbounds", R, [(workloads.BF16, (3000,)), (workloads.F32, (777,))],
                                  2048, reps)
    g = _gpu_pipeline(w)
    ref = oracle.signature(_host_reps(w), w.metas, w.chunk_bytes)
    compare_all_records(g["records"], ref)
    st, bm, mj = oracle.vote_exact(ref["sig"])
    assert np.array_equal(g["status"], st) and np.array_equal(g["bitmap"], bm)
    assert np.array_equal(g["maj"], mj)


def test_argument_errors():
    _print_case("argument errors")
    x = torch.randn(4096, device=DEV)
    with pytest.raises(c3.C3Error, match="at least one replica"):
        c3.signature([], 1024)                                    # handled in Python
    L = c3.lib()
    metas = c3.make_metas([x])
    rec = torch.empty(16 * 64, dtype=torch.uint8, device=DEV)
    ws = torch.empty(1 << 20, dtype=torch.uint8, device=DEV)
    p1 = (ctypes.c_void_p * 1)(x.data_ptr())
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert L.c3_signature(p1, metas, 1, 0, 1024, ctypes.c_void_p(rec.data_ptr()),
                          ctypes.c_void_p(ws.data_ptr()), ws.numel(), s) == -1    # R = 0
    p2 = (ctypes.c_void_p * 2)(x.data_ptr(), x.data_ptr())
    assert L.c3_signature(p2, metas, 1, 2, 1000, ctypes.c_void_p(rec.data_ptr()),
                          ctypes.c_void_p(ws.data_ptr()), ws.numel(), s) == -1    # chunk
    p3 = (ctypes.c_void_p * 2)(x.data_ptr(), x.data_ptr() + 4)
    assert L.c3_signature(p3, metas, 1, 2, 1024, ctypes.c_void_p(rec.data_ptr()),
                          ctypes.c_void_p(ws.data_ptr()), ws.numel(), s) == -2    # alignment
    assert L.c3_signature(p2, metas, 1, 2, 1024, ctypes.c_void_p(rec.data_ptr()),
                          ctypes.c_void_p(ws.data_ptr()), 16, s) == -4            # workspace
    assert L.c3_signature(p2, metas, 1, 257, 1024, ctypes.c_void_p(rec.data_ptr()),
                          ctypes.c_void_p(ws.data_ptr()), ws.numel(), s) == -1    # R > 256
    torch.cuda.synchronize()


def test_reused_plan_sees_new_data():
    _print_case("reused plan")
    w = workloads.make(1, device=DEV, scale="small")
    plan = c3.SignaturePlan(w.replicas, w.chunk_bytes)
    rec = plan.new_records()
    ws = plan.new_workspace()
    plan.run(rec, ws)
    first = c3.records_numpy(rec)
    w.replicas[0][0].view(torch.uint8)[100] ^= 0x10     # same pointers, new bytes
    plan.run(rec, ws, plan_staged=True)
    torch.cuda.synchronize()
    second = c3.records_numpy(rec)
    ref = oracle.signature(_host_reps(w), w.metas, w.chunk_bytes)
    compare_all_records(second, ref)
    assert second["sig"][0, 0] != first["sig"][0, 0]


def test_plan_larger_than_a_staging_slot():
    _print_case("large plan")
    R, T = 64, 600
    gen = torch.Generator(device=DEV)
    gen.manual_seed(600)
    base = torch.randn(T * 16, generator=gen, device=DEV)
    bufs = [base.clone() for _ in range(R)]
    bufs[37][16 * 599 + 3] = float("nan")
    reps = [[b[16 * t: 16 * t + 16] for t in range(T)] for b in bufs]
    w = workloads.ReplicaWorkload("many_tensors", R, [(workloads.F32, (16,))] * T, 1024, reps)
    g = _gpu_pipeline(w)
    ref = oracle.signature(_host_reps(w), w.metas, w.chunk_bytes)
    compare_all_records(g["records"], ref)
    assert g["outliers"]["replica"].tolist() == [37] and g["outliers"]["chunk"].tolist() == [599]


def test_grid_size_and_tile_size_invariance():
    _print_case("grid and tile invariance")
    w = workloads.make(4, device=DEV, scale="small")
    base = _gpu_pipeline(w)["records"]
    for grid in (1, 3, 64, 1000):
        g = _gpu_pipeline(w, grid_blocks=grid)["records"]
        assert g.tobytes() == base.tobytes(), grid
    ref = oracle.signature(_host_reps(w), w.metas, w.chunk_bytes)
    for tile in (1024, 16384, 1 << 20):
        g = _gpu_pipeline(w, tile_bytes=tile)["records"]
        for f in ("sig", "n_elems", "nan_count", "inf_count", "absmax", "tensor", "chunk_in_tensor"):
            assert np.array_equal(g[f], base[f]), (tile, f)
        compare_all_records(g, ref)


# ---------------------------------------------------------------------------
# consensus, localize and confirm on synthetic evidence
# ---------------------------------------------------------------------------
def test_singleton_group_vote_is_an_error():
    """Sec. 4: one replica provides no comparison.  Through the C ABI on the
    GPU, votes, localization, confirmation and the timing path return
    C3_E_INVAL for R = 1 and write nothing; signing one replica is valid."""
    _print_case("singleton group")
    ev = torch.arange(10, dtype=torch.int64, device=DEV).reshape(10, 1)
    st = torch.full((10,), 0xAB, dtype=torch.uint8, device=DEV)
    bm = torch.zeros(10, dtype=torch.int64, device=DEV)
    mj = torch.zeros(10, dtype=torch.int32, device=DEV)
    for mode, x in ((c3.EXACT, ev), (c3.STATISTICAL, ev.float())):
        with pytest.raises(c3.C3Error, match=r"\(-1\)"):
            c3.consensus(x, mode, out=(st, bm, mj))
    with pytest.raises(c3.C3Error, match=r"\(-1\)"):
        c3.localize(st, bm, mj, None, R=1)
    with pytest.raises(c3.C3Error):
        c3.confirm(bm.reshape(10, 1), bm.reshape(10, 1), 1)
    fp = torch.zeros((4, 3, 1), dtype=torch.int64, device=DEV)
    with pytest.raises(c3.C3Error):
        c3.timing_consensus(fp, fp.float())
    torch.cuda.synchronize()
    assert (st == 0xAB).all().item()
    x = torch.randn(5000, device=DEV)
    rec = c3.signature([[x]], 4096)
    assert rec.shape[:2] == (1, 5)


@pytest.mark.parametrize("R", [2, 3, 4, 5, 7, 8, 9, 16, 31, 33, 64])
def test_exact_consensus_matches_oracle(R):
    _print_case("exact consensus", R)
    rng = np.random.default_rng(R)
    U = 5000
    ev = rng.integers(0, 3, size=(U, R)).astype(np.int64) * (2 ** 40 + 12345)
    ev[: U // 3] = 7
    ev[U // 3: U // 2, 0] = -1
    st, bm, mj = c3.consensus(torch.from_numpy(ev).to(DEV), c3.EXACT)
    ost, obm, omj = oracle.vote_exact(ev.view(np.uint64), replica_axis=1)
    assert np.array_equal(st.cpu().numpy(), ost)
    assert np.array_equal(bm.cpu().numpy().view(np.uint64), obm)
    assert np.array_equal(mj.cpu().numpy(), omj)


@pytest.mark.parametrize("R", [2, 3, 4, 5, 8, 13, 16, 64])
@pytest.mark.parametrize("dt", [np.float32, np.float64])
def test_statistical_consensus_matches_oracle(R, dt):
    _print_case("statistical consensus", R, dt)
    rng = np.random.default_rng(100 + R)
    U = 4000
    tau = np.exp(rng.standard_normal((U, R)) * 0.02).astype(dt)
    tau[::5, 0] *= 1.3
    tau[::9, -1] = tau[::9, 0]
    tau[::13, : R // 2 + 1] = 1.0
    tau[::17] = 2.0
    tau[1::19, 0] = np.nan
    tau[2::23, -1] = np.inf
    tau[3::29, : (R + 1) // 2] = np.nan
    st, bm, mj = c3.consensus(torch.from_numpy(tau).to(DEV), c3.STATISTICAL)
    ost, obm, omj = oracle.vote_statistical(tau, oracle.KAPPA_DEFAULT, replica_axis=1)
    assert np.array_equal(st.cpu().numpy(), ost)
    assert np.array_equal(bm.cpu().numpy().view(np.uint64), obm)
    assert np.array_equal(mj.cpu().numpy(), omj)


@pytest.mark.parametrize("R", [4, 5, 8, 16])
@pytest.mark.parametrize("dt", [np.float32, np.float64])
def test_statistical_consensus_extremes(R, dt):
    # magnitudes where the median's sum and the deviations overflow to inf,
    # subnormals, signed zeros and mixed signs at the top of the range
    _print_case("statistical extremes", R, dt)
    rng = np.random.default_rng(7 * R)
    big = np.finfo(dt).max
    tiny = np.finfo(dt).smallest_subnormal
    rows = []
    for _ in range(400):
        kind = rng.integers(0, 7)
        if kind == 0:
            v = rng.choice([big, -big], size=R)
        elif kind == 1:
            v = big * (1 - rng.random(R) * 1e-3)
        elif kind == 2:
            v = np.where(rng.random(R) < 0.5, big * 0.9, -big * 0.9)
        elif kind == 3:
            v = tiny * rng.integers(0, 5, size=R)
        elif kind == 4:
            v = rng.choice([0.0, -0.0, tiny, -tiny], size=R)
        elif kind == 5:
            v = np.concatenate([np.full(R - 1, big / 2), [-big]])
        else:
            v = (big / 8) * np.clip(rng.standard_normal(R), -6, 6)
        rows.append(v)
    tau = np.array(rows, dtype=dt)
    st, bm, mj = c3.consensus(torch.from_numpy(tau).to(DEV), c3.STATISTICAL)
    ost, obm, omj = oracle.vote_statistical(tau, oracle.KAPPA_DEFAULT, replica_axis=1)
    assert np.array_equal(st.cpu().numpy(), ost)
    assert np.array_equal(bm.cpu().numpy().view(np.uint64), obm)
    assert np.array_equal(mj.cpu().numpy(), omj)


def test_statistical_closed_forms_on_gpu():
    _print_case("statistical closed forms")
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "statistical_closed_forms.txt")
    for ln in open(path):
        if not ln.strip() or ln.startswith("#"):
            continue
        vals, status, bits, _ = [s.strip() for s in ln.split("|")]
        ev = torch.tensor([[float(v) for v in vals.split()]], dtype=torch.float64, device=DEV)
        st, bm, _ = c3.consensus(ev, c3.STATISTICAL)
        want = 0 if bits == "-" else sum(1 << int(b) for b in bits.split())
        code = {"AGREE": 0, "ATTRIBUTED": 1, "INCONCLUSIVE": 2}[status]
        assert (int(st[0]), int(bm[0])) == (code, want), ln


@pytest.mark.parametrize("U", [0, 1, 2047, 2048, 2049, 32768, 32769, 70000])
def test_localize_matches_oracle(U):
    _print_case("localize", U)
    rng = np.random.default_rng(U)
    R = 6
    ev = rng.integers(0, 2, size=(max(U, 1), R)).astype(np.int64)[:U]
    ev[rng.random(U) < 0.7] = 0
    evt = torch.from_numpy(ev).to(DEV) if U else torch.zeros((0, R), dtype=torch.int64, device=DEV)
    st, bm, mj = c3.consensus(evt, c3.EXACT, R=R)
    ost, obm, omj = oracle.vote_exact(ev.view(np.uint64).reshape(U, R), replica_axis=1) if U else \
        (np.zeros(0, np.uint8), np.zeros(0, np.uint64), np.zeros(0, np.int32))
    for cap in (None, 5):
        outl, und, cnt = c3.localize(st, bm, mj, None, R=R, out_cap=cap, und_cap=cap)
        torch.cuda.synchronize()
        loc = oracle.localize(ost, obm, omj, R, out_cap=cap, und_cap=cap)
        assert cnt.cpu().tolist() == loc["counts"].tolist()
        o = c3.outliers_numpy(outl, cnt)
        assert o["chunk"].tolist() == loc["unit"].tolist()
        assert o["replica"].tolist() == loc["replica"].tolist()
        assert o["majority_replica"].tolist() == loc["majority"].tolist()
        n_u = min(int(cnt[1]), und.numel())
        assert und.cpu().numpy()[:n_u].tolist() == loc["undecided"].tolist()


@pytest.mark.parametrize("R", [3, 8, 13, 20])
@pytest.mark.parametrize("T,W", [(200, 16), (64, 16), (65, 16), (10, 16), (1, 1), (130, 7),
                                 (200, 64), (200, 65), (90, 100), (300, 63), (300, 1), (129, 2)])
def test_confirm_matches_oracle(T, W, R):
    _print_case("confirm", T, W, R)
    rng = np.random.default_rng(T * 31 + W + 1000 * R)
    G = 37
    fpb = (rng.random((T, G, R)) < 0.02)
    tmb = (rng.random((T, G, R)) < np.where((np.arange(R)[None, None, :] + np.arange(G)[None, :, None]) % 11 == 0, 0.7, 0.05))
    pack = lambda b: (b.astype(np.uint64) << np.arange(R, dtype=np.uint64)).sum(-1).astype(np.uint64)
    fp, tm = pack(fpb), pack(tmb)
    out = c3.verdicts_numpy(c3.confirm(torch.from_numpy(fp.view(np.int64)).to(DEV),
                                       torch.from_numpy(tm.view(np.int64)).to(DEV), R, W))
    ref = oracle.confirm(fp, tm, R, W)
    assert np.array_equal(out["flags"], ref["flags"])
    assert np.array_equal(out["first_divergent_iter"], ref["first_div"])
    assert np.array_equal(out["divergent_count"], ref["div_count"])
    assert np.array_equal(out["slow_count"], ref["slow_count"])
    assert np.array_equal(out["max_window_slow"], ref["max_window"])
    assert np.array_equal(out["first_straggler_window"], ref["first_window"])


@pytest.mark.parametrize("R", [8, 20])
@pytest.mark.parametrize("W", [1, 2, 16, 80])
def test_confirm_pair_across_segments(W, R):
    # slow at t0 and t0 + 1 for one rank, across every segment boundary
    # of 32 and 64 iterations
    _print_case("confirm pair", W, R)
    T, G = 260, 5
    for t0 in (31, 63, 127, 191):
        fp = np.zeros((T, G), dtype=np.uint64)
        tm = np.zeros((T, G), dtype=np.uint64)
        tm[t0, 2] = tm[t0 + 1, 2] = np.uint64(1 << 3)
        out = c3.verdicts_numpy(c3.confirm(torch.from_numpy(fp.view(np.int64)).to(DEV),
                                           torch.from_numpy(tm.view(np.int64)).to(DEV), R, W))
        ref = oracle.confirm(fp, tm, R, W)
        assert ref["flags"][3 * G + 2] & 4
        for k, rk in (("flags", "flags"), ("slow_count", "slow_count"),
                      ("max_window_slow", "max_window"),
                      ("first_straggler_window", "first_window")):
            assert np.array_equal(out[k], ref[rk]), (t0, k)


# ---------------------------------------------------------------------------
# full sizes, benchmark launch configuration
# ---------------------------------------------------------------------------
def _oracle_records_streamed(w, workers=None):
    """Oracle records [R, C] of a full-size workload, every (replica, chunk):
    one (replica, tensor) is copied to the host at a time (8 GB at most for
    the Adam shard) and its chunks are signed by a pool of host threads (the
    oracle is plain C called through ctypes, which releases the GIL)."""
    from concurrent.futures import ThreadPoolExecutor
    import os
    workers = workers or max(1, min(16, len(os.sched_getaffinity(0))))
    C = oracle.num_chunks(w.metas, w.chunk_bytes)
    out = dict(sig=np.zeros((w.R, C), np.uint64), n_elems=np.zeros((w.R, C), np.uint64),
               nan=np.zeros((w.R, C), np.uint32), inf=np.zeros((w.R, C), np.uint32),
               absmax=np.zeros((w.R, C), np.float64), sum=np.zeros((w.R, C), np.float64),
               sumsq=np.zeros((w.R, C), np.float64), tensor=np.zeros((w.R, C), np.uint32),
               chunk=np.zeros((w.R, C), np.uint32))
    bases = _chunk_bases(w.metas, w.chunk_bytes)
    oracle.keys()                                   # load the library before the threads
    with ThreadPoolExecutor(workers) as pool:
        for r in range(w.R):
            for t, (d, shape) in enumerate(w.metas):
                host = workloads.host_bytes(w.replicas[r][t])
                nb = host.size
                nc = int(bases[t + 1] - bases[t])

                def one(k, host=host, d=d, shape=shape, nb=nb):
                    lo = k * w.chunk_bytes
                    return k, oracle.chunk_signature(host[lo:min(nb, lo + w.chunk_bytes)], d,
                                                     list(shape), k)
                for k, ref in pool.map(one, range(nc)):
                    c = int(bases[t]) + k
                    for f in ("sig", "n_elems", "nan", "inf", "absmax", "sum", "sumsq"):
                        out[f][r, c] = ref[f]
                    out["tensor"][r, c] = t
                    out["chunk"][r, c] = k
                del host
    return out


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_full_config_parity(k):
    """Every configuration at its full size, in the benchmark's launch
    configuration: every record of every replica against the oracle, the
    votes and lists against the oracle's on those records, the planted faults
    exactly, and signature equality equal to byte equality on every chunk."""
    _print_case("full config", k)
    torch.cuda.empty_cache()
    w = workloads.make(k, device=DEV, scale="full")
    g = _gpu_pipeline(w)
    C = g["records"].shape[1]
    # the planted faults are exactly the outliers / undecided chunks
    want_out, want_und = _expected(w)
    assert set(zip(g["outliers"]["replica"].tolist(), g["outliers"]["chunk"].tolist())) == want_out
    assert set(g["undecided"].tolist()) == want_und
    if k == 1:
        # the workload's stated answer: replica 2, the chunk of the flipped element
        f = w.faults[0]
        assert [(int(c), int(r)) for c, r in zip(g["outliers"]["chunk"], g["outliers"]["replica"])] \
            == [(f.byte_offset // w.chunk_bytes, 2)]
    # signature equality <=> byte equality with replica 0, every chunk
    bases = _chunk_bases(w.metas, w.chunk_bytes)
    for r in range(1, w.R):
        same = np.zeros(C, bool)
        for t in range(len(w.metas)):
            a = w.replicas[0][t].view(-1).view(torch.uint8)
            b = w.replicas[r][t].view(-1).view(torch.uint8)
            nb = a.numel()
            nfull = nb // w.chunk_bytes
            eq = []
            if nfull:
                av = a[: nfull * w.chunk_bytes].view(torch.int64).view(nfull, -1)
                bv = b[: nfull * w.chunk_bytes].view(torch.int64).view(nfull, -1)
                eq += (av == bv).all(dim=1).cpu().tolist()
            if nb % w.chunk_bytes or nb == 0:
                eq.append(bool(torch.equal(a[nfull * w.chunk_bytes:], b[nfull * w.chunk_bytes:])))
            same[int(bases[t]): int(bases[t + 1])] = eq
        assert np.array_equal(same, g["records"]["sig"][r] == g["records"]["sig"][0]), r
    # every record of every replica against the oracle
    print("CASE full config", k, "oracle over", w.total_bytes, "bytes", flush=True)
    ref = _oracle_records_streamed(w)
    compare_all_records(g["records"], ref)
    # votes and lists against the oracle's on the oracle's own records
    ost, obm, omj = oracle.vote_exact(ref["sig"])
    assert np.array_equal(g["status"], ost) and np.array_equal(g["bitmap"], obm)
    assert np.array_equal(g["maj"], omj)
    loc = oracle.localize(ost, obm, omj, w.R)
    assert g["counts"].tolist() == loc["counts"].tolist()
    assert g["outliers"]["chunk"].tolist() == loc["unit"].tolist()
    assert g["outliers"]["replica"].tolist() == loc["replica"].tolist()
    assert g["outliers"]["majority_replica"].tolist() == loc["majority"].tolist()
    assert g["undecided"].tolist() == loc["undecided"].tolist()
    for i, (c, r, m) in enumerate(zip(loc["unit"], loc["replica"], loc["majority"])):
        o = g["outliers"][i]
        for z, rr in ((0, r), (1, m)):
            assert int(o["nan_count"][z]) == int(ref["nan"][rr, c])
            assert int(o["inf_count"][z]) == int(ref["inf"][rr, c])
            assert float(o["absmax"][z]) == float(ref["absmax"][rr, c])
    del w, g, ref
    torch.cuda.empty_cache()


def test_full_config5_timing_consensus():
    _print_case("full config 5")
    torch.cuda.empty_cache()
    w = workloads.make(5, device=DEV, scale="full")
    T, G, R = w.T, w.G, w.R
    fst, fbm, fmj = c3.consensus(w.fingerprints, c3.EXACT)
    tst, tbm, tmj = c3.consensus(w.times, c3.STATISTICAL)
    ver = c3.verdicts_numpy(c3.confirm(fbm.view(T, G), tbm.view(T, G), R, 16))
    fp = w.fingerprints.cpu().numpy().view(np.uint64).reshape(T * G, R)
    tau = w.times.cpu().numpy().reshape(T * G, R)
    ost, obm, omj = oracle.vote_exact(fp, replica_axis=1)
    assert np.array_equal(fst.cpu().numpy(), ost) and np.array_equal(fbm.cpu().numpy().view(np.uint64), obm)
    assert np.array_equal(fmj.cpu().numpy(), omj)
    sst, sbm, smj = oracle.vote_statistical(tau, oracle.KAPPA_DEFAULT, replica_axis=1)
    assert np.array_equal(tst.cpu().numpy(), sst) and np.array_equal(tbm.cpu().numpy().view(np.uint64), sbm)
    assert np.array_equal(tmj.cpu().numpy(), smj)
    ref = oracle.confirm(obm.reshape(T, G), sbm.reshape(T, G), R, 16)
    assert np.array_equal(ver["flags"], ref["flags"])
    assert np.array_equal(ver["first_divergent_iter"], ref["first_div"])
    assert np.array_equal(ver["max_window_slow"], ref["max_window"])
    # ground truth: exactly the planted ranks
    strag = set(np.nonzero(ver["flags"] & c3.RANK_STRAGGLER)[0].tolist())
    proto = {int(r): int(ver["first_divergent_iter"][r])
             for r in np.nonzero(ver["flags"] & c3.RANK_PROTOCOL)[0]}
    assert strag == set(w.stragglers)
    assert proto == w.divergent


# ---------------------------------------------------------------------------
# checkpoint certification fed by GPU verdicts (Sec. 8, Algorithm 3)
# ---------------------------------------------------------------------------
def test_checkpoint_gate_fed_by_gpu_verdicts():
    """The paper's two-recipe scenario driven by real verdicts on Adam-shard
    state: steps 1-4 clean, SDC at step 5 -> recover the step-2 checkpoint."""
    _print_case("checkpoint gate")
    w = workloads.make(4, device=DEV, scale="small")
    clean_src = next(r for r in range(w.R) if all(f.replica != r for f in w.faults))
    clean = [[t.clone() for t in w.replicas[clean_src]] for _ in range(w.R)]
    gate = c3.CheckpointGate(K=2)
    for step in range(1, 6):
        reps = w.replicas if step == 5 else clean
        rec = c3.signature(reps, w.chunk_bytes)
        st, bm, mj = c3.consensus(rec, c3.EXACT)
        _, _, cnt = c3.localize(st, bm, mj, rec)
        torch.cuda.synchronize()
        counts = cnt.cpu().tolist()
        outcome = c3.job_outcome(counts[1] + counts[2], 0, 0)
        act = gate.save(outcome, step)
        if step < 5:
            assert outcome == c3.OUTCOME_OK and act.captured == 1
        else:
            assert outcome == c3.OUTCOME_SDC and act.retrieve == 1 and act.retrieve_id == 2
    assert (gate.state.candidate, gate.state.verified) == (4, 2)
