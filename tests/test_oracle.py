"""Pins of the CPU oracle against what the paper and mathematics fix.

These tests never touch the HIP path.  Each pin is independent of the oracle's
own code: published test vectors, closed forms worked by hand, numpy / math
library routines, brute force over tiny inputs, and the byte-equality
definition of the exact result.
"""
import collections
import ctypes
import itertools
import math
import os

import numpy as np
import pytest

import oracle
import workloads

GOLD = os.path.join(os.path.dirname(__file__), "golden")
M64 = (1 << 64) - 1
STATUS = {"AGREE": oracle.AGREE, "ATTRIBUTED": oracle.ATTRIBUTED, "INCONCLUSIVE": oracle.INCONCLUSIVE}


def _lines(name):
    with open(os.path.join(GOLD, name)) as f:
        return [ln.strip() for ln in f if ln.strip() and not ln.startswith("#")]


# ---------------------------------------------------------------------------
# primitives
# ---------------------------------------------------------------------------
def test_splitmix64_published_vectors():
    rows = [ln.split() for ln in _lines("splitmix64_vectors.txt")]
    for seed in {int(r[0]) for r in rows}:
        want = {int(r[1]): int(r[2], 16) for r in rows if int(r[0]) == seed}
        got = oracle.splitmix64_stream(seed, max(want) + 1)
        for i, v in want.items():
            assert int(got[i]) == v, (seed, i)


def _fmix64_inverse(h):
    # Inverse of fmix64 derived independently: x ^= x >> 33 is an involution on
    # 64-bit words (shift >= 32), and multiplication by an odd constant is
    # undone by its inverse modulo 2^64.
    c1, c2 = 0xFF51AFD7ED558CCD, 0xC4CEB9FE1A85EC53
    i1, i2 = pow(c1, -1, 1 << 64), pow(c2, -1, 1 << 64)
    h ^= h >> 33
    h = (h * i2) & M64
    h ^= h >> 33
    h = (h * i1) & M64
    h ^= h >> 33
    return h


def test_fmix64_is_the_murmur3_bijection():
    rng = np.random.default_rng(7)
    xs = [0, 1, M64, 1 << 63] + [int(v) for v in rng.integers(0, 2 ** 63, 200)]
    for x in xs:
        assert _fmix64_inverse(oracle.fmix64(x)) == x
    assert oracle.fmix64(0) == 0


def test_fmix64_avalanche():
    rng = np.random.default_rng(8)
    flips = []
    for x in rng.integers(0, 2 ** 63, 64):
        x = int(x)
        h = oracle.fmix64(x)
        for b in range(64):
            flips.append(bin(h ^ oracle.fmix64(x ^ (1 << b))).count("1"))
    assert 31.0 < np.mean(flips) < 33.0
    assert min(flips) >= 8


def test_key_table_properties():
    K = oracle.keys()
    st = oracle.splitmix64_stream(0x43335349472D3101, 258)
    assert np.array_equal(K, (st & np.uint64(0xFFFFFFFF)).astype(np.uint32))
    # K[i] != K[i + 2] guarantees that a change confined to one word moves A or B
    assert all(K[i] != K[i + 2] for i in range(256))


def _nh_bigint(data: bytes):
    """Third implementation of the NH fold with Python integers."""
    K = [int(k) for k in oracle.keys()]
    n = len(data)
    D = 4 * ((n + 15) // 16)
    pad = data + bytes(4 * D - n)
    m = [int.from_bytes(pad[4 * j:4 * j + 4], "little") for j in range(D)]
    A = B = 0
    for p in range(0, D, 2):
        q, beta = p % 256, ((p // 256) * 0x9E3779B9) % (1 << 32)
        w = lambda x, k: (x + k + beta) % (1 << 32)
        A += w(m[p], K[q]) * w(m[p + 1], K[q + 1])
        B += w(m[p], K[q + 2]) * w(m[p + 1], K[q + 3])
    return A % (1 << 64), B % (1 << 64)


@pytest.mark.parametrize("n", [0, 1, 3, 4, 15, 16, 17, 1000, 1024, 1040, 2051, 4096])
def test_nh_matches_bigint(n):
    rng = np.random.default_rng(n)
    data = rng.integers(0, 256, n, dtype=np.uint8)
    assert oracle.nh(data) == _nh_bigint(data.tobytes())


def test_nh_empty_is_zero_and_padding_counts():
    assert oracle.nh(np.zeros(0, np.uint8)) == (0, 0)
    # a zero-padded tail is hashed (D = 4 ceil(n / 16)) but n enters the
    # finalizer, so 15 and 16 zero bytes have equal folds and distinct signatures
    z15, z16 = np.zeros(15, np.uint8), np.zeros(16, np.uint8)
    assert oracle.nh(z15) == oracle.nh(z16)
    assert oracle.chunk_signature(z15, oracle.RAW, [15], 0)["sig"] != \
        oracle.chunk_signature(z16, oracle.RAW, [16], 0)["sig"]
    # same dtype, shape and chunk index, lengths 1033 and 1040 (the chunk plan
    # of a 1040-byte tensor under two chunk sizes): equal folds, the length
    # alone must separate the signatures (the evidence covers the bytes)
    z1033, z1040 = np.zeros(1033, np.uint8), np.zeros(1040, np.uint8)
    assert oracle.nh(z1033) == oracle.nh(z1040)
    assert oracle.chunk_signature(z1033, oracle.RAW, [1040], 0)["sig"] != \
        oracle.chunk_signature(z1040, oracle.RAW, [1040], 0)["sig"]


def test_signature_is_sensitive_to_metadata():
    d = np.arange(64, dtype=np.float32).view(np.uint8)
    s = oracle.chunk_signature(d, oracle.F32, [64], 0)["sig"]
    assert s != oracle.chunk_signature(d, oracle.F32, [8, 8], 0)["sig"]   # shape
    assert oracle.chunk_signature(d, oracle.F32, [8, 8], 0)["sig"] != \
        oracle.chunk_signature(d, oracle.F32, [4, 16], 0)["sig"]          # dims, same rank
    assert s != oracle.chunk_signature(d, oracle.RAW, [64], 0)["sig"]     # dtype
    assert s != oracle.chunk_signature(d, oracle.F32, [64], 1)["sig"]     # position
    # same bytes, same metadata -> same signature (determinism)
    assert s == oracle.chunk_signature(d.copy(), oracle.F32, [64], 0)["sig"]


def test_signature_is_position_sensitive():
    rng = np.random.default_rng(3)
    words = rng.integers(0, 2 ** 32, 512, dtype=np.uint64).astype(np.uint32)
    base = oracle.chunk_signature(words.view(np.uint8), oracle.RAW, [2048], 0)["sig"]
    for i, j in [(0, 1), (0, 2), (1, 3), (5, 300), (0, 256), (10, 266)]:
        w = words.copy()
        w[i], w[j] = w[j], w[i]
        if w[i] == w[j]:
            continue
        assert oracle.chunk_signature(w.view(np.uint8), oracle.RAW, [2048], 0)["sig"] != base


# ---------------------------------------------------------------------------
# exhaustive single-bit detection at the right chunk
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dtype,np_dtype", [(oracle.F32, np.float32), (oracle.BF16, np.uint16),
                                            (oracle.F16, np.float16), (oracle.RAW, np.uint8)])
def test_every_single_bit_flip_is_detected(dtype, np_dtype):
    rng = np.random.default_rng(11 + dtype)
    es = oracle.ELEM_SIZE[dtype]
    n_el = 3 * 64 + 5                                     # 3 full chunks + ragged tail
    if dtype == oracle.BF16:
        raw = (rng.standard_normal(n_el).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    elif dtype == oracle.RAW:
        raw = rng.integers(0, 256, n_el, dtype=np.uint8)
    else:
        raw = rng.standard_normal(n_el).astype(np_dtype)
    data = raw.view(np.uint8).copy()
    chunk = 64 * es
    clean = [oracle.chunk_signature(data[k:k + chunk], dtype, [n_el], k // chunk)["sig"]
             for k in range(0, data.size, chunk)]
    for byte in range(data.size):
        k = byte // chunk
        lo = k * chunk
        for bit in range(8):
            d = data[lo:lo + chunk].copy()
            d[byte - lo] ^= 1 << bit
            assert oracle.chunk_signature(d, dtype, [n_el], k)["sig"] != clean[k], (byte, bit)


def test_single_flip_localized_through_the_pipeline():
    rng = np.random.default_rng(5)
    metas = [(oracle.F32, (1000,)), (oracle.BF16, (333,))]
    chunk_bytes = 1024
    base = [rng.standard_normal(1000).astype(np.float32).view(np.uint8),
            (rng.standard_normal(333).astype(np.float32).view(np.uint32) >> 16)
            .astype(np.uint16).view(np.uint8)]
    R = 3
    for t, byte, bit in [(0, 0, 0), (0, 3999, 7), (0, 2048, 3), (1, 665, 6), (1, 100, 0)]:
        for fr in range(R):
            reps = [[b.copy() for b in base] for _ in range(R)]
            reps[fr][t][byte] ^= 1 << bit
            rec = oracle.signature(reps, metas, chunk_bytes)
            st, bm, mj = oracle.vote_exact(rec["sig"])
            loc = oracle.localize(st, bm, mj, R)
            chunk = (0 if t == 0 else 4) + byte // chunk_bytes
            assert list(loc["unit"]) == [chunk] and list(loc["replica"]) == [fr]
            assert loc["counts"].tolist() == [1, 0, 1]


# ---------------------------------------------------------------------------
# numerical summary vs numpy / math.fsum
# ---------------------------------------------------------------------------
def _special_f32():
    specials = np.array([0x00000000, 0x80000000, 0x00000001, 0x807FFFFF, 0x7F7FFFFF, 0xFF7FFFFF,
                         0x7F800000, 0xFF800000, 0x7FC00000, 0x7F800001, 0xFFFFFFFF, 0x3F800000],
                        dtype=np.uint32)
    return specials


def _values(dtype, raw_u8):
    if dtype == oracle.F32:
        return raw_u8.view(np.float32).astype(np.float64)
    if dtype == oracle.F16:
        return raw_u8.view(np.float16).astype(np.float64)
    # bfloat16 is the upper half of an IEEE binary32
    return (raw_u8.view(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


@pytest.mark.parametrize("dtype", [oracle.F32, oracle.BF16, oracle.F16])
@pytest.mark.parametrize("case", ["normal", "specials", "tiny", "huge", "cancel", "absorb"])
def test_stats_match_numpy_and_fsum(dtype, case):
    rng = np.random.default_rng(hash((dtype, case)) % 2 ** 32)
    n = 5000
    if case == "normal":
        x = rng.standard_normal(n)
    elif case == "tiny":
        x = rng.standard_normal(n) * 1e-40
    elif case == "huge":
        x = rng.standard_normal(n) * (1e38 if dtype != oracle.F16 else 6e4)
    elif case == "cancel":
        x = np.concatenate([rng.standard_normal(n // 2) * 1e3, [0.0]])
        x = np.concatenate([x, -x])
    elif case == "absorb":
        # a huge value absorbs many small ones in a plain fp64 sum; the exact
        # sum is the small ones (a compensated sum recovers them)
        big = 2.0 ** 60 if dtype != oracle.F16 else 2.0 ** 15
        small = 1.0 if dtype != oracle.F16 else 2.0 ** -10
        x = np.concatenate([[big], np.full(1000, small), [-big]])
    else:
        x = rng.standard_normal(n)
    if dtype == oracle.F32:
        raw = x.astype(np.float32).view(np.uint32)
        if case == "specials":
            raw[:12] = _special_f32()
            raw[100:110] = rng.integers(0, 2 ** 23, 10).astype(np.uint32)      # denormals
    elif dtype == oracle.F16:
        raw = x.astype(np.float16).view(np.uint16)
        if case == "specials":
            raw[:8] = np.array([0, 0x8000, 1, 0x83FF, 0x7BFF, 0x7C00, 0xFC00, 0x7E00], np.uint16)
    else:
        raw = (x.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        if case == "specials":
            raw[:10] = np.array([0, 0x8000, 1, 0x807F, 0x7F7F, 0x7F80, 0xFF80, 0x7FC0, 0x7F81, 0xFFFF],
                                np.uint16)
    data = raw.view(np.uint8)
    vals = _values(dtype, data)
    rec = oracle.chunk_signature(data, dtype, [raw.size], 0)
    fin = np.isfinite(vals)
    assert rec["nan"] == int(np.isnan(vals).sum())
    assert rec["inf"] == int(np.isinf(vals).sum())
    assert rec["n_elems"] == raw.size
    assert rec["absmax"] == (float(np.max(np.abs(vals[fin]))) if fin.any() else 0.0)
    f = vals[fin]
    exact_sum = math.fsum(f.tolist())
    exact_sq = math.fsum((f * f).tolist())          # squares are exact in fp64 here
    sabs = math.fsum(np.abs(f).tolist())
    tol = 2.0 ** -52 * abs(exact_sum) + f.size * 2.0 ** -104 * sabs
    assert abs(rec["sum"] - exact_sum) <= tol
    assert abs(rec["sumsq"] - exact_sq) <= 2.0 ** -52 * exact_sq + f.size * 2.0 ** -104 * exact_sq


def test_raw_chunks_carry_hash_only():
    d = np.arange(100, dtype=np.uint8)
    rec = oracle.chunk_signature(d, oracle.RAW, [100], 0)
    assert rec["n_elems"] == 100 and rec["nan"] == 0 and rec["sum"] == 0.0 and rec["absmax"] == 0.0


# ---------------------------------------------------------------------------
# exact vote: paper cases, brute force, Boyer-Moore MJRTY
# ---------------------------------------------------------------------------
def test_exact_vote_paper_cases():
    for ln in _lines("exact_vote_paper_cases.txt"):
        labels, status, bits, maj = [s.strip() for s in ln.split("|")]
        labels = labels.split()
        code = {v: i + 100 for i, v in enumerate(sorted(set(labels)))}
        ev = np.array([[code[v] for v in labels]], np.uint64)
        if status == "REJECTED":
            with pytest.raises(ValueError):
                oracle.vote_exact(ev, replica_axis=1)
            continue
        st, bm, mj = oracle.vote_exact(ev, replica_axis=1)
        want_bits = 0 if bits == "-" else sum(1 << int(b) for b in bits.split())
        assert (int(st[0]), int(bm[0]), int(mj[0])) == (STATUS[status], want_bits, int(maj)), ln


@pytest.mark.parametrize("R", [2, 3, 4, 5, 6, 7])
def test_exact_vote_brute_force_all_label_vectors(R):
    ev = np.array(list(itertools.product(range(R), repeat=R)), dtype=np.uint64).reshape(-1, R)
    st, bm, mj = oracle.vote_exact(ev, replica_axis=1)
    # vectorized direct definition: c* = max count; strict majority iff 2 c* > R
    cnt = (ev[:, :, None] == ev[:, None, :]).sum(2)
    cstar = cnt.max(1)
    has = 2 * cstar > R
    first = cnt.argmax(1)
    vstar = ev[np.arange(ev.shape[0]), first]
    diff = (ev != vstar[:, None]) & has[:, None]
    want_bm = (diff.astype(np.uint64) << np.arange(R, dtype=np.uint64)).sum(1)
    want_st = np.where(~has, oracle.INCONCLUSIVE, np.where(want_bm != 0, oracle.ATTRIBUTED, oracle.AGREE))
    assert np.array_equal(st, want_st.astype(np.uint8))
    assert np.array_equal(bm, want_bm.astype(np.uint64))
    assert np.array_equal(mj, np.where(has, first, -1).astype(np.int32))


def test_singleton_group_is_rejected():
    """Sec. 4: a group of one peer provides no comparison.  The C functions
    themselves return -1 (not only the Python wrappers), for every vote,
    localization and confirmation."""
    L = oracle._load()
    ev = np.array([7, 8, 9], np.uint64)
    f = np.array([1.0, 2.0, 3.0])
    st, bm, mj = np.zeros(3, np.uint8), np.zeros(3, np.uint64), np.zeros(3, np.int32)
    P = oracle._p
    assert L.c3o_vote_exact(P(ev), oracle.EV_U64, 8, 8, 1, 3, P(st), P(bm), P(mj)) == -1
    assert L.c3o_vote_statistical(P(f), oracle.EV_F64, 8, 8, 1, 3, ctypes.c_double(5.0),
                                  P(st), P(bm), P(mj)) == -1
    chunks = (ctypes.c_void_p * 3)(*[ev.ctypes.data + 8 * i for i in range(3)])
    lens = np.full(3, 8, np.uint64)
    assert L.c3o_vote_bytes(chunks, P(lens), 1, 3, P(st), P(bm), P(mj)) == -1
    ou, orr, om, und, cnt = (np.zeros(3, np.int64), np.zeros(3, np.int32), np.zeros(3, np.int32),
                             np.zeros(3, np.int64), np.zeros(3, np.int64))
    assert L.c3o_localize(P(st), P(bm), P(mj), 1, 3, P(ou), P(orr), P(om), 3, P(und), 3,
                          P(cnt)) == -1
    out = [np.zeros(3, np.uint32), np.zeros(3, np.int32), np.zeros(3, np.uint32),
           np.zeros(3, np.uint32), np.zeros(3, np.uint32), np.zeros(3, np.int32)]
    assert L.c3o_confirm(P(bm), P(bm), 1, 3, 1, 16, *[P(a) for a in out]) == -1
    for call in (lambda: oracle.vote_exact(ev.reshape(1, 3)),
                 lambda: oracle.vote_statistical(f.reshape(1, 3)),
                 lambda: oracle.localize(st, bm, mj, 1),
                 lambda: oracle.confirm(bm.reshape(3, 1), bm.reshape(3, 1), 1)):
        with pytest.raises(ValueError):
            call()
    # two peers are a group (Sec. 4): agreement certifies, disagreement is inconclusive
    st2, bm2, mj2 = oracle.vote_exact(np.array([[5, 5], [5, 6]], np.uint64), replica_axis=1)
    assert st2.tolist() == [oracle.AGREE, oracle.INCONCLUSIVE]


def _mjrty(vals):
    # Boyer & Moore, "MJRTY - a fast majority vote algorithm" (1991)
    cand, k = None, 0
    for v in vals:
        if k == 0:
            cand, k = v, 1
        elif v == cand:
            k += 1
        else:
            k -= 1
    return cand if 2 * sum(v == cand for v in vals) > len(vals) else None


def test_exact_vote_agrees_with_mjrty():
    rng = np.random.default_rng(13)
    for R in range(2, 65, 3):
        ev = rng.integers(0, 3, size=(400, R)).astype(np.uint64)
        ev[::3] = 1
        st, bm, mj = oracle.vote_exact(ev, replica_axis=1)
        for u in range(ev.shape[0]):
            m = _mjrty(ev[u].tolist())
            if m is None:
                assert st[u] == oracle.INCONCLUSIVE and bm[u] == 0
            else:
                want = sum(1 << r for r in range(R) if ev[u, r] != m)
                assert int(bm[u]) == want and ev[u, mj[u]] == m
                assert mj[u] == min(r for r in range(R) if ev[u, r] == m)


def _row_int(bm, u, R):
    """Outlier bitmap of unit u as one Python integer (bit r = replica r)."""
    w = np.asarray(bm, np.uint64).reshape(-1, oracle.bitmap_words(R))[u]
    return sum(int(x) << (64 * i) for i, x in enumerate(w))


def _wide_rows(R, rng):
    """Rows of R labels with their vote fixed by construction, not counted:
    (labels, status, outlier set, majority replica)."""
    rows = []
    for kind in range(6):
        for _ in range(8):
            if kind == 0:      # everyone agrees
                lab = np.full(R, 7)
                rows.append((lab, oracle.AGREE, set(), 0))
            elif kind == 1:    # a majority class of k > R/2 at random positions
                k = int(rng.integers(R // 2 + 1, R + 1))
                pos = rng.choice(R, size=k, replace=False)
                lab = 1000 + np.arange(R)                 # all others distinct
                lab[pos] = 5
                out = set(range(R)) - set(pos.tolist())
                rows.append((lab, oracle.ATTRIBUTED if out else oracle.AGREE, out, int(pos.min())))
            elif kind == 2:    # replica 0 outside a bare majority
                k = R // 2 + 1
                pos = rng.choice(np.arange(1, R), size=k, replace=False)
                lab = np.full(R, 3)
                lab[pos] = 9
                out = set(range(R)) - set(pos.tolist())
                rows.append((lab, oracle.ATTRIBUTED, out, int(pos.min())))
            elif kind == 3:    # two classes of R/2 (or a largest class below R/2)
                lab = np.where(rng.permutation(R) < R // 2, 1, 2)
                if R % 2:   # class 2 has (R + 1) / 2: move one of its members out
                    lab[int(rng.choice(np.flatnonzero(lab == 2)))] = 3
                rows.append((lab, oracle.INCONCLUSIVE, set(), -1))
            elif kind == 4:    # many small classes
                lab = rng.integers(0, 5, size=R)
                while (np.bincount(lab).max() * 2) > R:
                    lab = rng.integers(0, 5, size=R)
                rows.append((lab, oracle.INCONCLUSIVE, set(), -1))
            else:              # majority of exactly floor(R/2) + 1, rest in one other class
                k = R // 2 + 1
                pos = rng.choice(R, size=k, replace=False)
                lab = np.full(R, 4)
                lab[pos] = 8
                out = set(range(R)) - set(pos.tolist())
                rows.append((lab, oracle.ATTRIBUTED, out, int(pos.min())))
    return rows


@pytest.mark.parametrize("R", [65, 100, 127, 128, 129, 192, 255, 256])
def test_exact_vote_wide_groups_by_construction(R):
    """Peer groups above 64 (the paper's Table 2 lists degrees up to 192):
    multi-word bitmaps, every word's bits where the construction puts them."""
    rng = np.random.default_rng(R)
    rows = _wide_rows(R, rng)
    ev = np.array([r[0] for r in rows], np.uint64)
    st, bm, mj = oracle.vote_exact(ev, replica_axis=1)
    assert bm.shape == (len(rows), (R + 63) // 64)
    for u, (_, want_st, out, want_mj) in enumerate(rows):
        assert int(st[u]) == want_st, (u, want_st)
        assert _row_int(bm, u, R) == sum(1 << r for r in out), u
        assert int(mj[u]) == want_mj, u
    # the replica-major layout gives the same votes
    st2, bm2, mj2 = oracle.vote_exact(np.ascontiguousarray(ev.T), replica_axis=0)
    assert np.array_equal(st, st2) and np.array_equal(bm, bm2) and np.array_equal(mj, mj2)


def test_exact_vote_wide_groups_agree_with_mjrty():
    rng = np.random.default_rng(29)
    for R in (65, 96, 160, 192, 256):
        ev = rng.integers(0, 3, size=(60, R)).astype(np.uint64)
        ev[::3, : R // 2 + 2] = 1
        st, bm, mj = oracle.vote_exact(ev, replica_axis=1)
        for u in range(ev.shape[0]):
            m = _mjrty(ev[u].tolist())
            if m is None:
                assert st[u] == oracle.INCONCLUSIVE and _row_int(bm, u, R) == 0
            else:
                assert _row_int(bm, u, R) == sum(1 << r for r in range(R) if ev[u, r] != m)
                assert mj[u] == min(r for r in range(R) if ev[u, r] == m)


def test_byte_vote_wide_group_by_construction():
    rng = np.random.default_rng(31)
    R = 130
    rows = _wide_rows(R, rng)[::4]
    chunks = [[np.full(24, lab[r] % 251, np.uint8) if lab[r] < 1000 else
               np.frombuffer(int(lab[r]).to_bytes(24, "little"), np.uint8) for _, lab in
               enumerate([row[0] for row in rows])] for r in range(R)]
    st, bm, mj = oracle.vote_bytes(chunks)
    for u, (_, want_st, out, want_mj) in enumerate(rows):
        assert (int(st[u]), _row_int(bm, u, R), int(mj[u])) == (want_st, sum(1 << r for r in out),
                                                                 want_mj), u


def test_wide_groups_out_of_range():
    with pytest.raises(ValueError):
        oracle.vote_exact(np.zeros((257, 2), np.uint64))


# ---------------------------------------------------------------------------
# byte-equality definition == signature vote
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_byte_vote_equals_signature_vote_on_small_configs(k):
    w = workloads.make(k, device="cpu", scale="small")
    reps = [[workloads.host_bytes(t) for t in rep] for rep in w.replicas]
    rec = oracle.signature(reps, w.metas, w.chunk_bytes)
    s1 = oracle.vote_exact(rec["sig"])
    s2 = oracle.vote_bytes(oracle.chunk_views(reps, w.metas, w.chunk_bytes))
    for a, b in zip(s1, s2):
        assert np.array_equal(a, b)


def test_byte_vote_equals_signature_vote_random_splits():
    rng = np.random.default_rng(21)
    for trial in range(40):
        R = int(rng.integers(2, 9))
        n = int(rng.integers(1, 3000))
        base = rng.integers(0, 256, n, dtype=np.uint8)
        variants = [base]
        for _ in range(3):
            v = base.copy()
            v[rng.integers(0, n)] ^= np.uint8(1 << int(rng.integers(0, 8)))
            variants.append(v)
        reps = [[variants[int(rng.integers(0, 4)) if rng.random() < 0.4 else 0].copy()]
                for _ in range(R)]
        metas = [(oracle.RAW, (n,))]
        rec = oracle.signature(reps, metas, 1024)
        s1 = oracle.vote_exact(rec["sig"])
        s2 = oracle.vote_bytes(oracle.chunk_views(reps, metas, 1024))
        for a, b in zip(s1, s2):
            assert np.array_equal(a, b), trial


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_tensor_vote_equals_whole_tensor_byte_vote(k):
    w = workloads.make(k, device="cpu", scale="small")
    reps = [[workloads.host_bytes(t) for t in rep] for rep in w.replicas]
    rec = oracle.signature(reps, w.metas, w.chunk_bytes)
    ts = oracle.tensor_signature(rec, len(w.metas))
    s1 = oracle.vote_exact(ts)
    s2 = oracle.vote_bytes([[a for a in rep] for rep in reps])
    for a, b in zip(s1, s2):
        assert np.array_equal(a, b)
    assert s1[0].max() > 0                                # some tensor is not unanimous


def test_tensor_signature_moves_only_with_its_own_bytes():
    rng = np.random.default_rng(23)
    metas = [(oracle.F32, (700,)), (oracle.BF16, (1500,)), (oracle.RAW, (2500,))]
    base = [rng.integers(0, 256, 2800, dtype=np.uint8), rng.integers(0, 256, 3000, dtype=np.uint8),
            rng.integers(0, 256, 2500, dtype=np.uint8)]
    ref = oracle.tensor_signature(oracle.signature([base, base], metas, 1024), 3)[0]
    for t, a in enumerate(base):
        for pos in list(range(0, a.size, 1024)) + [a.size - 1]:
            mod = [b.copy() for b in base]
            mod[t][pos] ^= 0x40
            got = oracle.tensor_signature(oracle.signature([mod, base], metas, 1024), 3)[0]
            assert [got[i] != ref[i] for i in range(3)] == [i == t for i in range(3)], (t, pos)


def test_tensor_signature_sees_shape_and_chunk_count():
    d = np.arange(512, dtype=np.float32).view(np.uint8)
    r1 = oracle.signature([[d], [d.copy()]], [(oracle.F32, (512,))], 1024)
    r2 = oracle.signature([[d], [d.copy()]], [(oracle.F32, (16, 32))], 1024)
    r3 = oracle.signature([[d], [d.copy()]], [(oracle.F32, (512,))], 2048)
    t1, t2, t3 = (oracle.tensor_signature(r, 1) for r in (r1, r2, r3))
    assert t1[0, 0] == t1[1, 0] and t1[0, 0] != t2[0, 0] and t1[0, 0] != t3[0, 0]


# ---------------------------------------------------------------------------
# statistical vote: closed forms and numpy
# ---------------------------------------------------------------------------
def test_statistical_closed_forms():
    for ln in _lines("statistical_closed_forms.txt"):
        vals, status, bits, _d = [s.strip() for s in ln.split("|")]
        ev = np.array([[float(v) for v in vals.split()]], np.float64)
        st, bm, _ = oracle.vote_statistical(ev, replica_axis=1)
        want = 0 if bits == "-" else sum(1 << int(b) for b in bits.split())
        assert (int(st[0]), int(bm[0])) == (STATUS[status], want), ln


def _stat_numpy(tau, kappa):
    tau = np.asarray(tau, np.float64)
    fin = np.isfinite(tau)
    R = tau.size
    if 2 * fin.sum() <= R:
        return oracle.INCONCLUSIVE, 0
    f = tau[fin]
    m = np.median(f)
    dev = np.abs(f - m)
    d = np.median(dev)
    if d == 0:
        q1, q3 = np.percentile(f, [25, 75], method="linear")
        d = (q3 - q1) * 0.5
    if d == 0:
        d = (f.max() - f.min()) / f.size
    B = ~fin
    if d != 0:
        B = B | (fin & (np.abs(np.where(fin, tau, 0) - m) > kappa * d))
    bits = sum(1 << i for i in range(R) if B[i])
    return (oracle.ATTRIBUTED if bits else oracle.AGREE), bits


def test_statistical_vote_matches_numpy():
    rng = np.random.default_rng(17)
    k = oracle.KAPPA_DEFAULT
    for R in [2, 3, 4, 5, 7, 8, 16, 33, 64]:
        tau = np.exp(rng.standard_normal((300, R)) * 0.02).astype(np.float32)
        tau[::7, 0] *= 1.3
        tau[::11, -1] = tau[::11, 0]                    # ties
        tau[5, :R // 2 + 1] = 1.0                      # majority equal
        tau[13, 1] = np.nan
        tau[17, 0] = np.inf
        st, bm, mj = oracle.vote_statistical(tau, k, replica_axis=1)
        for u in range(tau.shape[0]):
            ws, wb = _stat_numpy(tau[u], k)
            assert (int(st[u]), int(bm[u])) == (ws, wb), (R, u)
            if ws != oracle.INCONCLUSIVE:
                fin = np.isfinite(tau[u].astype(np.float64))
                srt = np.sort(tau[u][fin])
                assert tau[u][mj[u]] == srt[(fin.sum() - 1) // 2]


@pytest.mark.parametrize("R", [65, 128, 192, 256])
def test_statistical_vote_wide_groups_match_numpy(R):
    rng = np.random.default_rng(37 + R)
    k = oracle.KAPPA_DEFAULT
    tau = np.exp(rng.standard_normal((80, R)) * 0.02)
    tau[::5, 70 % R] *= 1.4                            # a slow replica in a high word
    tau[::7, R - 1] *= 0.6
    tau[3, : R // 2 + 1] = 1.0                         # majority equal: MAD 0, IQR path
    tau[9] = 1.0
    tau[9, R - 2] = 1.5                                # all equal but one: range path
    tau[11, 64 % R] = np.nan
    tau[12, : R // 2] = np.inf                         # finite values a majority only for odd R
    for dt in (np.float32, np.float64):
        t = tau.astype(dt)
        st, bm, mj = oracle.vote_statistical(t, k, replica_axis=1)
        for u in range(t.shape[0]):
            ws, wb = _stat_numpy(t[u], k)
            assert (int(st[u]), _row_int(bm, u, R)) == (ws, wb), (R, dt, u)
            if ws != oracle.INCONCLUSIVE:
                x = t[u].astype(np.float64)
                fin = np.isfinite(x)
                order = [r for r in np.argsort(np.where(fin, x, np.inf), kind="stable") if fin[r]]
                assert mj[u] == order[(fin.sum() - 1) // 2]


def test_statistical_nonfinite_majority_is_inconclusive():
    ev = np.array([[1.0, np.nan, np.inf, 1.0]], np.float64)
    st, bm, mj = oracle.vote_statistical(ev, replica_axis=1)
    assert int(st[0]) == oracle.INCONCLUSIVE and int(bm[0]) == 0 and int(mj[0]) == -1


# ---------------------------------------------------------------------------
# localize and confirm: brute force
# ---------------------------------------------------------------------------
def test_localize_brute_force_and_truncation():
    rng = np.random.default_rng(19)
    R, U = 6, 500
    ev = rng.integers(0, 2, size=(U, R)).astype(np.uint64)
    ev[rng.random(U) < 0.6] = 0
    st, bm, mj = oracle.vote_exact(ev, replica_axis=1)
    want = [(u, r) for u in range(U) for r in range(R) if (int(bm[u]) >> r) & 1]
    und = [u for u in range(U) if st[u] == oracle.INCONCLUSIVE]
    loc = oracle.localize(st, bm, mj, R)
    assert list(zip(loc["unit"].tolist(), loc["replica"].tolist())) == want
    assert loc["undecided"].tolist() == und
    assert loc["counts"].tolist() == [len(want), len(und), int((bm != 0).sum())]
    assert all(loc["majority"][i] == mj[u] for i, (u, _) in enumerate(want))
    cut = oracle.localize(st, bm, mj, R, out_cap=3, und_cap=2)
    assert cut["counts"].tolist() == loc["counts"].tolist()
    assert list(zip(cut["unit"].tolist(), cut["replica"].tolist())) == want[:3]
    assert cut["undecided"].tolist() == und[:2]


@pytest.mark.parametrize("R", [65, 192, 256])
def test_localize_wide_groups_brute_force(R):
    rng = np.random.default_rng(41 + R)
    U = 300
    ev = rng.integers(0, 2, size=(U, R)).astype(np.uint64)
    ev[rng.random(U) < 0.6] = 0
    ev[::9, R - 3:] = 5                                  # outliers in the last word
    st, bm, mj = oracle.vote_exact(ev, replica_axis=1)
    want = [(u, r) for u in range(U) for r in range(R) if (_row_int(bm, u, R) >> r) & 1]
    und = [u for u in range(U) if st[u] == oracle.INCONCLUSIVE]
    assert any(r >= 64 for _, r in want)
    loc = oracle.localize(st, bm, mj, R)
    assert list(zip(loc["unit"].tolist(), loc["replica"].tolist())) == want
    assert loc["undecided"].tolist() == und
    n_att = sum(1 for u in range(U) if _row_int(bm, u, R) != 0)
    assert loc["counts"].tolist() == [len(want), len(und), n_att]
    cut = oracle.localize(st, bm, mj, R, out_cap=5, und_cap=1)
    assert list(zip(cut["unit"].tolist(), cut["replica"].tolist())) == want[:5]
    assert cut["counts"].tolist() == loc["counts"].tolist()


@pytest.mark.parametrize("T,W", [(64, 16), (10, 16), (40, 5), (1, 16)])
def test_confirm_brute_force(T, W):
    rng = np.random.default_rng(T * 100 + W)
    R, G = 5, 7
    fpb = np.zeros((T, G), np.uint64)
    tmb = np.zeros((T, G), np.uint64)
    for t in range(T):
        for g in range(G):
            for r in range(R):
                if rng.random() < 0.02:
                    fpb[t, g] |= np.uint64(1 << r)
                if rng.random() < (0.7 if (r + g) % 9 == 0 else 0.05):
                    tmb[t, g] |= np.uint64(1 << r)
    out = oracle.confirm(fpb, tmb, R, W)
    Wt = min(W, T)
    for r in range(R):
        for g in range(G):
            rank = r * G + g
            slow = np.array([(int(tmb[t, g]) >> r) & 1 for t in range(T)])
            div = np.array([(int(fpb[t, g]) >> r) & 1 for t in range(T)])
            cs = np.concatenate([[0], np.cumsum(slow)])
            win = cs[Wt:] - cs[:-Wt] if Wt else np.array([])
            hit = np.nonzero(2 * win > Wt)[0]
            assert out["max_window"][rank] == (win.max() if win.size else 0)
            assert out["first_window"][rank] == (hit[0] if hit.size else -1)
            assert out["slow_count"][rank] == slow.sum()
            assert out["div_count"][rank] == div.sum()
            assert out["first_div"][rank] == (np.nonzero(div)[0][0] if div.any() else -1)
            consec = bool(np.any(slow[1:] & slow[:-1])) if T > 1 else False
            want = (1 if hit.size else 0) | (2 if div.any() else 0) | (4 if consec else 0)
            assert out["flags"][rank] == want


def test_confirm_needs_more_than_half_of_a_window():
    # reading: a confirmed straggler is flagged in a strict majority of some
    # window (the strict-majority principle applied over time)
    T, W = 16, 16
    for flagged, want in ((8, 0), (9, 1)):
        tmb = np.zeros((T, 1), np.uint64)
        tmb[:flagged, 0] = 1
        out = oracle.confirm(np.zeros((T, 1), np.uint64), tmb, 2, W)
        assert int(out["flags"][0] & 1) == want and out["max_window"][0] == flagged
        assert out["flags"][1] == 0 and out["max_window"][1] == 0   # replica 1 never flagged


def test_empty_tensor_is_one_empty_chunk():
    # reading: an empty tensor keeps one chunk so its dtype and shape are compared
    assert oracle.num_chunks([(oracle.F32, (0,))], 1024) == 1
    assert oracle.num_chunks([(oracle.F32, (0,)), (oracle.BF16, (5, 0, 3))], 1024) == 2
    e = np.zeros(0, np.uint8)
    r1 = oracle.signature([[e], [e]], [(oracle.F32, (0,))], 1024)
    r2 = oracle.signature([[e], [e]], [(oracle.F32, (0, 4))], 1024)
    assert r1["sig"].shape == (2, 1) and r1["sig"][0, 0] != r2["sig"][0, 0]
    assert r1["n_elems"][0, 0] == 0


def test_confirm_rank_layout_matches_paper_peer_groups():
    # Sec. 4 example: 4-way DP x 2-way TP, rank = 2 d + t
    for ln in _lines("peer_groups_4x2.txt"):
        g, ranks = [s.strip() for s in ln.split("|")]
        g = int(g)
        ranks = [int(x) for x in ranks.split()]
        for r, want_rank in enumerate(ranks):
            fpb = np.zeros((1, 2), np.uint64)
            fpb[0, g] = np.uint64(1 << r)
            out = oracle.confirm(fpb, np.zeros((1, 2), np.uint64), 4, 16)
            assert np.nonzero(out["flags"] & 2)[0].tolist() == [want_rank]


# ---------------------------------------------------------------------------
# ground truth on the small configs (3-step protocol: clean, fault, clean)
# ---------------------------------------------------------------------------
def _expected(w):
    """Expected (replica, chunk) outliers and undecided chunks from planted faults."""
    bases = np.cumsum([0] + [oracle.num_chunks([m], w.chunk_bytes) for m in w.metas])
    out = set()
    for f in w.faults:
        for b in range(f.byte_offset, f.byte_offset + f.byte_len):
            out.add((f.replica, int(bases[f.tensor]) + b // w.chunk_bytes))
    und = set()
    for f in w.split_faults:
        und.add(int(bases[f.tensor]) + f.byte_offset // w.chunk_bytes)
    return out, und


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_small_configs_three_step_protocol(k):
    w = workloads.make(k, device="cpu", scale="small")
    faulty = [[workloads.host_bytes(t) for t in rep] for rep in w.replicas]
    clean = [[a.copy() for a in faulty[0]] for _ in range(w.R)]
    if any(f.replica == 0 for f in w.faults + w.split_faults):
        clean_src = 1 if all(f.replica != 1 for f in w.faults + w.split_faults) else None
        assert clean_src is not None
        clean = [[a.copy() for a in faulty[clean_src]] for _ in range(w.R)]
    want_out, want_und = _expected(w)
    for step, reps in (("clean", clean), ("fault", faulty), ("clean-again", clean)):
        rec = oracle.signature(reps, w.metas, w.chunk_bytes)
        st, bm, mj = oracle.vote_exact(rec["sig"])
        loc = oracle.localize(st, bm, mj, w.R)
        got = set(zip(loc["replica"].tolist(), loc["unit"].tolist()))
        if step == "fault":
            assert got == want_out
            assert set(loc["undecided"].tolist()) == want_und
        else:
            assert not got and loc["counts"].tolist() == [0, 0, 0]
