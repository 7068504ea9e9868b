"""Pins of C3SIG-1's exact bits (Sec. 5.2 read per chunk) on the CPU.

Three things are compared, none derived from another:
* ``c3sig1_spec``: the construction restated in Python integers from its
  specification (SplitMix64 keys, NH fold, fmix64 chain, per-tensor combine);
* ``golden/c3sig1_vectors.txt``: known-answer vectors frozen by
  ``golden/make_c3sig1_vectors.py`` from the oracle;
* the oracle itself, recomputed now.
A mistake anywhere in the oracle's chain (a swapped pair of finalizer terms, a
wrong tag, a dropped dim, a wrong key index) separates it from the Python
restatement and from the frozen vectors.
"""
import os

import numpy as np
import pytest

import oracle
import workloads
import c3sig1_spec as spec

GOLD = os.path.join(os.path.dirname(__file__), "golden")
DT = {"F32": oracle.F32, "BF16": oracle.BF16, "F16": oracle.F16, "RAW": oracle.RAW}


def _shape(text):
    return () if text == "scalar" else tuple(int(d) for d in text.split(","))


def _vectors():
    chunks, tensors = [], []
    for ln in open(os.path.join(GOLD, "c3sig1_vectors.txt")):
        if not ln.strip() or ln.startswith("#"):
            continue
        f = [x.strip() for x in ln.split("|")]
        if f[0] == "chunk":
            chunks.append(dict(name=f[1], dtype=DT[f[2]], shape=_shape(f[3]), cb=int(f[4]),
                               seed=int(f[5]), k=int(f[6]), n=int(f[7]), A=int(f[8], 16),
                               B=int(f[9], 16), sig=int(f[10], 16)))
        else:
            assert f[0] == "tensor", ln
            tensors.append(dict(name=f[1], dtype=DT[f[2]], shape=_shape(f[3]), cb=int(f[4]),
                                seed=int(f[5]), C=int(f[6]), tsig=int(f[7], 16)))
    return chunks, tensors


def _tensor_bytes(v):
    return workloads.lcg_bytes(v["seed"], spec.tensor_nbytes(v["dtype"], v["shape"]))


def _chunk_bytes(v):
    data = _tensor_bytes(v)
    return data[v["k"] * v["cb"]:v["k"] * v["cb"] + v["n"]]


def test_lcg_pattern_first_states():
    # x1 = 1013904223 from x0 = 0, x2 = 1664525 x1 + 1013904223 mod 2^32
    x1 = 1013904223
    x2 = (1664525 * x1 + 1013904223) % 2 ** 32
    assert workloads.lcg_bytes(0, 2).tolist() == [x1 >> 24, x2 >> 24]


def test_spec_splitmix64_published_vectors():
    rows = [ln.split() for ln in open(os.path.join(GOLD, "splitmix64_vectors.txt"))
            if ln.strip() and not ln.startswith("#")]
    for seed in {int(r[0]) for r in rows}:
        want = {int(r[1]): int(r[2], 16) for r in rows if int(r[0]) == seed}
        got = spec.splitmix64(seed, max(want) + 1)
        for i, v in want.items():
            assert got[i] == v, (seed, i)


def test_spec_fmix64_is_invertible_and_fixes_zero():
    inv1 = pow(0xFF51AFD7ED558CCD, -1, 1 << 64)
    inv2 = pow(0xC4CEB9FE1A85EC53, -1, 1 << 64)
    rng = np.random.default_rng(5)
    for x in [0, 1, spec.M64] + [int(v) for v in rng.integers(0, 2 ** 63, 50)]:
        h = spec.fmix64(x)
        h ^= h >> 33
        h = (h * inv2) & spec.M64
        h ^= h >> 33
        h = (h * inv1) & spec.M64
        h ^= h >> 33
        assert h == x
    assert spec.fmix64(0) == 0


def test_vectors_cover_the_cases_that_matter():
    chunks, tensors = _vectors()
    assert {v["dtype"] for v in chunks} == set(DT.values())
    ns = [v["n"] for v in chunks]
    assert 0 in ns and 1 in ns                                   # empty and one byte
    assert any(n % 16 for n in ns)                               # ragged word padding
    assert any(n > 1024 for n in ns)                             # beta != 0 (past one key period)
    assert any(v["k"] > 0 for v in chunks)                       # chunk index enters
    assert any(v["n"] < v["cb"] and v["k"] > 0 for v in chunks)  # partial last chunk
    assert any(len(v["shape"]) == 0 for v in chunks)             # scalar
    assert any(len(v["shape"]) >= 3 for v in chunks)             # multi-dim shapes
    assert any(len(v["shape"]) == 8 for v in chunks)
    assert any(v["cb"] >= 32768 for v in chunks)                 # many GPU tiles per chunk
    assert any(t["C"] > 2 for t in tensors) and len(tensors) >= 15


def test_vectors_equal_the_bigint_restatement():
    chunks, tensors = _vectors()
    for v in chunks:
        A, B, sig = spec.chunk_signature(_chunk_bytes(v).tobytes(), v["dtype"], v["shape"], v["k"])
        assert (A, B, sig) == (v["A"], v["B"], v["sig"]), v["name"]
    for t in tensors:
        data = _tensor_bytes(t).tobytes()
        assert len(spec.chunks(data, t["cb"])) == t["C"], t["name"]
        assert spec.tensor_signature(data, t["dtype"], t["shape"], t["cb"]) == t["tsig"], t["name"]


def test_oracle_reproduces_the_vectors():
    chunks, tensors = _vectors()
    for v in chunks:
        c = _chunk_bytes(v)
        assert oracle.nh(c) == (v["A"], v["B"]), v["name"]
        assert oracle.chunk_signature(c, v["dtype"], list(v["shape"]), v["k"])["sig"] == v["sig"]
        assert oracle.finalize(v["dtype"], list(v["shape"]), v["k"], v["n"], v["A"], v["B"]) == \
            v["sig"], v["name"]
    for t in tensors:
        meta = [(t["dtype"], t["shape"])]
        rec = oracle.signature([[_tensor_bytes(t)]], meta, t["cb"])
        assert rec["sig"].shape[1] == t["C"]
        assert int(oracle.tensor_signature(rec, 1)[0, 0]) == t["tsig"], t["name"]


@pytest.mark.parametrize("seed", range(6))
def test_oracle_equals_bigint_on_random_plans(seed):
    """Whole plans of several tensors (random dtypes, ranks 0-8, dims, chunk
    sizes, bytes): every chunk signature and every tensor signature."""
    rng = np.random.default_rng(1000 + seed)
    T = int(rng.integers(1, 6))
    metas, datas = [], []
    for _ in range(T):
        dt = int(rng.integers(0, 4))
        nd = int(rng.integers(0, 9))
        shape = tuple(int(rng.integers(1, 4)) for _ in range(nd))
        if nd:
            shape = shape[:-1] + (int(rng.integers(0, 900)),)
        nb = spec.tensor_nbytes(dt, shape)
        metas.append((dt, shape))
        datas.append(rng.integers(0, 256, nb, dtype=np.uint8))
    cb = 1024 * int(rng.integers(1, 5))
    rec = oracle.signature([datas], metas, cb)
    g = 0
    for t, ((dt, shape), d) in enumerate(zip(metas, datas)):
        s = 0
        for k, c in enumerate(spec.chunks(d.tobytes(), cb)):
            sig = spec.chunk_signature(c, dt, shape, k)[2]
            assert int(rec["sig"][0, g]) == sig, (seed, t, k)
            assert int(rec["tensor"][0, g]) == t and int(rec["chunk"][0, g]) == k
            s = (s + sig) & spec.M64
            g += 1
        assert int(oracle.tensor_signature(rec, T)[0, t]) == spec.fmix64(spec.TAG_TENSOR ^ s)
    assert g == rec["sig"].shape[1]
