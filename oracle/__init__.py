"""C3 oracle: the plain CPU implementation that the HIP path is checked against.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It shares no code with
the HIP implementation and never imports it.

The arithmetic lives in ``c3_oracle.c`` (plain C, single-threaded, fp64 for
floating point); this module marshals numpy arrays into it with ctypes.  Each
function cites the paper passage it follows:

* ``signature``        Sec. 5.2 (comparable evidence H_w over dtype, shape,
                       bytes), read per chunk as C3SIG-1; numerical summary
                       (NaN/Inf counts, absmax, compensated sum and sum of
                       squares of the finite elements).
* ``tensor_signature`` Sec. 5.2 at the paper's own granularity: one value per
                       tensor, combined from its chunk signatures.
* ``vote_exact``       Sec. 5.3, Algorithm 1 Exact branch.
* ``vote_bytes``       the plain definition of the exact result: equality of
                       raw chunk bytes instead of equality of signatures.
* ``vote_statistical`` Sec. 5.4, Algorithm 1 Statistical branch.
* ``localize``         Sec. 5.1: bitmap bit i names peer i; the result keeps
                       which peers disagree.

Peer groups hold up to ``MAX_PEERS`` replicas (the paper's Table 2 lists
data-parallel peer degrees up to 192).  A unit's outlier bitmap is then
ceil(R / 64) 64-bit words, bit b of word w naming replica 64 w + b: the vote
functions return bitmaps of shape [U] for R <= 64 and [U, ceil(R / 64)] above.
* ``confirm``          Sec. 10 protocol: stragglers are confirmed across
                       repeated timing rounds.
* ``adamw``            Sec. 9 optimizer boundary: the replayed AdamW step on a
                       rotating slice and the check built on it (module
                       ``oracle.adamw``).

Parity: the paper fixes no hash construction, so the bits of C3SIG-1 are
this implementation's definition.  They are pinned by a restatement of that
definition in Python integers and by frozen known-answer vectors (see the
header of ``c3_oracle.c``).
"""
import ctypes
import os

import numpy as np

from . import build as _build

F32, BF16, F16, RAW = 0, 1, 2, 3
AGREE, ATTRIBUTED, INCONCLUSIVE = 0, 1, 2
EV_U64, EV_U32, EV_F32, EV_F64 = 0, 1, 2, 3
KAPPA_DEFAULT = 3.5 / 0.6745          # Iglewicz-Hoaglin modified z > 3.5
MAX_PEERS = 256
ELEM_SIZE = {F32: 4, BF16: 2, F16: 2, RAW: 1}

_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _lib = ctypes.CDLL(_build.LIB)
        u64, i64, u32, i32, vp, dbl = (ctypes.c_uint64, ctypes.c_int64, ctypes.c_uint32,
                                       ctypes.c_int32, ctypes.c_void_p, ctypes.c_double)
        _lib.c3o_splitmix64_next.restype = u64
        _lib.c3o_splitmix64_next.argtypes = [ctypes.POINTER(u64)]
        _lib.c3o_fmix64.restype = u64
        _lib.c3o_fmix64.argtypes = [u64]
        _lib.c3o_keys.argtypes = [vp]
        _lib.c3o_nh.argtypes = [vp, u64, vp, vp, vp]
        _lib.c3o_finalize.restype = u64
        _lib.c3o_finalize.argtypes = [ctypes.c_int, ctypes.c_int, vp, u64, u64, u64, u64]
        _lib.c3o_chunk_signature.argtypes = [vp, u64, ctypes.c_int, ctypes.c_int, vp, u64, vp,
                                             vp, vp, vp, vp, vp, vp, vp]
        _lib.c3o_num_chunks.restype = i64
        _lib.c3o_num_chunks.argtypes = [vp, vp, vp, ctypes.c_int, u64]
        _lib.c3o_signature.argtypes = [vp, vp, vp, vp, ctypes.c_int, ctypes.c_int, u64,
                                       vp, vp, vp, vp, vp, vp, vp, vp, vp]
        _lib.c3o_tensor_signature.argtypes = [vp, vp, ctypes.c_int, i64, ctypes.c_int, vp]
        _lib.c3o_vote_exact.argtypes = [vp, ctypes.c_int, i64, i64, ctypes.c_int, i64,
                                        vp, vp, vp]
        _lib.c3o_vote_bytes.argtypes = [vp, vp, ctypes.c_int, i64, vp, vp, vp]
        _lib.c3o_vote_statistical.argtypes = [vp, ctypes.c_int, i64, i64, ctypes.c_int, i64,
                                              dbl, vp, vp, vp]
        _lib.c3o_localize.argtypes = [vp, vp, vp, ctypes.c_int, i64, vp, vp, vp, i64,
                                      vp, i64, vp]
        _lib.c3o_confirm.argtypes = [vp, vp, ctypes.c_int, i64, i64, ctypes.c_int,
                                     vp, vp, vp, vp, vp, vp]
        del u32, i32
    return _lib


def _ok(rc):
    if rc != 0:
        raise ValueError(f"oracle call rejected its arguments ({rc})")


def _p(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None and a.size else ctypes.c_void_p(0)


# --------------------------------------------------------------------------
# primitives
# --------------------------------------------------------------------------
def splitmix64_stream(seed: int, n: int) -> np.ndarray:
    """First n SplitMix64 outputs from ``seed`` (Steele, Lea, Flood 2014)."""
    lib = _load()
    st = ctypes.c_uint64(seed)
    return np.array([lib.c3o_splitmix64_next(ctypes.byref(st)) for _ in range(n)], dtype=np.uint64)


def fmix64(x: int) -> int:
    """MurmurHash3's 64-bit finalizer."""
    return int(_load().c3o_fmix64(ctypes.c_uint64(int(x) & (2 ** 64 - 1))))


def keys() -> np.ndarray:
    """C3SIG-1 key table K[0..257] (u32)."""
    k = np.zeros(258, dtype=np.uint32)
    _load().c3o_keys(_p(k))
    return k


def nh(data: np.ndarray):
    """NH fold (A, B) of a chunk's bytes (uint8 array)."""
    data = np.ascontiguousarray(data, dtype=np.uint8)
    k = keys()
    a = np.zeros(1, np.uint64)
    b = np.zeros(1, np.uint64)
    _load().c3o_nh(_p(data), ctypes.c_uint64(data.size), _p(k), _p(a), _p(b))
    return int(a[0]), int(b[0])


def finalize(dtype: int, shape, chunk_in_tensor: int, n: int, A: int, B: int) -> int:
    sh = np.zeros(8, np.int64)
    sh[:len(shape)] = shape
    return int(_load().c3o_finalize(dtype, len(shape), _p(sh), chunk_in_tensor, n, A, B))


def chunk_signature(data: np.ndarray, dtype: int, shape, chunk_in_tensor: int) -> dict:
    """Signature and numerical summary of one chunk (Sec. 5.2, per chunk)."""
    data = np.ascontiguousarray(data, dtype=np.uint8)
    sh = np.zeros(8, np.int64)
    sh[:len(shape)] = shape
    k = keys()
    out_u64 = np.zeros(2, np.uint64)
    out_u32 = np.zeros(2, np.uint32)
    out_f = np.zeros(3, np.float64)
    vp = ctypes.c_void_p
    base64, base32, basef = out_u64.ctypes.data, out_u32.ctypes.data, out_f.ctypes.data
    _load().c3o_chunk_signature(_p(data), ctypes.c_uint64(data.size), dtype, len(shape), _p(sh),
                                ctypes.c_uint64(chunk_in_tensor), _p(k),
                                vp(base64), vp(base64 + 8), vp(base32), vp(base32 + 4),
                                vp(basef), vp(basef + 8), vp(basef + 16))
    return dict(sig=int(out_u64[0]), n_elems=int(out_u64[1]), nan=int(out_u32[0]),
                inf=int(out_u32[1]), absmax=float(out_f[0]), sum=float(out_f[1]),
                sumsq=float(out_f[2]))


# --------------------------------------------------------------------------
# chunk plan and signatures of R replicas
# --------------------------------------------------------------------------
def _metas(metas):
    T = len(metas)
    dt = np.array([m[0] for m in metas], np.int32)
    nd = np.array([len(m[1]) for m in metas], np.int32)
    sh = np.zeros((T, 8), np.int64)
    for i, m in enumerate(metas):
        sh[i, :len(m[1])] = m[1]
    return dt, nd, sh


def num_chunks(metas, chunk_bytes: int) -> int:
    """Chunks over all tensors: ceil(bytes / chunk_bytes) each, at least one."""
    dt, nd, sh = _metas(metas)
    return int(_load().c3o_num_chunks(_p(dt), _p(nd), _p(sh), len(metas), chunk_bytes))


def signature(replicas, metas, chunk_bytes: int) -> dict:
    """Per-(replica, chunk) records of R replicas.

    replicas: list of R lists of T contiguous uint8 numpy arrays (raw bytes).
    metas:    list of T (dtype_code, shape) pairs shared by all replicas.
    Returns a dict of [R, C] arrays: sig, n_elems, nan, inf, absmax, sum, sumsq,
    tensor, chunk.
    """
    R, T = len(replicas), len(metas)
    dt, nd, sh = _metas(metas)
    C = num_chunks(metas, chunk_bytes)
    keep = [np.ascontiguousarray(a, dtype=np.uint8) for rep in replicas for a in rep]
    ptrs = (ctypes.c_void_p * (R * T))(*[a.ctypes.data for a in keep])
    out = dict(sig=np.zeros((R, C), np.uint64), n_elems=np.zeros((R, C), np.uint64),
               nan=np.zeros((R, C), np.uint32), inf=np.zeros((R, C), np.uint32),
               absmax=np.zeros((R, C), np.float64), sum=np.zeros((R, C), np.float64),
               sumsq=np.zeros((R, C), np.float64), tensor=np.zeros((R, C), np.uint32),
               chunk=np.zeros((R, C), np.uint32))
    _load().c3o_signature(ptrs, _p(dt), _p(nd), _p(sh), T, R, ctypes.c_uint64(chunk_bytes),
                          _p(out["sig"]), _p(out["n_elems"]), _p(out["nan"]), _p(out["inf"]),
                          _p(out["absmax"]), _p(out["sum"]), _p(out["sumsq"]),
                          _p(out["tensor"]), _p(out["chunk"]))
    return out


def chunk_views(replicas, metas, chunk_bytes: int):
    """[R][C] list of uint8 views of each chunk (same plan as ``signature``)."""
    views = []
    for rep in replicas:
        row = []
        for a, m in zip(rep, metas):
            a = np.ascontiguousarray(a, dtype=np.uint8)
            nb = a.size
            nc = max(1, -(-nb // chunk_bytes))
            for k in range(nc):
                row.append(a[k * chunk_bytes:min(nb, (k + 1) * chunk_bytes)])
        views.append(row)
    return views


def tensor_signature(rec: dict, T: int) -> np.ndarray:
    """Per-tensor signatures [R, T] from the chunk records of ``signature``."""
    sig = np.ascontiguousarray(rec["sig"], np.uint64)
    tid = np.ascontiguousarray(rec["tensor"], np.uint32)
    R, C = sig.shape
    out = np.zeros((R, T), np.uint64)
    _load().c3o_tensor_signature(_p(sig), _p(tid), R, C, T, _p(out))
    return out


# --------------------------------------------------------------------------
# votes
# --------------------------------------------------------------------------
def bitmap_words(R: int) -> int:
    """64-bit words of one unit's outlier bitmap."""
    return (R + 63) // 64


def _check_group(R: int):
    # Sec. 4: a singleton group provides no comparison, so no vote over it
    if not 2 <= R <= MAX_PEERS:
        raise ValueError(f"R = {R} outside 2..{MAX_PEERS}")


def _new_bitmap(U: int, R: int) -> np.ndarray:
    _check_group(R)
    return np.zeros(U, np.uint64) if R <= 64 else np.zeros((U, bitmap_words(R)), np.uint64)


def bitmap_bits(bitmap: np.ndarray, R: int) -> np.ndarray:
    """[U, R] bool array: replica r is flagged at unit u."""
    b = np.ascontiguousarray(bitmap, np.uint64).reshape(-1, bitmap_words(R))
    r = np.arange(R)
    return ((b[:, r // 64] >> (r % 64).astype(np.uint64)) & np.uint64(1)).astype(bool)
def _ev_kind(ev: np.ndarray) -> int:
    return {np.dtype(np.uint64): EV_U64, np.dtype(np.int64): EV_U64, np.dtype(np.uint32): EV_U32,
            np.dtype(np.int32): EV_U32, np.dtype(np.float32): EV_F32,
            np.dtype(np.float64): EV_F64}[ev.dtype]


def vote_exact(ev: np.ndarray, replica_axis: int = 0):
    """Exact consensus per unit.  ev: 2-D [R, U] (replica_axis=0) or [U, R]."""
    ev = np.ascontiguousarray(ev)
    if replica_axis == 0:
        R, U = ev.shape
        rs, us = ev.strides
    else:
        U, R = ev.shape
        us, rs = ev.strides
    st = np.zeros(U, np.uint8)
    bm = _new_bitmap(U, R)
    mj = np.zeros(U, np.int32)
    _ok(_load().c3o_vote_exact(_p(ev), _ev_kind(ev), rs, us, R, U, _p(st), _p(bm), _p(mj)))
    return st, bm, mj


def vote_bytes(chunks):
    """Byte-equality vote. chunks: [R][U] list of uint8 arrays (equal lengths per unit)."""
    R, U = len(chunks), len(chunks[0])
    keep = [np.ascontiguousarray(c, dtype=np.uint8) for row in chunks for c in row]
    ptrs = (ctypes.c_void_p * (R * U))(*[c.ctypes.data if c.size else 0 for c in keep])
    lens = np.array([c.size for c in chunks[0]], np.uint64)
    st = np.zeros(U, np.uint8)
    bm = _new_bitmap(U, R)
    mj = np.zeros(U, np.int32)
    _ok(_load().c3o_vote_bytes(ptrs, _p(lens), R, U, _p(st), _p(bm), _p(mj)))
    return st, bm, mj


def vote_statistical(ev: np.ndarray, kappa: float = KAPPA_DEFAULT, replica_axis: int = 0):
    """Statistical consensus per unit.  ev: float32/float64 [R, U] or [U, R]."""
    ev = np.ascontiguousarray(ev)
    if replica_axis == 0:
        R, U = ev.shape
        rs, us = ev.strides
    else:
        U, R = ev.shape
        us, rs = ev.strides
    st = np.zeros(U, np.uint8)
    bm = _new_bitmap(U, R)
    mj = np.zeros(U, np.int32)
    _ok(_load().c3o_vote_statistical(_p(ev), _ev_kind(ev), rs, us, R, U, ctypes.c_double(kappa),
                                     _p(st), _p(bm), _p(mj)))
    return st, bm, mj


def localize(status, bitmap, majority_idx, R: int, out_cap=None, und_cap=None):
    """Outlier (unit, replica, majority replica) list and undecided units.
    bitmap: [U] (R <= 64) or [U, ceil(R / 64)] uint64."""
    _check_group(R)
    status = np.ascontiguousarray(status, np.uint8)
    U = status.size
    bitmap = np.ascontiguousarray(bitmap, np.uint64).reshape(U * bitmap_words(R))
    majority_idx = np.ascontiguousarray(majority_idx, np.int32)
    if out_cap is None:
        out_cap = int(sum(bin(int(b)).count("1") for b in bitmap)) if U < 100000 else U * R
    if und_cap is None:
        und_cap = U
    ou = np.zeros(max(out_cap, 1), np.int64)
    orr = np.zeros(max(out_cap, 1), np.int32)
    om = np.zeros(max(out_cap, 1), np.int32)
    und = np.zeros(max(und_cap, 1), np.int64)
    counts = np.zeros(3, np.int64)
    _ok(_load().c3o_localize(_p(status), _p(bitmap), _p(majority_idx), R, U, _p(ou), _p(orr), _p(om),
                             out_cap, _p(und), und_cap, _p(counts)))
    n_o = min(int(counts[0]), out_cap)
    n_u = min(int(counts[1]), und_cap)
    return dict(unit=ou[:n_o], replica=orr[:n_o], majority=om[:n_o], undecided=und[:n_u],
                counts=counts)


def confirm(fp_bitmap, time_bitmap, R: int, W: int = 16):
    """Per-rank temporal confirmation; bitmaps are [T, G] uint64; rank = r*G + g."""
    if not 2 <= R <= 64:
        raise ValueError(f"R = {R} outside 2..64")
    fp_bitmap = np.ascontiguousarray(fp_bitmap, np.uint64)
    time_bitmap = np.ascontiguousarray(time_bitmap, np.uint64)
    T, G = fp_bitmap.shape
    n = R * G
    out = dict(flags=np.zeros(n, np.uint32), first_div=np.zeros(n, np.int32),
               div_count=np.zeros(n, np.uint32), slow_count=np.zeros(n, np.uint32),
               max_window=np.zeros(n, np.uint32), first_window=np.zeros(n, np.int32))
    _ok(_load().c3o_confirm(_p(fp_bitmap), _p(time_bitmap), R, G, T, W,
                            _p(out["flags"]), _p(out["first_div"]), _p(out["div_count"]),
                            _p(out["slow_count"]), _p(out["max_window"]), _p(out["first_window"])))
    return out
