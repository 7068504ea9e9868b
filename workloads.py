"""Seeded synthetic workloads for the C3 hot path.

This module only makes input bytes and records where faults were planted.  It
holds none of the method's arithmetic (no hashing, voting or statistics): the
HIP path and the oracle both consume the bytes it produces, and tests turn
the planted fault positions into expected chunk ids with the oracle's chunk
plan.

Recipe (values stand in for LLM pre-training state; the paper's own workload
is a deterministic three-block Transformer and names no public dataset):

* values: ``torch.randn`` from a ``torch.Generator`` on the target device,
  seeded with the config number, scaled by sigma, then rounded to the dtype;
* faults: positions and bit patterns from ``numpy.random.Generator(PCG64(100 +
  k))``, applied through integer views so NaN payloads survive;
* replicas: R copies of one clean replica, faults applied afterwards.

Configs (k = 1..6), ``scale="full"`` is the benchmark size, ``"small"`` keeps
the structure (dtypes, fault kinds, ragged tails, several chunks per tensor)
at a size the oracle finishes in well under a second.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

F32, BF16, F16, RAW = 0, 1, 2, 3
TORCH_DTYPE = {F32: torch.float32, BF16: torch.bfloat16, F16: torch.float16, RAW: torch.uint8}
INT_VIEW = {F32: torch.int32, BF16: torch.int16, F16: torch.int16, RAW: torch.uint8}
ELEM_SIZE = {F32: 4, BF16: 2, F16: 2, RAW: 1}
KIB, MIB = 1024, 1024 * 1024


@dataclass
class Fault:
    """One planted change: replica, tensor index, first byte, byte length, kind."""
    replica: int
    tensor: int
    byte_offset: int
    byte_len: int
    kind: str


@dataclass
class ReplicaWorkload:
    name: str
    R: int
    metas: list                      # [(dtype_code, shape tuple)] per tensor
    chunk_bytes: int
    replicas: list                   # R lists of T contiguous device tensors
    faults: list = field(default_factory=list)
    # chunk-level groups the faults were designed to create:
    # "split" faults (same change on several replicas, no strict majority)
    split_faults: list = field(default_factory=list)

    @property
    def bytes_per_replica(self) -> int:
        return sum(int(np.prod(s, dtype=np.int64)) * ELEM_SIZE[d] for d, s in self.metas)

    @property
    def total_bytes(self) -> int:
        return self.R * self.bytes_per_replica


@dataclass
class TimingWorkload:
    name: str
    R: int
    G: int
    T: int
    fingerprints: torch.Tensor       # [T, G, R] int64 (raw 64-bit patterns)
    times: torch.Tensor              # [T, G, R] float32 seconds
    divergent: dict                  # rank -> first divergent iteration
    stragglers: list                 # ranks slowed by the factor at every iteration
    slow_factor: float = 1.3

    @property
    def total_bytes(self) -> int:
        return self.T * self.G * self.R * (8 + 4)


def _randn(shape, sigma, dtype_code, gen, device):
    x = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    x.mul_(sigma)
    return x.to(TORCH_DTYPE[dtype_code])


def _clean_replica(metas, sigmas, seed, device, absolute=None):
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    out = []
    for i, ((d, shape), s) in enumerate(zip(metas, sigmas)):
        t = _randn(shape, s, d, gen, device)
        if absolute is not None and absolute[i]:
            t.abs_()
        out.append(t.contiguous())
    return out


def _replicate(clean, R):
    reps = [clean]
    for _ in range(R - 1):
        reps.append([t.clone() for t in clean])
    return reps


def _flat_int(t: torch.Tensor, d: int) -> torch.Tensor:
    return t.view(-1).view(INT_VIEW[d])


def _xor_bit(t: torch.Tensor, d: int, elem: int, bit: int):
    v = _flat_int(t, d)
    width = 8 * ELEM_SIZE[d]
    mask = 1 << bit
    if mask >= 1 << (width - 1):
        mask -= 1 << width          # two's complement for the sign bit
    v[elem] ^= mask


def _set_bits(t: torch.Tensor, d: int, elem: int, pattern: int):
    v = _flat_int(t, d)
    width = 8 * ELEM_SIZE[d]
    if pattern >= 1 << (width - 1):
        pattern -= 1 << width
    v[elem] = pattern


# --------------------------------------------------------------------------
# config 1: R=3 fp32 [1,048,576] ~N(0,1), chunk 4096 elements, one bit flip
# --------------------------------------------------------------------------
def config1(device="cuda", scale="full") -> ReplicaWorkload:
    n = 1_048_576 if scale == "full" else 4096 * 8 + 100
    metas = [(F32, (n,))]
    rng = np.random.Generator(np.random.PCG64(101))
    reps = _replicate(_clean_replica(metas, [1.0], 1, device), 3)
    elem = int(rng.integers(0, n))
    bit = int(rng.integers(0, 32))
    _xor_bit(reps[2][0], F32, elem, bit)
    faults = [Fault(2, 0, elem * 4, 4, f"bitflip{bit}")]
    return ReplicaWorkload("r3_f32_1m_chunk4096el", 3, metas, 4096 * 4, reps, faults)


# --------------------------------------------------------------------------
# config 2: R=4 Llama-7B layer gradients bf16 ~N(0,1e-3), chunk 64K elements;
# a 2-vs-2 split on one chunk (replicas 2 and 3 share one change) and one
# exponent-bit flip on one replica in another chunk
# --------------------------------------------------------------------------
def _llama_layer(h, f):
    return [(BF16, (h, h))] * 4 + [(BF16, (f, h))] * 2 + [(BF16, (h, f))]


def config2(device="cuda", scale="full") -> ReplicaWorkload:
    metas = _llama_layer(4096, 11008) if scale == "full" else _llama_layer(512, 1376)
    chunk_bytes = 65536 * 2
    R = 4
    rng = np.random.Generator(np.random.PCG64(102))
    reps = _replicate(_clean_replica(metas, [1e-3] * len(metas), 2, device), R)
    sizes = [int(np.prod(s)) for _, s in metas]
    # split chunk X: same element, same bit, on replicas 2 and 3
    tx = int(rng.integers(0, len(metas)))
    ex = int(rng.integers(0, sizes[tx]))
    bx = int(rng.integers(0, 16))
    for r in (2, 3):
        _xor_bit(reps[r][tx], BF16, ex, bx)
    # exponent flip on one replica in a different chunk Y
    rf = int(rng.integers(0, R))
    while True:
        ty = int(rng.integers(0, len(metas)))
        ey = int(rng.integers(0, sizes[ty]))
        if ty != tx or (ey * 2) // chunk_bytes != (ex * 2) // chunk_bytes:
            break
    by = int(rng.integers(7, 15))
    _xor_bit(reps[rf][ty], BF16, ey, by)
    faults = [Fault(rf, ty, ey * 2, 2, f"bitflip{by}")]
    split = [Fault(2, tx, ex * 2, 2, f"bitflip{bx}"), Fault(3, tx, ex * 2, 2, f"bitflip{bx}")]
    return ReplicaWorkload("r4_llama7b_layer_grads_bf16_chunk64kel", R, metas, chunk_bytes, reps,
                           faults, split)


# --------------------------------------------------------------------------
# config 3: R=8 1B bf16 parameters ~N(0,0.02) in layer-shaped tensors,
# chunk 1 MiB; one seeded replica gets 16 bit flips in bits 0-14, one NaN
# (0x7FC0) and one zeroed 4 KiB-aligned block
# --------------------------------------------------------------------------
def _model_1b(layers, h, f):
    metas = []
    for _ in range(layers):
        metas += [(BF16, (h, h))] * 4 + [(BF16, (f, h))] * 2 + [(BF16, (h, f))]
        metas += [(BF16, (h,))] * 2
    return metas


def config3(device="cuda", scale="full") -> ReplicaWorkload:
    if scale == "full":
        metas = _model_1b(16, 2048, 8192)       # 1,073,807,360 elements
    else:
        metas = _model_1b(2, 512, 2048) + [(BF16, (2047,))]
    R = 8
    rng = np.random.Generator(np.random.PCG64(103))
    reps = _replicate(_clean_replica(metas, [0.02] * len(metas), 3, device), R)
    sizes = [int(np.prod(s)) for _, s in metas]
    cum = np.cumsum([0] + sizes)
    rf = int(rng.integers(0, R))
    faults = []

    def pick():
        g = int(rng.integers(0, cum[-1]))
        t = int(np.searchsorted(cum, g, side="right") - 1)
        return t, g - int(cum[t])

    for _ in range(16):
        t, e = pick()
        b = int(rng.integers(0, 15))
        _xor_bit(reps[rf][t], BF16, e, b)
        faults.append(Fault(rf, t, 2 * e, 2, f"bitflip{b}"))
    t, e = pick()
    _set_bits(reps[rf][t], BF16, e, 0x7FC0)
    faults.append(Fault(rf, t, 2 * e, 2, "nan"))
    # zeroed 4 KiB block, aligned to 4 KiB within a tensor of at least 4 KiB
    while True:
        t, e = pick()
        if sizes[t] * 2 >= 4096:
            break
    blk = (2 * e // 4096) * 4096
    blk = min(blk, (sizes[t] * 2 // 4096 - 1) * 4096)
    _flat_int(reps[rf][t], BF16)[blk // 2: blk // 2 + 2048] = 0
    faults.append(Fault(rf, t, blk, 4096, "zero4k"))
    return ReplicaWorkload("r8_1b_bf16_params_chunk1mib", R, metas, MIB, reps, faults)


# --------------------------------------------------------------------------
# config 4: checkpoint certification, R=3 fp32 Adam shard of 2e9 params
# (param ~N(0,0.02), exp_avg ~N(0,1e-4), exp_avg_sq ~|N(0,1e-8)|), chunk 4 MiB;
# 8 sign flips and one +Inf in exp_avg_sq of one replica
# --------------------------------------------------------------------------
def config4(device="cuda", scale="full") -> ReplicaWorkload:
    n = 2_000_000_000 if scale == "full" else 2_500_003
    metas = [(F32, (n,))] * 3
    R = 3
    rng = np.random.Generator(np.random.PCG64(104))
    clean = _clean_replica(metas, [0.02, 1e-4, 1e-8], 4, device, absolute=[False, False, True])
    reps = _replicate(clean, R)
    rf = int(rng.integers(0, R))
    faults = []
    for _ in range(8):
        e = int(rng.integers(0, n))
        _xor_bit(reps[rf][2], F32, e, 31)
        faults.append(Fault(rf, 2, 4 * e, 4, "signflip"))
    e = int(rng.integers(0, n))
    _set_bits(reps[rf][2], F32, e, 0x7F800000)
    faults.append(Fault(rf, 2, 4 * e, 4, "inf"))
    return ReplicaWorkload("r3_adam_shard_2b_f32_chunk4mib", R, metas, 4 * MIB, reps, faults)


# --------------------------------------------------------------------------
# config 5: 32,768 ranks = 4096 groups of 8, 1024 iterations; record = 64-bit
# collective fingerprint + fp32 step time ~LogNormal(ln 1 s, 0.02);
# 3 divergent-fingerprint ranks (from a seeded iteration on) and 5 stragglers
# at 1.3x; rank = r * G + g (row-major, data-parallel index major)
# --------------------------------------------------------------------------
def config5(device="cuda", scale="full") -> TimingWorkload:
    T, G, R = (1024, 4096, 8) if scale == "full" else (64, 64, 8)
    rng = np.random.Generator(np.random.PCG64(105))
    gen = torch.Generator(device=device)
    gen.manual_seed(5)
    lo, hi = -(2 ** 63), 2 ** 63 - 1
    healthy = torch.randint(lo, hi, (T, G, 1), generator=gen, device=device, dtype=torch.int64)
    fp = healthy.expand(T, G, R).contiguous()
    tau = torch.randn((T, G, R), generator=gen, device=device, dtype=torch.float32)
    tau.mul_(0.02).exp_()
    ranks = rng.choice(R * G, size=8, replace=False)
    divergent, stragglers = {}, []
    for rank in ranks[:3]:
        rank = int(rank)
        r, g = divmod(rank, G)
        t0 = int(rng.integers(0, T))
        x = int(rng.integers(1, 2 ** 62)) * (1 if rng.integers(0, 2) else -1)
        fp[t0:, g, r] ^= x
        divergent[rank] = t0
    for rank in ranks[3:]:
        rank = int(rank)
        r, g = divmod(rank, G)
        tau[:, g, r] *= 1.3
        stragglers.append(rank)
    return TimingWorkload("ranks32768_g8_iters1024_fp64_time_f32" if scale == "full"
                          else "ranks512_g8_iters64", R, G, T, fp, tau, divergent, stragglers)


# --------------------------------------------------------------------------
# config 6: optimizer-boundary check, R=8 data-parallel replicas of an AdamW
# state of 134,217,728 fp32 parameters (param ~N(0,0.02), grad ~N(0,1e-3),
# exp_avg ~N(0,1e-4), exp_avg_sq ~|N(0,1e-6)|); 64K-element rotating slices;
# lr 3e-4, betas (0.9, 0.95), eps 1e-8, weight decay 0.1, step 1000.
# Faults, all in slice s1 except the last: an exponent-bit flip in one
# replica's gradient, a sign flip in another replica's exp_avg_sq (the
# replayed square root turns it into NaN) and, in slice s2, a low mantissa
# bit of a third replica's parameter.  The small scale keeps a ragged last
# slice.
# --------------------------------------------------------------------------
@dataclass
class OptimizerWorkload:
    name: str
    R: int
    numel: int
    state: list                      # [4][R] device fp32 tensors: param, grad, exp_avg, exp_avg_sq
    hparams: dict
    faults: list
    fault_slices: list               # slice indices (k) that hold the planted faults
    slice_elems: int = 65536

    @property
    def bytes_per_check(self) -> int:
        """Bytes the replay reads and writes per check (16 in, 12 out per element)."""
        return self.R * min(self.slice_elems, self.numel) * 28


OPT_TENSORS = ("param", "grad", "exp_avg", "exp_avg_sq")


def config6(device="cuda", scale="full") -> OptimizerWorkload:
    S = 65536
    numel = 134_217_728 if scale == "full" else 3 * S + 1000
    R = 8
    rng = np.random.Generator(np.random.PCG64(106))
    metas = [(F32, (numel,))] * 4
    clean = _clean_replica(metas, [0.02, 1e-3, 1e-4, 1e-6], 6, device,
                           absolute=[False, False, False, True])
    reps = _replicate(clean, R)
    n_slices = -(-numel // S)
    s1 = int(rng.integers(0, n_slices))
    s2 = (s1 + 1 + int(rng.integers(0, n_slices - 1))) % n_slices
    ra, rb, rc = (int(x) for x in rng.choice(R, size=3, replace=False))

    def elem_in(slice_k):
        lo = slice_k * S
        return lo + int(rng.integers(0, min(S, numel - lo)))

    e1, e2, e3 = elem_in(s1), elem_in(s1), elem_in(s2)
    b1 = int(rng.integers(23, 30))
    _xor_bit(reps[ra][1], F32, e1, b1)
    _xor_bit(reps[rb][3], F32, e2, 31)
    b3 = int(rng.integers(0, 4))
    _xor_bit(reps[rc][0], F32, e3, b3)
    faults = [Fault(ra, 1, 4 * e1, 4, f"bitflip{b1}"), Fault(rb, 3, 4 * e2, 4, "signflip"),
              Fault(rc, 0, 4 * e3, 4, f"bitflip{b3}")]
    state = [[reps[r][t] for r in range(R)] for t in range(4)]
    hp = dict(lr=3e-4, betas=(0.9, 0.95), eps=1e-8, weight_decay=0.1, step=1000)
    name = "r8_adamw_134m_fp32_slice64kel" if scale == "full" else "r8_adamw_small_ragged"
    return OptimizerWorkload(name, R, numel, state, hp, faults, [s1, s1, s2], S)


CONFIGS = {1: config1, 2: config2, 3: config3, 4: config4, 5: config5, 6: config6}


# --------------------------------------------------------------------------
# wide peer groups (the vote over gathered tables of 33 to 256 peers, Table 2's
# data-parallel degrees): U units x R peers, unit-major.  Step times
# ~LogNormal(ln 1 s, 0.02) in fp32, with a 1.5x slow peer in every 7th unit,
# a tie in every 11th, a majority of equal values (MAD 0: the IQR fallback)
# in every 13th, a NaN in every 23rd; fingerprints: one seeded 64-bit value
# per unit on every peer, one peer changed in every 9th unit and a two-way
# split in every 97th.
# --------------------------------------------------------------------------
def wide_votes(R: int, U: int, device="cuda", seed: int = 8):
    gen = torch.Generator(device=device)
    gen.manual_seed(seed * 1000 + R)
    tau = torch.randn((U, R), generator=gen, device=device, dtype=torch.float32)
    tau.mul_(0.02).exp_()
    tau[::7, 0] *= 1.5
    tau[::11, R // 3] = tau[::11, 1]
    tau[3::13, : R // 2 + 1] = 1.0
    tau[9::23, R - 1] = float("nan")
    lo, hi = -(2 ** 63), 2 ** 63 - 1
    fp = torch.randint(lo, hi, (U, 1), generator=gen, device=device, dtype=torch.int64)
    fp = fp.expand(U, R).contiguous()
    fp[::9, R - 1] ^= 0x5A5A
    fp[::97, : R // 2] ^= 3
    return tau, fp


def make(k: int, device="cuda", scale="full"):
    return CONFIGS[k](device=device, scale=scale)


def host_bytes(t: torch.Tensor) -> np.ndarray:
    """Raw bytes of a tensor as a contiguous host uint8 array."""
    return t.detach().contiguous().view(-1).view(torch.uint8).cpu().numpy()


def lcg_bytes(seed: int, n: int) -> np.ndarray:
    """n pattern bytes for known-answer vectors: the top byte of each state of
    the 32-bit linear congruential generator x <- 1664525 x + 1013904223 mod
    2^32 (the constants of Numerical Recipes' ranqd1), started at x = seed;
    byte i comes from the state after i + 1 steps."""
    out = np.empty(n, np.uint8)
    x = seed & 0xFFFFFFFF
    for i in range(n):
        x = (1664525 * x + 1013904223) & 0xFFFFFFFF
        out[i] = x >> 24
    return out
