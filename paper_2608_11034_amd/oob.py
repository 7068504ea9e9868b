"""Python binding of libc3_oob.so (include/c3_oob.h): out-of-band hang
localization (Sec. 7; Sec. 9 progress path and communication).

Trainer side: ``ProgressPublisher`` writes the rank's progress coordinate and,
around a collective that may block, the collective's fingerprint into its
shared-memory slot.  Observer side: ``Observer`` (a CPU-only process per
rank) waits until that slot's visible progress has been silent beyond a
threshold, gathers every rank's record over a Gloo group of the observers
only, and classifies the hang with exact C3 (``classify``).

Argument marshalling only; the record, the fingerprints and the vote are in
the C++ library.  Nothing here touches a GPU.
"""
from __future__ import annotations

import contextlib
import ctypes
import os

from . import build as _build

PENDING = 1
COLL = dict(all_reduce=1, all_gather=2, reduce_scatter=3, broadcast=4, reduce=5, all_to_all=6,
            barrier=7, send=8, recv=9)
GROUP_STALL, RANK_DIVERGENCE, INCONCLUSIVE = 0, 1, 2
CLASS_NAMES = {GROUP_STALL: "group_stall", RANK_DIVERGENCE: "rank_divergence",
               INCONCLUSIVE: "inconclusive"}
REASON_NONE, REASON_PROGRESS, REASON_PROTOCOL = 0, 1, 2
REASON_NAMES = {REASON_NONE: "none", REASON_PROGRESS: "progress", REASON_PROTOCOL: "protocol"}
MAX_RANKS = 64


class OOBError(RuntimeError):
    pass


class Progress(ctypes.Structure):
    _fields_ = [("step", ctypes.c_uint64), ("op_id", ctypes.c_uint64),
                ("fingerprint", ctypes.c_uint64), ("publish_ns", ctypes.c_uint64),
                ("publishes", ctypes.c_uint64), ("flags", ctypes.c_uint32),
                ("pid", ctypes.c_uint32)]

    def as_dict(self):
        return {f: int(getattr(self, f)) for f, _ in self._fields_}


class Collective(ctypes.Structure):
    _fields_ = [("process_group", ctypes.c_uint64), ("kind", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("reduce_op", ctypes.c_int32), ("root", ctypes.c_int32),
                ("ndim", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("shape", ctypes.c_int64 * 8)]


class HangVerdict(ctypes.Structure):
    _fields_ = [("cls", ctypes.c_int32), ("majority_idx", ctypes.c_int32),
                ("bitmap", ctypes.c_uint64), ("reason", ctypes.c_uint8 * MAX_RANKS)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.OOB_LIB):
            raise OOBError(f"{_build.OOB_LIB} is not built; run __graft_entry__.build() first")
        L = ctypes.CDLL(_build.OOB_LIB)
        vp, i32, u32, u64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_uint32, ctypes.c_uint64
        L.c3_oob_abi_version.restype = i32
        L.c3_progress_open.restype = i32
        L.c3_progress_open.argtypes = [ctypes.c_char_p, i32, i32, ctypes.POINTER(vp)]
        L.c3_progress_close.restype = i32
        L.c3_progress_close.argtypes = [vp, i32]
        L.c3_progress_slots.restype = i32
        L.c3_progress_slots.argtypes = [vp]
        L.c3_progress_publish.restype = i32
        L.c3_progress_publish.argtypes = [vp, i32, u64, u64, u64, u32]
        L.c3_progress_read.restype = i32
        L.c3_progress_read.argtypes = [vp, i32, vp]
        L.c3_progress_wait_silence.restype = i32
        L.c3_progress_wait_silence.argtypes = [vp, i32, u64, u64, u64, vp]
        L.c3_group_id.restype = u64
        L.c3_group_id.argtypes = [vp, i32]
        L.c3_collective_fingerprint.restype = u64
        L.c3_collective_fingerprint.argtypes = [vp]
        L.c3_progress_evidence.restype = u64
        L.c3_progress_evidence.argtypes = [vp]
        L.c3_hang_classify.restype = i32
        L.c3_hang_classify.argtypes = [vp, i32, vp]
        if L.c3_oob_abi_version() != 1:
            raise OOBError("libc3_oob.so ABI version mismatch")
        _lib = L
    return _lib


def _check(rc, what):
    if rc < 0:
        raise OOBError(f"{what} failed ({rc})")
    return rc


class ProgressSegment:
    """A mapped progress segment: one record slot per local rank."""

    def __init__(self, name: str, n_slots: int = 0, create: bool = False):
        self.name = name if name.startswith("/") else "/" + name
        h = ctypes.c_void_p()
        _check(lib().c3_progress_open(self.name.encode(), int(n_slots), int(create), ctypes.byref(h)),
               f"c3_progress_open({self.name})")
        self.h = h
        self.n_slots = lib().c3_progress_slots(h)

    def publish(self, slot: int, step: int, op_id: int, fingerprint: int = 0, pending=False):
        _check(lib().c3_progress_publish(self.h, slot, step, op_id, fingerprint,
                                         PENDING if pending else 0), "c3_progress_publish")

    def read(self, slot: int) -> Progress:
        p = Progress()
        _check(lib().c3_progress_read(self.h, slot, ctypes.byref(p)), "c3_progress_read")
        return p

    def wait_silence(self, slot: int, silence_s: float, poll_s: float = 0.01,
                     max_wait_s: float = 60.0):
        """(silent, snapshot): silent once the slot's publication counter has
        not moved for silence_s; False after max_wait_s."""
        p = Progress()
        rc = _check(lib().c3_progress_wait_silence(self.h, slot, int(silence_s * 1e9),
                                                   max(1, int(poll_s * 1e9)),
                                                   int(max_wait_s * 1e9), ctypes.byref(p)),
                    "c3_progress_wait_silence")
        return rc == 1, p

    def close(self, unlink: bool = False):
        if self.h:
            lib().c3_progress_close(self.h, int(unlink))
            self.h = None


def group_id(ranks) -> int:
    arr = (ctypes.c_int32 * len(ranks))(*ranks)
    return int(lib().c3_group_id(arr, len(ranks)))


def collective_fingerprint(kind, group_ranks, dtype: int, shape=(), reduce_op: int = -1,
                           root: int = -1, rank_dependent_shape: bool = False) -> int:
    c = Collective()
    c.process_group = group_id(group_ranks)
    c.kind = COLL[kind] if isinstance(kind, str) else int(kind)
    c.dtype, c.reduce_op, c.root = int(dtype), int(reduce_op), int(root)
    if rank_dependent_shape:
        c.ndim = -1
    else:
        if len(shape) > 8:
            raise OOBError("at most 8 dimensions")
        c.ndim = len(shape)
        for d, n in enumerate(shape):
            c.shape[d] = int(n)
    fp = int(lib().c3_collective_fingerprint(ctypes.byref(c)))
    if fp == 0:
        raise OOBError("invalid collective description")
    return fp


def evidence(p: Progress) -> int:
    return int(lib().c3_progress_evidence(ctypes.byref(p)))


def _records_array(records):
    arr = (Progress * len(records))()
    for i, r in enumerate(records):
        if isinstance(r, Progress):
            arr[i] = r
        else:
            for f, _ in Progress._fields_:
                setattr(arr[i], f, int(r.get(f, 0)))
    return arr


def classify(records) -> dict:
    """Exact C3 over gathered progress records (Progress or dicts)."""
    R = len(records)
    if not 2 <= R <= MAX_RANKS:
        raise OOBError("2..64 records (a single rank has no peer to compare with)")
    v = HangVerdict()
    _check(lib().c3_hang_classify(_records_array(records), R, ctypes.byref(v)), "c3_hang_classify")
    return {"class": CLASS_NAMES[v.cls], "cls": int(v.cls), "majority_idx": int(v.majority_idx),
            "bitmap": int(v.bitmap), "outliers": [i for i in range(R) if v.bitmap >> i & 1],
            "reasons": {i: REASON_NAMES[v.reason[i]] for i in range(R) if v.bitmap >> i & 1}}


# ---------------------------------------------------------------------------
# trainer side
# ---------------------------------------------------------------------------
class ProgressPublisher:
    """The trainer rank's writer of its progress slot.

    ``advance(op_id)`` marks a boundary of the current step;
    ``step_done()`` moves to the next optimizer step; ``collective(...)``
    wraps a collective call: the fingerprint is published as pending before
    the call (intent before entering, Sec. 7) and cleared after it returns.
    """

    def __init__(self, seg_name: str, slot: int, n_slots: int):
        self.seg = ProgressSegment(seg_name, n_slots, create=True)
        self.slot = slot
        self.step = 0
        self.op_id = 0
        self.seg.publish(slot, 0, 0)

    def advance(self, op_id: int = None):
        self.op_id = self.op_id + 1 if op_id is None else int(op_id)
        self.seg.publish(self.slot, self.step, self.op_id)

    def step_done(self):
        self.step += 1
        self.op_id = 0
        self.seg.publish(self.slot, self.step, self.op_id)

    @contextlib.contextmanager
    def collective(self, kind, group_ranks, dtype: int, shape=(), reduce_op: int = -1,
                   root: int = -1, rank_dependent_shape: bool = False):
        fp = collective_fingerprint(kind, group_ranks, dtype, shape, reduce_op, root,
                                    rank_dependent_shape)
        self.op_id += 1
        self.seg.publish(self.slot, self.step, self.op_id, fp, pending=True)
        yield fp
        self.seg.publish(self.slot, self.step, self.op_id)

    def close(self):
        self.seg.close()


# ---------------------------------------------------------------------------
# observer side
# ---------------------------------------------------------------------------
class Observer:
    """CPU-only observer of one rank (Sec. 7, an independent observer).

    Its Gloo group is rendezvoused separately from the training
    communicator (``init_method``), at construction by default, so a blocked
    trainer or communicator does not block it and a hang costs only the
    exchange.  ``watch`` returns None while progress is visible and
    a verdict once silence has lasted ``silence_s`` and every observer has
    contributed its record.
    """

    def __init__(self, seg_name: str, slot: int, rank: int, world: int, init_method: str,
                 exchange_timeout_s: float = 60.0, connect: bool = True):
        self.seg = ProgressSegment(seg_name)
        self.slot, self.rank, self.world = slot, rank, world
        self.init_method = init_method
        self.exchange_timeout_s = exchange_timeout_s
        self._pg = None
        if connect:          # rendezvous now, so a hang only costs the exchange itself
            self._group()

    def _group(self):
        if self._pg is None:
            import datetime

            import torch.distributed as dist
            dist.init_process_group("gloo", init_method=self.init_method, rank=self.rank,
                                    world_size=self.world,
                                    timeout=datetime.timedelta(seconds=self.exchange_timeout_s))
            self._pg = dist.group.WORLD
        return self._pg

    def exchange(self, rec: Progress):
        """All observers' records, in rank order (a Gloo all_gather of 6 words)."""
        import torch
        import torch.distributed as dist
        self._group()
        words = [rec.step, rec.op_id, rec.fingerprint, rec.publish_ns, rec.publishes,
                 rec.flags | (rec.pid << 32)]
        mine = torch.tensor([w - (1 << 64) if w >= 1 << 63 else w for w in words], dtype=torch.int64)
        out = [torch.empty_like(mine) for _ in range(self.world)]
        dist.all_gather(out, mine)
        recs = []
        for t in out:
            w = [int(x) & ((1 << 64) - 1) for x in t.tolist()]
            p = Progress()
            p.step, p.op_id, p.fingerprint, p.publish_ns, p.publishes = w[:5]
            p.flags, p.pid = w[5] & 0xFFFFFFFF, w[5] >> 32
            recs.append(p)
        return recs

    def watch(self, silence_s: float, poll_s: float = 0.01, max_wait_s: float = 60.0,
              armed_after_first_publish: bool = True):
        """Verdict dict once this rank's progress has been silent for
        silence_s (after its first publication, by default); None if
        max_wait_s passes first."""
        import time
        t0 = time.monotonic()
        if armed_after_first_publish:
            while self.seg.read(self.slot).publishes == 0:
                if time.monotonic() - t0 > max_wait_s:
                    return None
                time.sleep(poll_s)
        left = max(0.0, max_wait_s - (time.monotonic() - t0))
        silent, rec = self.seg.wait_silence(self.slot, silence_s, poll_s, left)
        if not silent:
            return None
        recs = self.exchange(rec)
        v = classify(recs)
        v["records"] = [r.as_dict() for r in recs]
        return v

    def close(self):
        if self._pg is not None:
            import torch.distributed as dist
            dist.destroy_process_group()
            self._pg = None
        self.seg.close()
