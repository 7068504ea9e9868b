"""Python binding of libc3.so (include/c3.h) for torch tensors on a ROCm device.

Argument marshalling only: every step of the hot path runs in the HIP
kernels of libc3.so.  There is no CPU fallback; if the library is missing or
the tensors are not on a GPU the functions raise.

Entry points (same names as the C ABI):

* ``signature(replicas, chunk_bytes)``  -> records [R, C] (64-byte rows)
* ``check(replicas, chunk_bytes)``      -> records, votes and lists in one call
* ``tensor_signature(records, T)``       -> per-tensor signatures [R, T]
* ``consensus(evidence, mode, ...)``     -> status, bitmap, majority index
* ``localize(status, bitmap, majority_idx, records, R)`` -> lists + counts
* ``localize_noalloc(...)``              the same without a workspace
* ``confirm(fp_bitmap, time_bitmap, R, window)`` -> per-rank verdicts
* ``timing_consensus(fingerprints, times, window)`` -> verdicts (and per-unit
                                         results): both votes + confirmation
* ``adamw_slice(params, grads, exp_avgs, exp_avg_sqs, offset, n, hp)``
                                         -> updated slices [R, 3, n] fp32
* ``OptimizerBoundaryCheck``             replay + signature + vote + localize
                                         on a rotating optimizer-state slice

Records, outliers and verdicts are returned as raw device tensors
(``torch.uint8`` rows); ``records_numpy`` & co. view host copies as numpy
structured arrays with the C field names.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch  # imported before libc3.so so both use torch's HIP runtime

from . import build as _build

F32, BF16, F16, RAW = 0, 1, 2, 3
EXACT, STATISTICAL = 0, 1
EV_U64, EV_U32, EV_F32, EV_F64 = 0, 1, 2, 3
AGREE, ATTRIBUTED, INCONCLUSIVE = 0, 1, 2
KAPPA_DEFAULT = 3.5 / 0.6745
MAX_REPLICAS = 64    # fused entry points: timing consensus, confirm, AdamW replay, optimizer check
MAX_PEERS = 256      # signature, tensor signature, consensus, localize
RANK_STRAGGLER, RANK_PROTOCOL, RANK_CONSEC2 = 1, 2, 4
OUTCOME_OK, OUTCOME_STRAGGLER, OUTCOME_SDC, OUTCOME_HANG = 0, 1, 2, 3
OPT_PLAN_STAGED = 1

RECORD_DTYPE = np.dtype([("sig", "<u8"), ("n_elems", "<u8"), ("nan_count", "<u4"),
                         ("inf_count", "<u4"), ("tensor", "<u4"), ("chunk_in_tensor", "<u4"),
                         ("absmax", "<f8"), ("sum", "<f8"), ("sumsq", "<f8"), ("reserved", "<u8")])
OUTLIER_DTYPE = np.dtype([("chunk", "<i8"), ("replica", "<i4"), ("majority_replica", "<i4"),
                          ("nan_count", "<u4", (2,)), ("inf_count", "<u4", (2,)),
                          ("absmax", "<f8", (2,)), ("sum", "<f8", (2,)), ("sumsq", "<f8", (2,))])
VERDICT_DTYPE = np.dtype([("flags", "<u4"), ("first_divergent_iter", "<i4"),
                          ("divergent_count", "<u4"), ("slow_count", "<u4"),
                          ("max_window_slow", "<u4"), ("first_straggler_window", "<i4")])
assert RECORD_DTYPE.itemsize == 64 and OUTLIER_DTYPE.itemsize == 80 and VERDICT_DTYPE.itemsize == 24

_TORCH_CODE = {torch.float32: F32, torch.bfloat16: BF16, torch.float16: F16, torch.uint8: RAW}


class C3Error(RuntimeError):
    pass


class CkptState(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int32), ("q", ctypes.c_int32), ("latest", ctypes.c_int64),
                ("candidate", ctypes.c_int64), ("verified", ctypes.c_int64)]


class CkptAction(ctypes.Structure):
    _fields_ = [("captured", ctypes.c_int32), ("promoted", ctypes.c_int32),
                ("retrieve", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("persisted_id", ctypes.c_int64), ("retrieve_id", ctypes.c_int64)]


class TensorMeta(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32), ("shape", ctypes.c_int64 * 8)]


class AdamwHparams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("beta1", ctypes.c_double), ("beta2", ctypes.c_double),
                ("eps", ctypes.c_double), ("weight_decay", ctypes.c_double),
                ("step", ctypes.c_int64)]


class OptimizerState(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p), ("exp_avg", ctypes.c_void_p),
                ("exp_avg_sq", ctypes.c_void_p), ("R", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("numel", ctypes.c_int64), ("slice_elems", ctypes.c_int64),
                ("tile_bytes", ctypes.c_uint64)]


class OptimizerCheckOut(ctypes.Structure):
    _fields_ = [(name, ctypes.c_void_p) for name in ("updated", "records", "status", "bitmap",
                                                      "majority_idx", "outliers", "undecided",
                                                      "counts")]


class LaunchOpts(ctypes.Structure):
    _fields_ = [("ev_kernel_begin", ctypes.c_void_p), ("ev_kernel_end", ctypes.c_void_p),
                ("grid_blocks", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("tile_bytes", ctypes.c_uint64)]


_lib = None


def library_path() -> str:
    return _build.LIB


def lib():
    """The loaded libc3.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            raise C3Error(f"{_build.LIB} is not built; run __graft_entry__.build() first")
        L = ctypes.CDLL(_build.LIB)
        vp, i32, i64, u64, sz, dbl = (ctypes.c_void_p, ctypes.c_int, ctypes.c_int64,
                                      ctypes.c_uint64, ctypes.c_size_t, ctypes.c_double)
        L.c3_abi_version.restype = i32
        L.c3_status_string.restype = ctypes.c_char_p
        L.c3_status_string.argtypes = [i32]
        L.c3_num_chunks.restype = i64
        L.c3_num_chunks.argtypes = [vp, i32, u64]
        L.c3_signature_workspace_size.restype = sz
        L.c3_signature_workspace_size.argtypes = [vp, i32, i32, u64]
        L.c3_signature_workspace_size_ex.restype = sz
        L.c3_signature_workspace_size_ex.argtypes = [vp, i32, i32, u64, u64]
        L.c3_signature.restype = i32
        L.c3_signature.argtypes = [vp, vp, i32, i32, u64, vp, vp, sz, vp]
        L.c3_signature_ex.restype = i32
        L.c3_signature_ex.argtypes = [vp, vp, i32, i32, u64, vp, vp, sz, vp, vp]
        L.c3_check_workspace_size.restype = sz
        L.c3_check_workspace_size.argtypes = [vp, i32, i32, u64, u64]
        L.c3_check.restype = i32
        L.c3_check.argtypes = [vp, vp, i32, i32, u64, vp, vp, vp, vp, vp, i64, vp, i64, vp, vp, sz,
                               vp, vp]
        L.c3_tensor_signature.restype = i32
        L.c3_tensor_signature.argtypes = [vp, i32, i64, i32, vp, vp]
        L.c3_consensus.restype = i32
        L.c3_consensus.argtypes = [vp, i32, i64, i64, i32, i64, i32, dbl, vp, vp, vp, vp]
        L.c3_localize_workspace_size.restype = sz
        L.c3_localize_workspace_size.argtypes = [i64]
        L.c3_localize.restype = i32
        L.c3_localize.argtypes = [vp, vp, vp, vp, i32, i64, vp, i64, vp, i64, vp, vp, sz, vp]
        L.c3_localize_noalloc.restype = i32
        L.c3_localize_noalloc.argtypes = [vp, vp, vp, vp, i32, i64, vp, i64, vp, i64, vp, vp]
        L.c3_confirm_workspace_size.restype = sz
        L.c3_confirm_workspace_size.argtypes = [i32, i64, i64]
        L.c3_confirm.restype = i32
        L.c3_confirm.argtypes = [vp, vp, i32, i64, i64, i32, vp, vp, sz, vp]
        L.c3_adamw_slice.restype = i32
        L.c3_adamw_slice.argtypes = [vp, vp, vp, vp, i32, i64, i64, i64, vp, vp, i64, vp]
        L.c3_optimizer_check_workspace_size.restype = sz
        L.c3_optimizer_check_workspace_size.argtypes = [vp]
        L.c3_optimizer_check.restype = i32
        L.c3_optimizer_check.argtypes = [vp, i64, vp, vp, vp, sz, vp]
        L.c3_timing_consensus_workspace_size.restype = sz
        L.c3_timing_consensus_workspace_size.argtypes = [i32, i64, i64, i32]
        L.c3_timing_consensus.restype = i32
        L.c3_timing_consensus.argtypes = [vp, vp, i32, i32, i64, i64, dbl, i32, vp, vp, vp, vp, vp,
                                          vp, vp, vp, sz, vp]
        L.c3_read_probe.restype = i32
        L.c3_read_probe.argtypes = [vp, u64, u64, vp, vp, vp, vp]
        L.c3_job_outcome.restype = i32
        L.c3_job_outcome.argtypes = [i64, i64, i64]
        L.c3_ckpt_init.restype = i32
        L.c3_ckpt_init.argtypes = [vp, i32]
        L.c3_ckpt_save.restype = i32
        L.c3_ckpt_save.argtypes = [vp, i32, i64, i32, i32, vp]
        L.c3_ckpt_retrieve.restype = i32
        L.c3_ckpt_retrieve.argtypes = [vp, i32, i32, i32, vp]
        if L.c3_abi_version() != 1:
            raise C3Error("libc3.so ABI version mismatch")
        _lib = L
    return _lib


def _check(rc: int, what: str):
    if rc != 0:
        raise C3Error(f"{what}: {lib().c3_status_string(rc).decode()} ({rc})")


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dev_tensor(t: torch.Tensor, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise C3Error(f"{name} must be a tensor on a ROCm GPU device")
    if not t.is_contiguous():
        raise C3Error(f"{name} must be contiguous")
    return t


def _check_out(t, dtype, numel: int, name: str):
    """A caller-supplied output must hold what the kernels write."""
    _dev_tensor(t, name)
    if t.dtype != dtype:
        raise C3Error(f"{name} must be {dtype}, got {t.dtype}")
    if t.numel() < numel:
        raise C3Error(f"{name} holds {t.numel()} values, needs {numel}")


def bitmap_words(R: int) -> int:
    """int64 words of one unit's outlier bitmap (C3_BITMAP_WORDS)."""
    return (R + 63) // 64


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _empty(shape, dtype, device):
    return torch.empty(shape, dtype=dtype, device=device)


def make_metas(tensors) -> ctypes.Array:
    """c3_tensor_meta_t[T] from torch tensors (dtype code and shape)."""
    metas = (TensorMeta * len(tensors))()
    for i, t in enumerate(tensors):
        if t.dtype not in _TORCH_CODE:
            raise C3Error(f"unsupported dtype {t.dtype}")
        if t.dim() > 8:
            raise C3Error("at most 8 dimensions")
        metas[i].dtype = _TORCH_CODE[t.dtype]
        metas[i].ndim = t.dim()
        for d, n in enumerate(t.shape):
            metas[i].shape[d] = int(n)
    return metas


def num_chunks(tensors, chunk_bytes: int) -> int:
    metas = make_metas(tensors)
    c = lib().c3_num_chunks(metas, len(tensors), chunk_bytes)
    if c < 0:
        _check(int(c), "c3_num_chunks")
    return int(c)


def signature_workspace_size(tensors, R: int, chunk_bytes: int, tile_bytes: int = 0) -> int:
    metas = make_metas(tensors)
    n = lib().c3_signature_workspace_size_ex(metas, len(tensors), R, chunk_bytes, tile_bytes)
    if n == 0:
        raise C3Error("invalid signature plan")
    return int(n)


class SignaturePlan:
    """Host-side marshalling of one replica set: pointer table and metadata.

    Building it once and calling ``run`` repeatedly only avoids re-marshalling
    in Python; the library still stages the plan on every call.
    """

    def __init__(self, replicas, chunk_bytes: int, tile_bytes: int = 0):
        if len(replicas) < 1:
            raise C3Error("need at least one replica")
        T = len(replicas[0])
        dev = replicas[0][0].device
        for r, rep in enumerate(replicas):
            if len(rep) != T:
                raise C3Error("every replica must hold the same tensors")
            for t, x in enumerate(rep):
                _dev_tensor(x, f"replicas[{r}][{t}]")
                if x.device != dev:
                    raise C3Error("all replicas must be on one device")
                ref = replicas[0][t]
                if x.dtype != ref.dtype or x.shape != ref.shape:
                    raise C3Error(f"tensor {t} differs in dtype or shape between replicas")
        self.R, self.T, self.device = len(replicas), T, dev
        self.chunk_bytes, self.tile_bytes = int(chunk_bytes), int(tile_bytes)
        self.keep = [x for rep in replicas for x in rep]
        self.ptrs = (ctypes.c_void_p * (self.R * T))(*[x.data_ptr() for x in self.keep])
        self.metas = make_metas(replicas[0])
        self.C = num_chunks(replicas[0], chunk_bytes)
        self.ws_bytes = signature_workspace_size(replicas[0], self.R, chunk_bytes, tile_bytes)

    def new_records(self):
        return _empty((self.R, self.C, 64), torch.uint8, self.device)

    def new_workspace(self):
        return _empty((self.ws_bytes,), torch.uint8, self.device)

    def run(self, records, workspace, stream=None, ev_begin=None, ev_end=None, grid_blocks=0,
            plan_staged=False):
        """Launch c3_signature.  plan_staged=True promises that `workspace` still
        holds the plan a previous run of this object staged (see
        C3_OPT_PLAN_STAGED)."""
        opts = LaunchOpts(ev_begin.cuda_event if ev_begin is not None else None,
                          ev_end.cuda_event if ev_end is not None else None,
                          int(grid_blocks), OPT_PLAN_STAGED if plan_staged else 0,
                          self.tile_bytes)
        rc = lib().c3_signature_ex(self.ptrs, self.metas, self.T, self.R, self.chunk_bytes,
                                   _ptr(records), _ptr(workspace), workspace.numel(),
                                   _stream(stream), ctypes.byref(opts))
        _check(rc, "c3_signature")
        return records


    # -- the whole exact check in one call (c3_check) ----------------------
    def check_workspace_size(self) -> int:
        n = lib().c3_check_workspace_size(self.metas, self.T, self.R, self.chunk_bytes,
                                          self.tile_bytes)
        if n == 0:
            raise C3Error("invalid check plan")
        return int(n)

    def new_check_outputs(self, out_cap: int = None, und_cap: int = None):
        """Device outputs of run_check: records [R, C, 64], status [C], bitmap
        [C] (or [C, words] above 64 replicas), majority [C], outliers
        [out_cap, 80], undecided [und_cap], counts [3]."""
        C, R, dev = self.C, self.R, self.device
        W = bitmap_words(R)
        out_cap = C * R if out_cap is None else out_cap
        und_cap = C if und_cap is None else und_cap
        return (self.new_records(), _empty((C,), torch.uint8, dev),
                _empty((C,) if W == 1 else (C, W), torch.int64, dev), _empty((C,), torch.int32, dev),
                _empty((max(out_cap, 1), 80), torch.uint8, dev), _empty((max(und_cap, 1),), torch.int64, dev),
                _empty((3,), torch.int64, dev))

    def run_check(self, outputs, workspace, stream=None, ev_begin=None, ev_end=None,
                  grid_blocks=0, plan_staged=False, out_cap: int = None, und_cap: int = None):
        """Launch c3_check into `outputs` (as new_check_outputs returns them)."""
        rec, st, bm, mj, outl, und, cnt = outputs
        C, R = self.C, self.R
        _check_out(rec, torch.uint8, R * C * 64, "records")
        _check_out(st, torch.uint8, C, "status")
        _check_out(bm, torch.int64, C * bitmap_words(R), "bitmap")
        _check_out(mj, torch.int32, C, "majority")
        _check_out(cnt, torch.int64, 3, "counts")
        out_cap = outl.shape[0] if out_cap is None else min(out_cap, outl.shape[0])
        und_cap = und.numel() if und_cap is None else min(und_cap, und.numel())
        opts = LaunchOpts(ev_begin.cuda_event if ev_begin is not None else None,
                          ev_end.cuda_event if ev_end is not None else None,
                          int(grid_blocks), OPT_PLAN_STAGED if plan_staged else 0,
                          self.tile_bytes)
        rc = lib().c3_check(self.ptrs, self.metas, self.T, R, self.chunk_bytes, _ptr(rec), _ptr(st),
                            _ptr(bm), _ptr(mj), _ptr(outl), out_cap, _ptr(und), und_cap, _ptr(cnt),
                            _ptr(workspace), workspace.numel(), _stream(stream), ctypes.byref(opts))
        _check(rc, "c3_check")
        return outputs


def check(replicas, chunk_bytes: int, stream=None, tile_bytes: int = 0):
    """c3_check: records, status, bitmap, majority, outliers, undecided and
    counts of R replica lists of T device tensors, in one call."""
    plan = SignaturePlan(replicas, chunk_bytes, tile_bytes)
    outs = plan.new_check_outputs()
    ws = _empty((plan.check_workspace_size(),), torch.uint8, plan.device)
    return plan.run_check(outs, ws, stream=stream)


def signature(replicas, chunk_bytes: int, stream=None, grid_blocks: int = 0, tile_bytes: int = 0):
    """Records [R, C, 64] (uint8) of R replica lists of T device tensors."""
    plan = SignaturePlan(replicas, chunk_bytes, tile_bytes)
    rec = plan.new_records()
    ws = plan.new_workspace()
    plan.run(rec, ws, stream=stream, grid_blocks=grid_blocks)
    return rec


def tensor_signature(records: torch.Tensor, T: int, stream=None) -> torch.Tensor:
    """Per-tensor signatures [R, T] (int64 bit patterns) from records [R, C, 64]."""
    _dev_tensor(records, "records")
    R, C = records.shape[0], records.shape[1]
    out = _empty((R, T), torch.int64, records.device)
    rc = lib().c3_tensor_signature(_ptr(records), R, C, T, _ptr(out), _stream(stream))
    _check(rc, "c3_tensor_signature")
    return out


def consensus(evidence: torch.Tensor, mode: int = EXACT, *, kind: int = None, R: int = None,
              replica_stride: int = None, unit_stride: int = None, n_units: int = None,
              kappa: float = KAPPA_DEFAULT, stream=None, out=None):
    """Per-unit status, bitmap and majority index.

    ``evidence`` is either the records tensor [R, C, 64] (signatures are voted)
    or a value tensor [U, R] / [..., R] of int64/float32/float64 with the
    replicas on the last axis.  Strides are in bytes.  The bitmap is [U]
    int64 for R <= 64 and [U, bitmap_words(R)] above (bit b of word w names
    replica 64 w + b).
    """
    _dev_tensor(evidence, "evidence")
    if evidence.dtype == torch.uint8 and evidence.dim() == 3 and evidence.shape[2] == 64:
        R_, C = evidence.shape[0], evidence.shape[1]
        kind = EV_U64 if kind is None else kind
        R = R_ if R is None else R
        replica_stride = C * 64 if replica_stride is None else replica_stride
        unit_stride = 64 if unit_stride is None else unit_stride
        n_units = C if n_units is None else n_units
    else:
        if kind is None:
            kind = {torch.int64: EV_U64, torch.int32: EV_U32, torch.float32: EV_F32,
                    torch.float64: EV_F64}[evidence.dtype]
        R = evidence.shape[-1] if R is None else R
        es = evidence.element_size()
        replica_stride = es if replica_stride is None else replica_stride
        unit_stride = R * es if unit_stride is None else unit_stride
        n_units = evidence.numel() // R if n_units is None else n_units
    dev = evidence.device
    W = bitmap_words(R) if 1 <= R <= MAX_PEERS else 1
    if out is not None:
        status, bitmap, maj = out
        _check_out(status, torch.uint8, n_units, "status")
        _check_out(bitmap, torch.int64, n_units * W, "bitmap")
        _check_out(maj, torch.int32, n_units, "majority")
    else:
        status = _empty((n_units,), torch.uint8, dev)
        bitmap = _empty((n_units,) if W == 1 else (n_units, W), torch.int64, dev)
        maj = _empty((n_units,), torch.int32, dev)
    rc = lib().c3_consensus(_ptr(evidence), kind, replica_stride, unit_stride, R, n_units, mode,
                            float(kappa), _ptr(status), _ptr(bitmap), _ptr(maj), _stream(stream))
    _check(rc, "c3_consensus")
    return status, bitmap, maj


def localize(status, bitmap, majority_idx, records=None, R: int = None, out_cap: int = None,
             und_cap: int = None, stream=None, out=None, workspace=None):
    """Outlier entries [out_cap, 80] (uint8), undecided [und_cap] int64, counts [3] int64.
    ``bitmap`` holds bitmap_words(R) int64 words per unit, as consensus writes it."""
    n_units = status.numel()
    if R is None:
        if records is None:
            raise C3Error("R is required without records")
        R = records.shape[0]
    if 1 <= R <= MAX_PEERS and n_units > 0:
        _check_out(bitmap, torch.int64, n_units * bitmap_words(R), "bitmap")
        _check_out(majority_idx, torch.int32, n_units, "majority")
    dev = status.device
    out_cap = n_units * R if out_cap is None else out_cap
    und_cap = n_units if und_cap is None else und_cap
    if out is not None:
        outliers, undecided, counts = out
        out_cap = min(out_cap, outliers.shape[0])
        und_cap = min(und_cap, undecided.numel())
    else:
        outliers = _empty((max(out_cap, 1), 80), torch.uint8, dev)
        undecided = _empty((max(und_cap, 1),), torch.int64, dev)
        counts = _empty((3,), torch.int64, dev)
    ws_bytes = int(lib().c3_localize_workspace_size(n_units))
    ws = _empty((ws_bytes,), torch.uint8, dev) if workspace is None else workspace
    if ws.numel() < ws_bytes:
        raise C3Error("localize workspace too small")
    ws_bytes = ws.numel()
    rc = lib().c3_localize(_ptr(status), _ptr(bitmap), _ptr(majority_idx), _ptr(records), R, n_units,
                           _ptr(outliers), out_cap, _ptr(undecided), und_cap, _ptr(counts),
                           _ptr(ws), ws_bytes, _stream(stream))
    _check(rc, "c3_localize")
    return outliers, undecided, counts


LOCALIZE_NOALLOC_MAX_UNITS = 1 << 26


def localize_noalloc(status, bitmap, majority_idx, records=None, R: int = None, out_cap: int = None,
                     und_cap: int = None, stream=None, out=None):
    """c3_localize_noalloc: localize without a workspace (the library's fixed
    per-device scratch array; calls that overlap on one device race).  Same
    results as ``localize``.  Pass ``out`` to allocate nothing here either."""
    n_units = status.numel()
    if R is None:
        if records is None:
            raise C3Error("R is required without records")
        R = records.shape[0]
    if 1 <= R <= MAX_PEERS and n_units > 0:
        _check_out(bitmap, torch.int64, n_units * bitmap_words(R), "bitmap")
        _check_out(majority_idx, torch.int32, n_units, "majority")
    dev = status.device
    out_cap = n_units * R if out_cap is None else out_cap
    und_cap = n_units if und_cap is None else und_cap
    if out is not None:
        outliers, undecided, counts = out
        out_cap = min(out_cap, outliers.shape[0])
        und_cap = min(und_cap, undecided.numel())
    else:
        outliers = _empty((max(out_cap, 1), 80), torch.uint8, dev)
        undecided = _empty((max(und_cap, 1),), torch.int64, dev)
        counts = _empty((3,), torch.int64, dev)
    rc = lib().c3_localize_noalloc(_ptr(status), _ptr(bitmap), _ptr(majority_idx), _ptr(records), R,
                                   n_units, _ptr(outliers), out_cap, _ptr(undecided), und_cap,
                                   _ptr(counts), _stream(stream))
    _check(rc, "c3_localize_noalloc")
    return outliers, undecided, counts


def localize_workspace_size(n_units: int) -> int:
    return int(lib().c3_localize_workspace_size(n_units))


def confirm_workspace_size(R: int, G: int, T: int) -> int:
    return int(lib().c3_confirm_workspace_size(R, G, T))


def confirm(fp_bitmap, time_bitmap, R: int, window: int = 16, stream=None, out=None,
            workspace=None):
    """Per-rank verdicts [R * G, 24] (uint8) from [T, G] bitmaps; rank = r * G + g."""
    _dev_tensor(fp_bitmap, "fp_bitmap")
    _dev_tensor(time_bitmap, "time_bitmap")
    T, G = fp_bitmap.shape
    dev = fp_bitmap.device
    if out is None:
        out = _empty((R * G, 24), torch.uint8, dev)
    ws_bytes = confirm_workspace_size(R, G, T)
    ws = _empty((max(ws_bytes, 256),), torch.uint8, dev) if workspace is None else workspace
    if ws.numel() < ws_bytes:
        raise C3Error("confirm workspace too small")
    ws_bytes = ws.numel()
    rc = lib().c3_confirm(_ptr(fp_bitmap), _ptr(time_bitmap), R, G, T, window, _ptr(out), _ptr(ws),
                          ws_bytes, _stream(stream))
    _check(rc, "c3_confirm")
    return out


def timing_consensus_workspace_size(R: int, G: int, T: int, window: int = 16) -> int:
    return int(lib().c3_timing_consensus_workspace_size(R, G, T, window))


def timing_consensus(fingerprints, times, window: int = 16, kappa: float = KAPPA_DEFAULT,
                     per_unit: bool = True, stream=None, out=None, workspace=None):
    """Exact vote on fingerprints [T, G, R] (int64 bit patterns), statistical
    vote on times [T, G, R] (float32/float64) and temporal confirmation.
    Returns (verdicts [R * G, 24] uint8, fp (status, bitmap, majority) or
    None, time (status, bitmap, majority) or None)."""
    _dev_tensor(fingerprints, "fingerprints")
    _dev_tensor(times, "times")
    if fingerprints.dtype != torch.int64 or fingerprints.dim() != 3:
        raise C3Error("fingerprints must be int64 [T, G, R]")
    if times.shape != fingerprints.shape:
        raise C3Error("times must have the fingerprints' shape [T, G, R]")
    kind = {torch.float32: EV_F32, torch.float64: EV_F64}.get(times.dtype)
    if kind is None:
        raise C3Error("times must be float32 or float64")
    T, G, R = fingerprints.shape
    dev = fingerprints.device
    if out is not None:
        verdicts, fp_out, t_out = out
    else:
        verdicts = _empty((R * G, 24), torch.uint8, dev)
        fp_out = t_out = None
        if per_unit:
            fp_out = (_empty((T * G,), torch.uint8, dev), _empty((T * G,), torch.int64, dev),
                      _empty((T * G,), torch.int32, dev))
            t_out = (_empty((T * G,), torch.uint8, dev), _empty((T * G,), torch.int64, dev),
                     _empty((T * G,), torch.int32, dev))
    need = timing_consensus_workspace_size(R, G, T, window)
    if need == 0:
        raise C3Error("invalid timing-consensus sizes")
    ws = _empty((need,), torch.uint8, dev) if workspace is None else workspace
    if ws.numel() < need:
        raise C3Error("timing-consensus workspace too small")
    fo = fp_out if fp_out is not None else (None, None, None)
    to = t_out if t_out is not None else (None, None, None)
    rc = lib().c3_timing_consensus(_ptr(fingerprints), _ptr(times), kind, R, G, T, float(kappa),
                                   int(window), _ptr(fo[0]), _ptr(fo[1]), _ptr(fo[2]), _ptr(to[0]),
                                   _ptr(to[1]), _ptr(to[2]), _ptr(verdicts), _ptr(ws), ws.numel(),
                                   _stream(stream))
    _check(rc, "c3_timing_consensus")
    return verdicts, fp_out, t_out


# ---------------------------------------------------------------------------
# optimizer-boundary check
# ---------------------------------------------------------------------------
SLICE_ELEMS = 65536


def adamw_hparams(lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=1e-2, step=1) -> AdamwHparams:
    return AdamwHparams(float(lr), float(betas[0]), float(betas[1]), float(eps),
                        float(weight_decay), int(step))


def _ptr_table(tensors, name, numel, dev):
    for i, t in enumerate(tensors):
        _dev_tensor(t, f"{name}[{i}]")
        if t.dtype != torch.float32 or t.numel() != numel or t.device != dev:
            raise C3Error(f"{name}[{i}] must be fp32 with {numel} elements on {dev}")
    return (ctypes.c_void_p * len(tensors))(*[t.data_ptr() for t in tensors])


def adamw_slice(params, grads, exp_avgs, exp_avg_sqs, offset: int, n: int, hp: AdamwHparams,
                out=None, out_stride: int = 0, stream=None, _tables=None):
    """Replay one AdamW step on elements [offset, offset + n) of R replicas'
    fp32 tensors.  Returns out: row (r, j) at element (3 r + j) * stride,
    stride = out_stride or n (by default a new [R, 3, n] tensor) holding the
    updated param (j = 0), exp_avg (1) and exp_avg_sq (2)."""
    R = len(params)
    if not (len(grads) == len(exp_avgs) == len(exp_avg_sqs) == R) or R < 1:
        raise C3Error("params, grads, exp_avgs and exp_avg_sqs need one tensor per replica")
    numel, dev = params[0].numel(), params[0].device
    tables = _tables or [_ptr_table(x, nm, numel, dev) for x, nm in
                         ((params, "params"), (grads, "grads"), (exp_avgs, "exp_avgs"),
                          (exp_avg_sqs, "exp_avg_sqs"))]
    stride = out_stride or n
    if out is None:
        out = _empty((R, 3, stride), torch.float32, dev)
    elif out.dtype != torch.float32 or out.numel() < (3 * R - 1) * stride + n:
        raise C3Error("out must be fp32 with room for R * 3 rows of the stride")
    rc = lib().c3_adamw_slice(tables[0], tables[1], tables[2], tables[3], R, numel, int(offset),
                              int(n), ctypes.byref(hp), _ptr(_dev_tensor(out, "out")), int(out_stride),
                              _stream(stream))
    _check(rc, "c3_adamw_slice")
    return out


def optimizer_slice(k: int, numel: int, slice_elems: int = SLICE_ELEMS):
    """(offset, n) of rotating check k: the (k mod S)-th window of slice_elems
    elements among the S = ceil(numel / slice_elems) windows of the tensor."""
    if numel <= 0:
        return 0, 0
    n_slices = -(-numel // slice_elems)
    off = (k % n_slices) * slice_elems
    return off, min(slice_elems, numel - off)


class OptimizerBoundaryCheck:
    """Scheduled optimizer-boundary checks over R replicas' AdamW state
    (c3_optimizer_check).

    Check k takes the rotating slice ``optimizer_slice(k, numel)`` and signs
    seven tensors per replica: the four pre-update input slices (param, grad,
    exp_avg, exp_avg_sq; whether the replicas start from identical values)
    and the three updated slices of the replayed step (param, exp_avg,
    exp_avg_sq).  Each is one chunk, so unit u of the vote is tensor u in
    ``UNITS`` order.  Exact C3 votes per unit and localize lists the outliers.
    All buffers are allocated here once; ``run`` enqueues one check.
    """

    UNITS = ("param", "grad", "exp_avg", "exp_avg_sq", "param_new", "exp_avg_new",
             "exp_avg_sq_new")

    def __init__(self, params, grads, exp_avgs, exp_avg_sqs, slice_elems: int = SLICE_ELEMS,
                 tile_bytes: int = 0):
        self.R = len(params)
        if self.R < 2:
            raise C3Error("need at least two replicas")
        self.numel, self.device = params[0].numel(), params[0].device
        self.state = (list(params), list(grads), list(exp_avgs), list(exp_avg_sqs))
        self.tables = [_ptr_table(x, nm, self.numel, self.device) for x, nm in
                       zip(self.state, ("params", "grads", "exp_avgs", "exp_avg_sqs"))]
        self.slice_elems = int(slice_elems)
        self.st = OptimizerState(ctypes.cast(self.tables[0], ctypes.c_void_p),
                                 ctypes.cast(self.tables[1], ctypes.c_void_p),
                                 ctypes.cast(self.tables[2], ctypes.c_void_p),
                                 ctypes.cast(self.tables[3], ctypes.c_void_p),
                                 self.R, 0, self.numel, self.slice_elems, int(tile_bytes))
        ws_bytes = int(lib().c3_optimizer_check_workspace_size(ctypes.byref(self.st)))
        if ws_bytes == 0:
            raise C3Error("invalid optimizer-check configuration")
        R, dev, U = self.R, self.device, len(self.UNITS)
        self.updated = _empty((R, 3, self.slice_elems), torch.float32, dev)
        self.records = _empty((R, U, 64), torch.uint8, dev)
        self.status = _empty((U,), torch.uint8, dev)
        self.bitmap = _empty((U,), torch.int64, dev)
        self.majority = _empty((U,), torch.int32, dev)
        self.outliers = _empty((U * R, 80), torch.uint8, dev)
        self.undecided = _empty((U,), torch.int64, dev)
        self.counts = _empty((3,), torch.int64, dev)
        self.workspace = _empty((ws_bytes,), torch.uint8, dev)
        self.out = OptimizerCheckOut(*[t.data_ptr() for t in (
            self.updated, self.records, self.status, self.bitmap, self.majority, self.outliers,
            self.undecided, self.counts)])

    def slice(self, k: int):
        return optimizer_slice(k, self.numel, self.slice_elems)

    def updated_slices(self, k: int):
        """[R, 3, n] view of the replayed values of check k (after it ran)."""
        return self.updated[:, :, : self.slice(k)[1]]

    def run(self, k: int, hp: AdamwHparams, stream=None):
        """Enqueue check k; returns (records, status, bitmap, majority, outliers,
        undecided, counts), device tensors owned by this object."""
        rc = lib().c3_optimizer_check(ctypes.byref(self.st), int(k), ctypes.byref(hp),
                                      ctypes.byref(self.out), _ptr(self.workspace),
                                      self.workspace.numel(), _stream(stream))
        _check(rc, "c3_optimizer_check")
        return (self.records, self.status, self.bitmap, self.majority, self.outliers,
                self.undecided, self.counts)


# ---------------------------------------------------------------------------
# measurement aid
# ---------------------------------------------------------------------------
def read_probe(buf: torch.Tensor, tile_bytes: int = 0, checksum=None, ev_begin=None,
               ev_end=None, stream=None):
    """c3_read_probe over the bytes of ``buf``: one read with the signature
    kernel's access pattern.  Returns the per-tile xor checksums [n_tiles]
    (int64 bit patterns)."""
    _dev_tensor(buf, "buf")
    nbytes = buf.numel() * buf.element_size()
    tb = tile_bytes or 256 * 1024
    n_tiles = -(-nbytes // tb)
    if checksum is None:
        checksum = _empty((max(n_tiles, 1),), torch.int64, buf.device)
    elif checksum.numel() < n_tiles:
        raise C3Error("checksum holds fewer values than tiles")
    rc = lib().c3_read_probe(_ptr(buf), nbytes, tile_bytes, _ptr(checksum),
                             ev_begin.cuda_event if ev_begin is not None else None,
                             ev_end.cuda_event if ev_end is not None else None, _stream(stream))
    _check(rc, "c3_read_probe")
    return checksum[:n_tiles]


# ---------------------------------------------------------------------------
# checkpoint certification (host-only)
# ---------------------------------------------------------------------------
def job_outcome(sdc_units: int, hang_signals: int, stragglers: int) -> int:
    rc = lib().c3_job_outcome(sdc_units, hang_signals, stragglers)
    if rc < 0:
        _check(rc, "c3_job_outcome")
    return rc


class CheckpointGate:
    """Algorithm 3 state (latest / candidate / verified) held by libc3."""

    def __init__(self, K: int):
        self.state = CkptState()
        _check(lib().c3_ckpt_init(ctypes.byref(self.state), K), "c3_ckpt_init")

    def save(self, outcome: int, checkpoint_id: int, machines_accessible=True,
             full_catalog_sdc=False) -> CkptAction:
        act = CkptAction()
        _check(lib().c3_ckpt_save(ctypes.byref(self.state), outcome, checkpoint_id,
                                  int(bool(machines_accessible)), int(bool(full_catalog_sdc)),
                                  ctypes.byref(act)), "c3_ckpt_save")
        return act

    def retrieve(self, outcome: int, machines_accessible=True, full_catalog_sdc=False) -> int:
        out = ctypes.c_int64(-1)
        _check(lib().c3_ckpt_retrieve(ctypes.byref(self.state), outcome,
                                      int(bool(machines_accessible)), int(bool(full_catalog_sdc)),
                                      ctypes.byref(out)), "c3_ckpt_retrieve")
        return out.value


# ---------------------------------------------------------------------------
# host views
# ---------------------------------------------------------------------------
def records_numpy(records: torch.Tensor) -> np.ndarray:
    a = records.detach().cpu().contiguous().numpy()
    return a.reshape(-1).view(RECORD_DTYPE).reshape(a.shape[:-1])


def outliers_numpy(outliers: torch.Tensor, counts: torch.Tensor) -> np.ndarray:
    n = min(int(counts[0]), outliers.shape[0])
    return outliers[:n].detach().cpu().contiguous().numpy().reshape(-1).view(OUTLIER_DTYPE)


def verdicts_numpy(verdicts: torch.Tensor) -> np.ndarray:
    return verdicts.detach().cpu().contiguous().numpy().reshape(-1).view(VERDICT_DTYPE)
