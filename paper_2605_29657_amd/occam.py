"""Thin ctypes binding of liboccam (include/occam.h).

Argument marshalling only: every step of the pruning path runs in the HIP
kernels of ``liboccam.so``.  PyTorch supplies device memory and the stream
(``torch.cuda.current_stream()`` unless one is passed).  If the library has
not been built, every call raises; there is no fallback.

The functions mirror the C entry points one to one and take torch tensors
(or ``None`` for nullable pointers).  Output tensors are passed in, exactly as
in C; :func:`prune_outputs` and :func:`workspace` only allocate them.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboccam.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = range(5)
F32, BF16 = 0, 1
REG_MEAN, REG_MAX, REG_SUM = 0, 1, 2
REF_CAND_MEAN = 3               # mean-based threshold of the component ablation
ROWS_MAX, ROWS_MEAN = 0, 1
MAX_ROW_TENSORS = 8

EXPORTS = ("occam_status_string", "occam_version", "occam_workspace_size", "occam_score",
           "occam_threshold", "occam_select", "occam_gather", "occam_prune",
           "occam_register_redirect", "occam_match_lambda", "occam_select_topk",
           "occam_prune_noalloc")


class OccamError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


class _Problem(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("num_registers", ctypes.c_int32), ("rows", ctypes.c_int32),
                ("cands", ctypes.c_int32), ("q_offsets", ctypes.c_void_p),
                ("key_offsets", ctypes.c_void_p), ("max_rows", ctypes.c_int32),
                ("max_cands", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float), ("visual_row_reduce", ctypes.c_int32)]


class _Rows(ctypes.Structure):
    _fields_ = [("src", ctypes.c_void_p), ("dst", ctypes.c_void_p),
                ("src_pad_rows", ctypes.c_int64), ("src_row0", ctypes.c_int64),
                ("src_row_stride_bytes", ctypes.c_int64),
                ("dst_row_stride_bytes", ctypes.c_int64), ("row_bytes", ctypes.c_int64)]


_lib = None


def lib():
    """The loaded liboccam.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("liboccam.so is not built (python -m paper_2605_29657_amd.build)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
        P = ctypes.POINTER(_Problem)
        RP = ctypes.POINTER(_Rows)
        L.occam_status_string.argtypes = [i32]
        L.occam_status_string.restype = ctypes.c_char_p
        L.occam_version.argtypes = []
        L.occam_version.restype = i32
        L.occam_workspace_size.argtypes = [P]
        L.occam_workspace_size.restype = sz
        L.occam_score.argtypes = [P, vp, vp, vp, vp, vp, sz, vp]
        L.occam_score.restype = i32
        L.occam_threshold.argtypes = [P, vp, f32, i32, vp, vp]
        L.occam_threshold.restype = i32
        L.occam_select.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.occam_select.restype = i32
        L.occam_select_topk.argtypes = [P, vp, i32, vp, vp, vp, vp, vp, sz, vp]
        L.occam_select_topk.restype = i32
        L.occam_gather.argtypes = [P, i32, RP, vp, vp, vp]
        L.occam_gather.restype = i32
        L.occam_prune.argtypes = [P, vp, vp, vp, f32, i32, vp, i32, RP, vp, vp, vp, vp, vp, vp,
                                  sz, vp]
        L.occam_prune.restype = i32
        L.occam_prune_noalloc.argtypes = [P, vp, vp, vp, f32, i32, vp, i32, RP, vp, vp, vp, vp,
                                          vp, vp]
        L.occam_prune_noalloc.restype = i32
        L.occam_register_redirect.argtypes = [P, vp, i32, ctypes.c_int64, vp, i32, i32, vp]
        L.occam_register_redirect.restype = i32
        L.occam_match_lambda.argtypes = [P, vp, i32, f32, vp, vp, vp, sz, vp]
        L.occam_match_lambda.restype = i32
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().occam_status_string(int(status)).decode()


def _check(status: int):
    if status != OK:
        raise OccamError(status, status_string(status))


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(stream)


class Problem:
    """occam_problem.  Offsets, when given, are int32 device tensors of length B+1."""

    def __init__(self, batch, num_heads, num_kv_heads, head_dim, num_registers, rows=1, cands=0,
                 q_offsets=None, key_offsets=None, max_rows=0, max_cands=0, dtype=BF16,
                 softmax_scale=0.0, visual_row_reduce=ROWS_MAX):
        if isinstance(dtype, str):
            dtype = {"bf16": BF16, "f32": F32}[dtype]
        self.q_offsets, self.key_offsets = q_offsets, key_offsets   # keep alive
        self.c = _Problem(int(batch), int(num_heads), int(num_kv_heads), int(head_dim),
                          int(num_registers), int(rows), int(cands), _ptr(q_offsets),
                          _ptr(key_offsets), int(max_rows), int(max_cands), int(dtype),
                          float(softmax_scale), int(visual_row_reduce))

    @property
    def ref(self):
        return ctypes.byref(self.c)


class Rows:
    """occam_rows: gather ``src`` rows into ``dst`` (2-D tensors, row-major rows)."""

    def __init__(self, src, dst, src_pad_rows=0, src_row0=0, row_bytes=None,
                 src_row_stride_bytes=None, dst_row_stride_bytes=None):
        self.src, self.dst = src, dst
        rb = row_bytes if row_bytes is not None else src.shape[1] * src.element_size()
        self.c = _Rows(_ptr(src), _ptr(dst), int(src_pad_rows), int(src_row0),
                       int(src_row_stride_bytes if src_row_stride_bytes is not None
                           else src.stride(0) * src.element_size()),
                       int(dst_row_stride_bytes if dst_row_stride_bytes is not None
                           else dst.stride(0) * dst.element_size()),
                       int(rb))


def _rows_array(rows):
    rows = list(rows or [])
    if not rows:
        return 0, None
    arr = (_Rows * len(rows))(*[r.c for r in rows])
    return len(rows), arr


def workspace_size(problem: Problem) -> int:
    return int(lib().occam_workspace_size(problem.ref))


def workspace(problem: Problem, device="cuda") -> torch.Tensor:
    n = workspace_size(problem)
    if n == 0:
        raise OccamError(ERR_INVALID_ARG, "invalid problem (workspace size 0)")
    return torch.empty(n, dtype=torch.uint8, device=device)


def score(problem, q, k, scores, ws, row_lse=None, stream=None):
    _check(lib().occam_score(problem.ref, _ptr(q), _ptr(k), _ptr(row_lse), _ptr(scores),
                             _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)))


def threshold(problem, scores, lam, reduce, tau, stream=None):
    _check(lib().occam_threshold(problem.ref, _ptr(scores), float(lam), int(reduce), _ptr(tau),
                                 _stream(stream)))


def select(problem, scores, tau, kept_idx, kept_count, kept_offsets, ws, index_map=None,
           stream=None):
    _check(lib().occam_select(problem.ref, _ptr(scores), _ptr(tau), _ptr(index_map),
                              _ptr(kept_idx), _ptr(kept_count), _ptr(kept_offsets), _ptr(ws),
                              0 if ws is None else ws.numel(), _stream(stream)))


def gather(problem, rows, kept_idx, kept_offsets, stream=None):
    n, arr = _rows_array(rows)
    _check(lib().occam_gather(problem.ref, n, arr, _ptr(kept_idx), _ptr(kept_offsets),
                              _stream(stream)))


def select_topk(problem, scores, k_keep, kept_idx, kept_count, kept_offsets, ws, index_map=None,
                stream=None):
    _check(lib().occam_select_topk(problem.ref, _ptr(scores), int(k_keep), _ptr(index_map),
                                   _ptr(kept_idx), _ptr(kept_count), _ptr(kept_offsets),
                                   _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)))


def prune(problem, q, k, lam, kept_idx, kept_count, kept_offsets, ws, reduce=REG_MEAN,
          rows=None, scores=None, tau=None, row_lse=None, index_map=None, stream=None):
    n, arr = _rows_array(rows)
    _check(lib().occam_prune(problem.ref, _ptr(q), _ptr(k), _ptr(row_lse), float(lam), int(reduce),
                             _ptr(index_map), n, arr, _ptr(scores), _ptr(tau), _ptr(kept_idx),
                             _ptr(kept_count), _ptr(kept_offsets), _ptr(ws),
                             0 if ws is None else ws.numel(), _stream(stream)))


def prune_noalloc(problem, q, k, lam, kept_idx, kept_count, kept_offsets, reduce=REG_MEAN,
                  rows=None, scores=None, tau=None, row_lse=None, index_map=None, stream=None):
    """occam_prune_noalloc: occam_prune on the library's built-in workspace."""
    n, arr = _rows_array(rows)
    _check(lib().occam_prune_noalloc(problem.ref, _ptr(q), _ptr(k), _ptr(row_lse), float(lam),
                                     int(reduce), _ptr(index_map), n, arr, _ptr(scores),
                                     _ptr(tau), _ptr(kept_idx), _ptr(kept_count),
                                     _ptr(kept_offsets), _stream(stream)))


def match_lambda(problem, scores, k_target, lam_out, ws, mean_kept=None, reduce=REG_MEAN,
                 stream=None):
    """occam_match_lambda: writes the budget-matched lambda into ``lam_out[0]``."""
    _check(lib().occam_match_lambda(problem.ref, _ptr(scores), int(reduce), float(k_target),
                                    _ptr(lam_out), _ptr(mean_kept), _ptr(ws),
                                    0 if ws is None else ws.numel(), _stream(stream)))


def register_redirect(problem, h, channels, reg_slot=0, stream=None):
    """occam_register_redirect on a 2-D activation tensor ``h`` ([rows, width], in place);
    ``channels`` an int32 device tensor of channel indices."""
    if h.dim() != 2:
        raise ValueError("h must be a 2-D [rows, width] tensor")
    _check(lib().occam_register_redirect(problem.ref, _ptr(h), int(h.shape[1]),
                                         int(h.stride(0) * h.element_size()), _ptr(channels),
                                         int(channels.numel()) if channels is not None else 0,
                                         int(reg_slot), _stream(stream)))


def prune_outputs(batch: int, total_cands: int, total_keys: int, device="cuda"):
    """Allocate the fused call's outputs: dict(scores, tau, kept_idx, kept_count, kept_offsets)."""
    return dict(scores=torch.empty(max(total_keys, 1), dtype=torch.float32, device=device),
                tau=torch.empty(batch, dtype=torch.float32, device=device),
                kept_idx=torch.empty(max(total_cands, 1), dtype=torch.int32, device=device),
                kept_count=torch.empty(batch, dtype=torch.int32, device=device),
                kept_offsets=torch.empty(batch + 1, dtype=torch.int32, device=device))
