"""Plain fp64 CPU oracle for OccamToken's register-anchored relative evidence test.

TEST INFRASTRUCTURE ONLY.  The tests, the smoke check and the benchmark's CPU
baseline leg are the only callers.  The GPU library neither imports nor links
anything here, and nothing here imports the GPU library.

The arithmetic lives in ``occam_oracle.c`` (double precision, plain loops,
OpenMP over the anchor rows of a sample); this module builds it with gcc, loads it with
ctypes and adds two small numpy helpers that the paper defines outside the hot
path:

* :func:`match_lambda` -- the budget-matching rule (Appendix, Eq.
  lambda2_budget_matching_appendix): the coefficient whose mean kept count over
  a calibration set is closest to a target budget.
* :func:`neff` -- the effective number of attended tokens (Sec. 3.2,
  Observation 1).

Inputs are host numpy arrays.  ``dtype`` is ``"f32"`` (``np.float32``) or
``"bf16"`` (raw bfloat16 bits held in ``np.uint16``); bf16 values are widened
to double exactly, so the oracle reads the very bits the GPU reads.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "occam_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboccam_oracle.so")
_lib = None
_lock = threading.Lock()

REG_MEAN, REG_MAX, REG_SUM = 0, 1, 2
CAND_MEAN = 3                   # ablation: reference = mean visual score instead of s(r)
ROWS_MAX, ROWS_MEAN = 0, 1      # visual keys: max over anchor rows (Stage II) or mean (mutual)
_DTYPES = {"f32": 0, "bf16": 1}


def build(force: bool = False) -> str:
    """Compile the C oracle with gcc (strict IEEE, no fast-math) and return its path."""
    if force or not os.path.exists(_LIB_PATH) or (
            os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                        "-Wall", "-Wextra", _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build()
            lib = ctypes.CDLL(_LIB_PATH)
            p = ctypes.c_void_p
            i32, i64, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_double
            lib.oracle_scores.argtypes = [i32, i32, i32, i32, i32, p, p, i32, p, p, f64, p, i32, p]
            lib.oracle_scores.restype = i32
            lib.oracle_threshold.argtypes = [i32, i32, p, p, f64, i32, p]
            lib.oracle_threshold.restype = i32
            lib.oracle_select.argtypes = [i32, i32, p, p, p, p, p, p, p]
            lib.oracle_select.restype = i32
            lib.oracle_select_topk.argtypes = [i32, i32, p, p, i64, p, p, p, p]
            lib.oracle_select_topk.restype = i32
            lib.oracle_gather.argtypes = [i32, i32, p, p, i64, i64, i64, p, i64, i64, p, p]
            lib.oracle_gather.restype = i32
            lib.oracle_register_redirect.argtypes = [i32, i32, p, i32, p, i64, i64, p, i32, i32]
            lib.oracle_register_redirect.restype = i32
            lib.oracle_neff.argtypes = [p, i64]
            lib.oracle_neff.restype = f64
            lib.oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
            lib.oracle_bf16_to_double.restype = f64
            _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _offsets(off):
    return np.ascontiguousarray(np.asarray(off, dtype=np.int64))


def uniform_offsets(B: int, per: int) -> np.ndarray:
    """Offsets [B+1] of a batch where every sample has ``per`` rows."""
    return np.arange(B + 1, dtype=np.int64) * per


def bf16_to_double(bits: int) -> float:
    return _load().oracle_bf16_to_double(int(bits))


def scores(q, k, q_off, k_off, H: int, Hkv: int, d: int, R: int, dtype: str = "bf16",
           scale: float | None = None, row_lse=None, row_reduce: int = ROWS_MAX) -> np.ndarray:
    """Scores of all keys: ``[sum_b (R + N_b)]`` float64, registers first per sample.

    One anchor row (T_b = 1) gives the CLS scores of Eq. EQ:CLS; several rows give the
    text scores of Eq. text_scoring (max over rows for visual keys, mean for registers),
    or with ``row_reduce=ROWS_MEAN`` the mutual scores of Eq. mutual_scoring (mean over
    rows for every key), each from the head-averaged softmax map.  ``scale`` defaults
    to 1/sqrt(d) (Eq. (1)).
    """
    lib = _load()
    q_off, k_off = _offsets(q_off), _offsets(k_off)
    B = len(q_off) - 1
    q = np.ascontiguousarray(q)
    k = np.ascontiguousarray(k)
    want = np.uint16 if dtype == "bf16" else np.float32
    if q.dtype != want or k.dtype != want:
        raise TypeError("q/k must be %s for dtype=%s" % (np.dtype(want).name, dtype))
    if q.size < q_off[-1] * H * d or k.size < k_off[-1] * Hkv * d:
        raise ValueError("q or k smaller than the offsets imply")
    lse = None
    if row_lse is not None:
        lse = np.ascontiguousarray(row_lse, dtype=np.float64)
        if lse.size < q_off[-1] * H:
            raise ValueError("row_lse smaller than sum(T_b) * H")
    out = np.empty(int(k_off[-1]), dtype=np.float64)
    sc = (1.0 / np.sqrt(d)) if scale is None else float(scale)
    rc = lib.oracle_scores(B, H, Hkv, d, R, _ptr(q_off), _ptr(k_off), _DTYPES[dtype],
                           _ptr(q), _ptr(k), sc, _ptr(lse), int(row_reduce), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_scores rejected the problem (rc=%d)" % rc)
    return out


def threshold(sc, k_off, R: int, lam: float, reduce: int = REG_MEAN) -> np.ndarray:
    """tau_b = lambda * s_b(r) (Eqs. stage1_threshold_appendix / stage2_set_appendix);
    with ``reduce=CAND_MEAN`` the ablation's mean-based threshold, lambda times the mean
    visual score (Table tab:qwen_compact_component_ablation)."""
    lib = _load()
    k_off = _offsets(k_off)
    B = len(k_off) - 1
    sc = np.ascontiguousarray(sc, dtype=np.float64)
    tau = np.empty(B, dtype=np.float64)
    rc = lib.oracle_threshold(B, R, _ptr(k_off), _ptr(sc), float(lam), int(reduce), _ptr(tau))
    if rc != 0:
        raise ValueError("oracle_threshold rejected the problem (rc=%d)" % rc)
    return tau


def select(sc, tau, k_off, R: int, index_map=None):
    """Ascending survivors ``s(v) >= tau`` per sample, packed: (kept_idx, count, offsets)."""
    lib = _load()
    k_off = _offsets(k_off)
    B = len(k_off) - 1
    sc = np.ascontiguousarray(sc, dtype=np.float64)
    tau = np.ascontiguousarray(tau, dtype=np.float64)
    ncand = int(k_off[-1] - R * B)
    im = None if index_map is None else np.ascontiguousarray(index_map, dtype=np.int32)
    kept = np.full(max(ncand, 1), -1, dtype=np.int32)
    cnt = np.zeros(B, dtype=np.int32)
    offs = np.zeros(B + 1, dtype=np.int32)
    rc = lib.oracle_select(B, R, _ptr(k_off), _ptr(sc), _ptr(tau), _ptr(im),
                           _ptr(kept), _ptr(cnt), _ptr(offs))
    if rc != 0:
        raise ValueError("oracle_select rejected the problem (rc=%d)" % rc)
    return kept[:offs[-1]].copy(), cnt, offs


def select_topk(sc, k_off, R: int, K: int, index_map=None):
    """Fixed-budget ablation (Table tab:qwen_compact_component_ablation): the K highest
    scores of each sample, lower index first among equal scores, listed ascending and
    packed: (kept_idx, count, offsets)."""
    lib = _load()
    k_off = _offsets(k_off)
    B = len(k_off) - 1
    sc = np.ascontiguousarray(sc, dtype=np.float64)
    ncand = int(k_off[-1] - R * B)
    im = None if index_map is None else np.ascontiguousarray(index_map, dtype=np.int32)
    kept = np.full(max(ncand, 1), -1, dtype=np.int32)
    cnt = np.zeros(B, dtype=np.int32)
    offs = np.zeros(B + 1, dtype=np.int32)
    rc = lib.oracle_select_topk(B, R, _ptr(k_off), _ptr(sc), int(K), _ptr(im), _ptr(kept),
                                _ptr(cnt), _ptr(offs))
    if rc != 0:
        raise ValueError("oracle_select_topk rejected the problem (rc=%d)" % rc)
    return kept[:offs[-1]].copy(), cnt, offs


def gather(src: np.ndarray, kept_idx, kept_offsets, k_off, R: int, src_pad_rows: int = 0,
           src_row0: int = 0) -> np.ndarray:
    """Byte copy of the survivors' rows of a 2-D row tensor ``src`` into a packed tensor.

    Sample b owns N_b + src_pad_rows consecutive rows of ``src``; its visual rows start
    at src_row0 (a visual-only hidden tensor: 0, 0; [registers ; visual] rows: R, R).
    """
    lib = _load()
    k_off = _offsets(k_off)
    B = len(k_off) - 1
    src = np.ascontiguousarray(src)
    kept_idx = np.ascontiguousarray(kept_idx, dtype=np.int32)
    kept_offsets = np.ascontiguousarray(kept_offsets, dtype=np.int32)
    rows = int(kept_offsets[-1])
    row_bytes = src.shape[1] * src.itemsize
    dst = np.zeros((rows, src.shape[1]), dtype=src.dtype)
    if rows == 0:
        return dst
    rc = lib.oracle_gather(B, R, _ptr(k_off), _ptr(src), int(src_pad_rows), int(src_row0),
                           row_bytes, _ptr(dst), row_bytes, row_bytes, _ptr(kept_idx),
                           _ptr(kept_offsets))
    if rc != 0:
        raise ValueError("oracle_gather rejected the problem (rc=%d)" % rc)
    return dst


def prune(q, k, q_off, k_off, H, Hkv, d, R, lam, dtype="bf16", reduce=REG_MEAN,
          scale=None, row_lse=None, index_map=None, row_reduce=ROWS_MAX):
    """All steps: returns dict(scores, tau, kept_idx, kept_count, kept_offsets)."""
    sc = scores(q, k, q_off, k_off, H, Hkv, d, R, dtype=dtype, scale=scale, row_lse=row_lse,
                row_reduce=row_reduce)
    tau = threshold(sc, k_off, R, lam, reduce)
    kept, cnt, offs = select(sc, tau, k_off, R, index_map=index_map)
    return {"scores": sc, "tau": tau, "kept_idx": kept, "kept_count": cnt, "kept_offsets": offs}


def neff(alpha) -> float:
    """n_eff = exp(-sum a ln a) of one attention distribution (Sec. 3.2, Obs. 1)."""
    a = np.ascontiguousarray(alpha, dtype=np.float64)
    return _load().oracle_neff(_ptr(a), a.size)


def register_reference(sc, k_off, R: int, reduce: int = REG_MEAN) -> np.ndarray:
    """s_b(r) per sample: the threshold at lambda = 1."""
    return threshold(sc, k_off, R, 1.0, reduce)


def ratios(sc, k_off, R: int, reduce: int = REG_MEAN):
    """Per sample, s(v) / s(r) for every visual token (list of arrays)."""
    k_off = _offsets(k_off)
    sr = register_reference(sc, k_off, R, reduce)
    return [np.asarray(sc[k_off[b] + R:k_off[b + 1]]) / sr[b] for b in range(len(k_off) - 1)]


def match_lambda(ratio_lists, k_target: float) -> float:
    """Budget matching (Eq. lambda2_budget_matching_appendix).

    The mean kept count over the calibration set, as a function of lambda, is a step
    function that changes only at the observed ratios s(v)/s(r).  Every distinct
    ratio is tried as a breakpoint; among the count levels the one closest to
    ``k_target`` wins (ties: the smaller count, i.e. the larger lambda), and the
    returned lambda is the geometric midpoint of that level's interval, so that
    rounding lambda to fp32 cannot move the count.
    """
    allr = np.concatenate([np.asarray(r, dtype=np.float64) for r in ratio_lists])
    D = len(ratio_lists)
    if allr.size == 0:
        return 1.0
    u = np.unique(allr)[::-1]                      # descending distinct ratios
    counts = np.searchsorted(np.sort(allr), u, side="left")
    counts = allr.size - counts                    # #{ratio >= u_i}
    err = np.abs(counts / D - float(k_target))
    best = int(np.flatnonzero(err == err.min())[0])  # first = largest lambda
    hi = u[best]
    lo = u[best + 1] if best + 1 < u.size else 0.0
    if lo > 0.0 and hi > 0.0:
        return float(np.sqrt(hi * lo))
    return float(hi * 0.5 if hi > 0 else 0.0)


def register_redirect(h, k_off, R: int, channels, reg_slot: int = 0, dtype: str = "bf16"):
    """Test-time register construction (Algorithm 1; Eq. register_redirect_appendix) on a
    copy of the activation tensor ``h`` ([rows, width], uint16 bf16 bits or float32).

    For every listed channel k and sample b, the register row ``reg_slot`` takes the max
    of channel k over the sample's visual rows and those rows' channel k becomes 0.
    Returns the new tensor."""
    lib = _load()
    k_off = _offsets(k_off)
    want = np.uint16 if dtype == "bf16" else np.float32
    out = np.array(h, dtype=want, copy=True, order="C")
    if out.ndim != 2 or out.shape[0] < k_off[-1]:
        raise ValueError("h must be [rows >= sum_b (R + N_b), width]")
    ch = np.ascontiguousarray(np.asarray(channels, dtype=np.int32))
    rc = lib.oracle_register_redirect(len(k_off) - 1, R, _ptr(k_off), _DTYPES[dtype], _ptr(out),
                                      out.shape[1], out.shape[1], _ptr(ch), int(ch.size),
                                      int(reg_slot))
    if rc != 0:
        raise ValueError("oracle_register_redirect rejected the problem (rc=%d)" % rc)
    return out
