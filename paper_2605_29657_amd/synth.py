"""Seeded synthetic inputs shaped like the paper's visual sequences.

This module builds inputs only: it draws Gaussian queries and keys, plants the
structure the pruning test is meant to react to (high-norm sink keys, keys
aligned with an anchor query, near-duplicate clusters, temporal repeats) and
rounds everything once to the workload's storage type.  It computes no
attention, score, threshold or selection.  The same bytes feed the GPU library
and the CPU oracle.

Randomness: every sample has its own ``numpy.random.Generator(Philox)`` keyed
by ``SeedSequence([0x0CCA7, workload id, split, seed, sample, stream])``, so a
sample's bytes do not depend on the batch size it is generated in.  Stream 0
draws the sample's shape and planted structure (shared by both stages), stream
1 the vision-stage tensors, stream 2 the text-stage tensors.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

from .workloads import WORKLOADS

_ROOT_KEY = 0x0CCA7


# ----------------------------------------------------------------------------- dtype helpers
def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit pattern (uint16), round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + r) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    return to_bf16_bits(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def _rng(wid: int, split: int, seed: int, b: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(
        np.random.SeedSequence([_ROOT_KEY, wid, split, seed, b, stream])))


# ----------------------------------------------------------------------------- data classes
@dataclass
class Payload:
    """A row tensor gathered with the survivors.

    Source row of visual token v of sample b: co_b + b * pad_rows + row0 + v,
    where co_b is the number of visual tokens of the samples before b.
    """
    name: str
    rows: np.ndarray          # [n_rows, width] (uint16 bf16 bits or float32)
    pad_rows: int
    row0: int


@dataclass
class StageBatch:
    """One stage's inputs for a batch: anchor queries, [registers ; visual] keys, payload."""
    workload: str
    stage: str                # "vis" (one CLS row) or "txt" (text rows)
    dtype: str
    B: int
    R: int
    H: int
    Hkv: int
    d: int
    T: np.ndarray             # [B] anchor rows per sample
    N: np.ndarray             # [B] visual candidates per sample
    q_off: np.ndarray         # [B+1] int64 prefix of T
    k_off: np.ndarray         # [B+1] int64 prefix of R + N
    q: np.ndarray             # [sum T, H, d]
    k: np.ndarray             # [sum (R+N), Hkv, d]
    payload: list = field(default_factory=list)
    sinks: list = field(default_factory=list)        # per sample: visual indices of planted sinks
    planted: list = field(default_factory=list)      # per sample: informative / relevant indices

    @property
    def ragged(self) -> bool:
        return bool(np.any(self.N != self.N[0]) or np.any(self.T != self.T[0]))

    @property
    def uniform_T(self) -> int:
        return int(self.T.max())

    @property
    def max_cands(self) -> int:
        return int(self.N.max())

    @property
    def max_rows(self) -> int:
        return int(self.T.max())


# ----------------------------------------------------------------------------- planting
def _unit(x: np.ndarray) -> np.ndarray:
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _aligned(rng, norm: np.ndarray, direction: np.ndarray, cos: float) -> np.ndarray:
    """Vectors of the given norms at exactly ``cos`` to ``direction`` (rows of unit vectors)."""
    dhat = _unit(direction)
    u = rng.standard_normal(dhat.shape, dtype=np.float32)
    u = u - np.sum(u * dhat, axis=-1, keepdims=True) * dhat
    u = _unit(u)
    return norm[..., None] * (cos * dhat + np.sqrt(1.0 - cos * cos) * u)


def _shape(w: dict, wid: int, split: int, seed: int, b: int) -> dict:
    """Per-sample shape and planted structure (shared by both stages)."""
    rng = _rng(wid, split, seed, b, 0)
    N = w["N"]
    if isinstance(N, tuple):
        lo, hi, step = N
        N = lo + step * int(rng.integers(0, (hi - lo) // step + 1))
    txt = w["txt"]
    T = txt["T"] if txt else 1
    if isinstance(T, tuple):
        T = int(rng.integers(T[0], T[1] + 1))
    ns = w["sinks"]
    if isinstance(ns, tuple):
        ns = int(rng.integers(ns[0], ns[1] + 1))
    ninf = int(round(w["informative"] * N / 576.0))
    nrel = int(rng.integers(w["relevant"][0], w["relevant"][1] + 1)) if w["relevant"] else 0
    perm = rng.permutation(N)
    sinks = np.sort(perm[:ns])
    informative = np.sort(perm[ns:ns + ninf])
    relevant = np.sort(perm[ns + ninf:ns + ninf + nrel])
    rel_row = rng.integers(0, T, size=nrel)
    protected = np.zeros(N, dtype=bool)
    protected[perm[:ns + ninf + nrel]] = True
    dups = []                              # (member index, source index)
    dup = w["dup"]
    if dup and dup[0] == "clusters":
        _, frac, clo, chi, _cos = dup
        free = [int(i) for i in perm[ns + ninf + nrel:]]
        target = int(round(frac * N))
        members = 0
        while members < target and len(free) >= 2:
            size = min(int(rng.integers(clo, chi + 1)), len(free), target - members)
            if size < 2:
                break
            grp = free[:size]
            free = free[size:]
            for m in grp[1:]:
                dups.append((m, grp[0]))
            members += size
    elif dup and dup[0] == "temporal":
        _, flen, frac, _cos = dup
        frames = N // flen
        for f in range(1, frames):
            pos = rng.permutation(flen)[:int(round(frac * flen))]
            for p in np.sort(pos):
                i = f * flen + int(p)
                if not protected[i] and not protected[i - flen]:
                    dups.append((i, i - flen))
    return dict(N=int(N), T=int(T), sinks=sinks, informative=informative,
                relevant=relevant, rel_row=rel_row, dups=dups)


def _stage_sample(w: dict, wid: int, split: int, seed: int, b: int, stage: str,
                  shp: dict, payload: bool) -> dict:
    cfg = w[stage]
    H, Hkv, d = cfg["H"], cfg["Hkv"], cfg["d"]
    R, N = w["R"], shp["N"]
    T = 1 if stage == "vis" else shp["T"]
    rng = _rng(wid, split, seed, b, 1 if stage == "vis" else 2)
    q = rng.standard_normal((T, H, d), dtype=np.float32)
    k = rng.standard_normal((R + N, Hkv, d), dtype=np.float32)
    kv = k[R:]                                        # visual keys (view)
    dupspec = w["dup"]
    if shp["dups"]:
        cos = dupspec[-1]
        mem = np.array([m for m, _ in shp["dups"]])
        # Sources are resolved in order, so a chain of repeats stays a chain.
        for m, s in shp["dups"]:
            nrm = np.linalg.norm(kv[m], axis=-1)
            kv[m] = _aligned(rng, nrm, kv[s], cos)
        del mem
    group = H // Hkv
    if stage == "vis" and len(shp["informative"]):
        idx = shp["informative"]
        nrm = np.linalg.norm(kv[idx], axis=-1)          # [n, Hkv]
        qdir = q[0][::group][None].repeat(len(idx), 0)  # CLS query of the first head of each group
        kv[idx] = _aligned(rng, nrm, qdir, 0.6)
    if stage == "txt" and len(shp["relevant"]):
        idx = shp["relevant"]
        nrm = np.linalg.norm(kv[idx], axis=-1)
        qdir = q[shp["rel_row"]][:, ::group]            # [n, Hkv, d]
        kv[idx] = _aligned(rng, nrm, qdir, 0.6)
    if len(shp["sinks"]):
        kv[shp["sinks"]] *= np.float32(w["sink_scale"])
    out = dict(q=_store(q, w["dtype"]), k=_store(k, w["dtype"]), T=T, N=N)
    if payload:
        hid = rng.standard_normal((N, cfg["hidden"]), dtype=np.float32)
        out["hidden"] = _store(hid, w["dtype"])
        if stage == "txt":
            v = rng.standard_normal((R + N, Hkv * d), dtype=np.float32)
            out["v"] = _store(v, w["dtype"])
    return out


def _workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _mutual_sample(w: dict, wid: int, split: int, seed: int, b: int, shp: dict,
                   payload: bool) -> dict:
    """The mutual-scoring Stage I of an encoder without a CLS row: the keys and payload
    of the vision stage, and one query row per register and visual token (their own
    query projections, drawn independently from stream 3)."""
    out = _stage_sample(w, wid, split, seed, b, "vis", shp, payload)
    cfg = w["vis"]
    rows = w["R"] + shp["N"]
    rng = _rng(wid, split, seed, b, 3)
    q = rng.standard_normal((rows, cfg["H"], cfg["d"]), dtype=np.float32)
    out["q"] = _store(q, w["dtype"])
    out["T"] = rows
    return out


def make_stage(name: str, stage: str, seed: int = 0, split: int = 0, B: int | None = None,
               payload: bool = True, samples=None) -> StageBatch:
    """Inputs of one stage of workload ``name``: "vis" (the CLS row, Stage I), "txt"
    (text rows, Stage II) or "mut" (every register and visual token as an anchor row,
    the mutual-scoring Stage I; the vision stage's keys).

    ``B`` limits the batch to its first B samples; ``samples`` picks explicit sample
    numbers instead (each sample's bytes depend only on its own number).
    """
    w = WORKLOADS[name]
    if stage == "txt" and w["txt"] is None:
        raise ValueError("workload %s has no text stage" % name)
    if stage not in ("vis", "txt", "mut"):
        raise ValueError("unknown stage %r" % stage)
    wid = w["id"]
    if samples is None:
        samples = list(range(w["B"] if B is None else B))
    samples = [int(s) for s in samples]
    shapes = [_shape(w, wid, split, seed, b) for b in samples]
    if stage == "mut":
        fn = lambda ib: _mutual_sample(w, wid, split, seed, ib[1], shapes[ib[0]], payload)
    else:
        fn = lambda ib: _stage_sample(w, wid, split, seed, ib[1], stage, shapes[ib[0]], payload)
    with ThreadPoolExecutor(_workers()) as ex:
        parts = list(ex.map(fn, list(enumerate(samples))))
    cfg = w["vis" if stage == "mut" else stage]
    R = w["R"]
    T = np.array([p["T"] for p in parts], dtype=np.int64)
    N = np.array([p["N"] for p in parts], dtype=np.int64)
    q_off = np.concatenate([[0], np.cumsum(T)]).astype(np.int64)
    k_off = np.concatenate([[0], np.cumsum(N + R)]).astype(np.int64)
    q = np.concatenate([p["q"] for p in parts], axis=0)
    k = np.concatenate([p["k"] for p in parts], axis=0)
    sb = StageBatch(workload=name, stage=stage, dtype=w["dtype"], B=len(samples), R=R,
                    H=cfg["H"], Hkv=cfg["Hkv"], d=cfg["d"], T=T, N=N, q_off=q_off,
                    k_off=k_off, q=q, k=k,
                    sinks=[s["sinks"] for s in shapes],
                    planted=[s["relevant"] if stage == "txt" else s["informative"]
                             for s in shapes])
    if payload:
        sb.payload.append(Payload("hidden", np.concatenate([p["hidden"] for p in parts], 0), 0, 0))
        if stage == "txt":
            sb.payload.append(Payload("k_rows", k.reshape(k.shape[0], -1), R, R))
            sb.payload.append(Payload("v_rows", np.concatenate([p["v"] for p in parts], 0), R, R))
    return sb


def keep_target(name: str, stage: str, N: float) -> float:
    """The calibration target mean kept count for a stage (absolute)."""
    w = WORKLOADS[name]
    t = w["keep1"] if stage == "vis" else w["keep2"]
    return float(t * N) if t < 1 else float(t)
