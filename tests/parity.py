"""Helpers shared by the GPU parity tests: run a stage on the GPU and on the oracle, compare.

Acceptance rules (from the method's definition, applied element by element):
  * scores: |gpu - oracle| <= rtol * |oracle| (rtol 1e-5 for float32 inputs, 2e-2 for
    bfloat16); oracle values below 1e-30 only need |gpu| < 1e-29;
  * tau: the same relative bound;
  * survivor sets: identical except for tokens whose oracle score lies within
    rtol * max(tau, score) of the oracle threshold (either decision is correct there);
  * survivor lists: strictly ascending, in range, offsets = exclusive prefix of counts;
  * gathered rows: byte-equal to the source rows at the GPU's own indices.
"""
from __future__ import annotations

import json
import os

import numpy as np

import oracle
from paper_2605_29657_amd import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
# The acceptance tolerance on scores and tau (float32 / bfloat16 inputs).
RTOL = {"f32": 1e-5, "bf16": 2e-2}
# Regression guard, tighter than the acceptance tolerance: every path computes in float32
# with fixed reduction orders and shows ~1e-6 relative error against the float64 oracle,
# so an error above 1e-4 means something regressed even where the 2e-2 contract holds.
GUARD = {"f32": 1e-5, "bf16": 1e-4}
# At most this many tokens of a sample may differ in their keep decision (each within the
# guard band of tau).
MAX_EXEMPT_PER_SAMPLE = 2


def lambdas() -> dict:
    with open(os.path.join(GOLDEN, "lambdas.json")) as f:
        return json.load(f)


def lam_for(name: str, stage: str) -> float:
    return float(np.float32(lambdas()[name][stage]["lam"]))


def f32_scale(d: int) -> float:
    """The library's default temperature: float32 1/sqrtf(d), widened exactly."""
    return float(np.float32(1.0) / np.sqrt(np.float32(d)))


def oracle_prune(sb: synth.StageBatch, lam: float, reduce: int = oracle.REG_MEAN, row_lse=None,
                 index_map=None) -> dict:
    rr = oracle.ROWS_MEAN if sb.stage == "mut" else oracle.ROWS_MAX
    return oracle.prune(sb.q, sb.k, sb.q_off, sb.k_off, sb.H, sb.Hkv, sb.d, sb.R, lam,
                        dtype=sb.dtype, reduce=reduce, scale=f32_scale(sb.d), row_lse=row_lse,
                        index_map=index_map, row_reduce=rr)


def guard_for(rtol: float) -> float:
    """The regression guard that goes with an acceptance tolerance."""
    return GUARD["f32"] if rtol <= RTOL["f32"] else GUARD["bf16"]


def check_scores(g: np.ndarray, o: np.ndarray, rtol: float, what: str = "scores") -> float:
    """|gpu - oracle| <= rtol |oracle| (the acceptance rule), and the regression guard."""
    g = np.asarray(g, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    assert g.shape == o.shape, (what, g.shape, o.shape)
    assert np.all(np.isfinite(g)), what + ": non-finite GPU values"
    tiny = np.abs(o) < 1e-30
    err = np.abs(g - o)
    rel = np.where(tiny, 0.0, err / np.where(tiny, 1.0, np.abs(o)))
    worst = int(np.argmax(rel)) if rel.size else 0
    assert np.all(rel <= rtol), "%s: max rel err %.3g at %d (gpu %r oracle %r)" % (
        what, rel[worst], worst, g[worst], o[worst])
    guard = guard_for(rtol)
    assert np.all(rel <= guard), "%s: max rel err %.3g at %d exceeds the regression guard %g" % (
        what, rel[worst], worst, guard)
    assert np.all(np.abs(g[tiny]) < 1e-29), what + ": tiny oracle values not reproduced"
    return float(rel.max()) if rel.size else 0.0


def check_bookkeeping(g: dict, sb: synth.StageBatch, ascending: bool = True):
    """Offsets are the exclusive prefix of the counts; each list is ascending and in range."""
    offs, cnt = np.asarray(g["kept_offsets"]), np.asarray(g["kept_count"])
    assert offs.shape == (sb.B + 1,) and cnt.shape == (sb.B,)
    assert offs[0] == 0 and np.array_equal(np.diff(offs), cnt)
    assert np.all(cnt >= 0) and np.all(cnt <= sb.N)
    kept = np.asarray(g["kept_idx"])
    assert kept.size == offs[-1]
    if ascending:
        for b in range(sb.B):
            seg = kept[offs[b]:offs[b + 1]]
            assert np.all(np.diff(seg) > 0), "sample %d: survivors not strictly ascending" % b
            assert np.all((seg >= 0) & (seg < sb.N[b])), "sample %d: index out of range" % b


def check_selection(g: dict, o: dict, sb: synth.StageBatch, rtol: float, index_map=None) -> dict:
    """Survivor-set rule + bookkeeping.  Returns counts of exempt differences.

    A token may be decided differently only if its oracle score lies within rtol of the
    oracle tau (the acceptance rule); as a regression guard it must also lie within the
    guard band, and a sample may have at most MAX_EXEMPT_PER_SAMPLE such tokens."""
    B, R = sb.B, sb.R
    check_bookkeeping(g, sb, ascending=index_map is None)
    offs = np.asarray(g["kept_offsets"])
    kept = np.asarray(g["kept_idx"])
    co = np.concatenate([[0], np.cumsum(sb.N)])
    o_off = o["kept_offsets"]
    exempt = 0
    for b in range(B):
        seg = kept[offs[b]:offs[b + 1]]
        oseg = o["kept_idx"][o_off[b]:o_off[b + 1]]
        diff = set(seg.tolist()) ^ set(oseg.tolist())
        if diff:
            s_o = o["scores"][sb.k_off[b] + R:sb.k_off[b + 1]]
            tau = o["tau"][b]
            if index_map is not None:
                inv = {int(index_map[co[b] + v]): v for v in range(sb.N[b])}
                diff = {inv[x] for x in diff}
            guard = guard_for(rtol)
            for v in diff:
                band = rtol * max(tau, s_o[v])
                assert abs(s_o[v] - tau) <= band, (
                    "sample %d token %d: decision differs outside the tolerance band "
                    "(score %r, tau %r)" % (b, v, s_o[v], tau))
                assert abs(s_o[v] - tau) <= guard * max(tau, s_o[v]), (
                    "sample %d token %d: decision differs outside the regression guard band "
                    "(score %r, tau %r)" % (b, v, s_o[v], tau))
            assert len(diff) <= MAX_EXEMPT_PER_SAMPLE, (
                "sample %d: %d tokens decided differently" % (b, len(diff)))
            exempt += len(diff)
    return {"exempt": exempt, "kept": int(offs[-1])}


def check_rows(g: dict, sb: synth.StageBatch, which=None):
    """Gathered rows are byte copies of the source rows at the GPU's survivor indices."""
    for i, pl in enumerate(sb.payload):
        if which is not None and pl.name not in which:
            continue
        want = oracle.gather(pl.rows, g["kept_idx"], g["kept_offsets"], sb.k_off, sb.R,
                             src_pad_rows=pl.pad_rows, src_row0=pl.row0)
        got = g["rows"][i]
        assert got.shape == want.shape, (pl.name, got.shape, want.shape)
        assert np.array_equal(got.view(np.uint8), want.view(np.uint8)), pl.name + " rows differ"


def custom_stage(B, R, H, Hkv, d, T, N, dtype="bf16", seed=0, hidden=64, sinks=2,
                 sink_scale=8.0, stage=None) -> synth.StageBatch:
    """A small hand-shaped batch (edge cases) with Gaussian q/k, a few sinks and payload rows."""
    rng = np.random.default_rng(seed)
    T = np.asarray(T, dtype=np.int64)
    N = np.asarray(N, dtype=np.int64)
    q_off = np.concatenate([[0], np.cumsum(T)]).astype(np.int64)
    k_off = np.concatenate([[0], np.cumsum(N + R)]).astype(np.int64)
    q = rng.standard_normal((int(q_off[-1]), H, d)).astype(np.float32)
    k = rng.standard_normal((int(k_off[-1]), Hkv, d)).astype(np.float32)
    for b in range(B):
        if N[b] > 0:
            idx = rng.choice(N[b], size=min(sinks, int(N[b])), replace=False)
            k[k_off[b] + R + idx] *= np.float32(sink_scale)
    store = (lambda x: synth.to_bf16_bits(x)) if dtype == "bf16" else (lambda x: x)
    if stage is None:
        stage = "txt" if T.max() > 1 else "vis"
    sb = synth.StageBatch(workload="custom", stage=stage, dtype=dtype,
                          B=B, R=R, H=H, Hkv=Hkv, d=d, T=T, N=N, q_off=q_off, k_off=k_off,
                          q=store(q), k=store(k))
    hid = store(rng.standard_normal((int(N.sum()), hidden)).astype(np.float32))
    sb.payload.append(synth.Payload("hidden", hid, 0, 0))
    sb.payload.append(synth.Payload("k_rows", sb.k.reshape(sb.k.shape[0], -1), R, R))
    return sb
