"""Throughput of the fused register-anchored prune on one MI355X.

One step = the whole pruning path over one batch of the LLaVA-NeXT-shaped workload
(B=32 images, 2880 visual tokens + 4 registers each, bfloat16):
  Stage I   occam_prune with the CLS row (H=16, d=64): scores, tau, survivors, and
            the gather of the survivors' 1024-wide vision hidden rows;
  Stage II  occam_prune with 128 text rows (H=32, d=128) over all 2880 visual tokens:
            scores, tau, survivors, and the gather of their 4096-wide LLM hidden rows
            and their key and value rows (32 x 128 each).
Inputs are resident in HBM before timing starts.  lambda_1 / lambda_2 come from the
budget matching of tests/golden/lambdas.json (523 and 40 kept tokens on average).

Prints one JSON line: images/s, whole-step algorithmic HBM GB/s, the roofline entry of
the dominant kernel (the Stage II scoring kernel, timed alone with HIP events on the
stream it runs on) and the oracle's CPU throughput on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, datasheet
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16, datasheet
# v_exp_f32 issue rate: 8 lanes per clock per SIMD x 1024 SIMDs x 2.4 GHz (a probe on the
# MI355X measured 18.8 T/s).
EXP_PEAK_TPS = 8 * 1024 * 2.4e9 / 1e12


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def settle(torch, fn, seconds: float = 0.05, min_calls: int = 10):
    """Untimed calls until ~`seconds` of GPU work have run (at least min_calls): after
    host-side set-up the GPU has idled, and its first calls run at lower clocks."""
    n, t0 = 0, time.perf_counter()
    while n < min_calls or time.perf_counter() - t0 < seconds:
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
        n += 5
        if n >= 2000:
            break
    return n


# Input copies that consecutive timed calls cycle through.  Each copy has its own input,
# output and workspace buffers, so a call never reads keys that the call before it left in
# the 256 MB memory-side cache, as with a batch of new images every step; three copies keep
# the working set between two uses of one copy above the cache's size at every shape here.
NCOPY = 3


def cycler(fns):
    """One callable that runs fns[0], fns[1], ..., fns[-1], fns[0], ... in turn."""
    it = [0]

    def one():
        fns[it[0] % len(fns)]()
        it[0] += 1
    return one


def stage_bytes(sb, kept_per_sample) -> dict:
    """Algorithmic HBM bytes of one fused prune over a batch.

    keys: every key row once; queries once; scores written once (4 B per key);
    gather: each survivor row read and written once; survivor lists 4 B each.
    """
    e = 2 if sb.dtype == "bf16" else 4
    keys = int(sb.k_off[-1]) * sb.Hkv * sb.d * e
    qry = int(sb.q_off[-1]) * sb.H * sb.d * e
    score_w = int(sb.k_off[-1]) * 4
    row_bytes = sum(pl.rows.shape[1] * pl.rows.itemsize for pl in sb.payload)
    kept = int(np.sum(kept_per_sample))
    gather = 2 * kept * row_bytes + 4 * kept
    return dict(keys=keys, q=qry, scores=score_w, gather=gather,
                total=keys + qry + score_w + gather)


def cpu_model() -> str:
    """The host CPU's model name (first entry of /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _gomp():
    """libgomp, the OpenMP runtime the C oracle is linked against (thread count control)."""
    import ctypes
    try:
        return ctypes.CDLL("libgomp.so.1")
    except OSError:
        return None


def _oracle_images(name, lam1, lam2, budget_s, max_samples):
    """The oracle over the first images of the workload, both stages, until ~budget_s:
    (images, seconds)."""
    import oracle
    from paper_2605_29657_amd import synth
    done, t_total = 0, 0.0
    while done < max_samples and t_total < budget_s:
        vis = synth.make_stage(name, "vis", samples=[done])
        txt = synth.make_stage(name, "txt", samples=[done])
        t0 = time.perf_counter()
        for sb, lam in ((vis, lam1), (txt, lam2)):
            scale = float(np.float32(1.0) / np.sqrt(np.float32(sb.d)))
            res = oracle.prune(sb.q, sb.k, sb.q_off, sb.k_off, sb.H, sb.Hkv, sb.d, sb.R, lam,
                               dtype=sb.dtype, scale=scale)
            for pl in sb.payload:
                oracle.gather(pl.rows, res["kept_idx"], res["kept_offsets"], sb.k_off, sb.R,
                              src_pad_rows=pl.pad_rows, src_row0=pl.row0)
        t_total += time.perf_counter() - t0
        done += 1
    return done, t_total


def cpu_baseline(name, lam1, lam2, budget_s=12.0, budget_1t_s=8.0, max_samples=256):
    """The oracle on the host cores over the first images of the workload (~budget_s), then
    again on one thread (~budget_1t_s).  The oracle runs one image per call with OpenMP over
    its anchor rows: the Stage II text rows (128 per image) spread over every thread, the
    Stage I CLS row runs on one."""
    import oracle
    oracle.build()
    gomp = _gomp()
    threads = int(gomp.omp_get_max_threads()) if gomp else int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    done, t_total = _oracle_images(name, lam1, lam2, budget_s, max_samples)
    out = {"value": done / t_total, "unit": "images/s", "cores": threads, "kind": "oracle",
           "sample": "first %d image(s) of %s, both stages (scores, tau, survivors, gather), "
                     "%.1f s, OpenMP over each image's anchor rows" % (done, name, t_total),
           "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
           "omp_num_threads_env": os.environ.get("OMP_NUM_THREADS")}
    if gomp:
        gomp.omp_set_num_threads(1)
        d1, t1 = _oracle_images(name, lam1, lam2, budget_1t_s, max_samples)
        gomp.omp_set_num_threads(threads)
        out["one_thread"] = {"value": d1 / t1, "unit": "images/s", "cores": 1,
                             "sample": "first %d image(s), %.1f s" % (d1, t1)}
    return out


def mutual_stage1(torch, steps: int, warmup: int, with_cpu: bool) -> dict:
    """The mutual-scoring Stage I (Eq. mutual_scoring) on the Qwen3-VL-shaped batch: every
    register and visual token is an anchor row.  Fused prune with the hidden-row gather,
    timed alone; its work is (R+N)^2 * H * d per sample, so it is graded against the bf16
    MFMA peak (algorithmic flops count one Q K^T).  The calls cycle through NCOPY input
    copies."""
    import oracle
    from paper_2605_29657_amd import synth
    from paper_2605_29657_amd.runner import DeviceStage
    name = "qwen3vl_ragged"
    with open(os.path.join(ROOT, "tests", "golden", "lambdas.json")) as f:
        lam = float(np.float32(json.load(f)[name]["mut"]["lam"]))
    sb = synth.make_stage(name, "mut")
    dss = [DeviceStage(sb, ragged=True) for _ in range(NCOPY)]
    ds = dss[0]
    call = cycler([(lambda d=d: d.prune(lam)) for d in dss])
    for _ in range(warmup):
        call()
    settle(torch, call)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    flops = float(np.sum(2.0 * sb.T.astype(np.float64) * (sb.N + sb.R) * sb.H * sb.d))
    # One exponential per (anchor row, key, head) in each of the two passes over the keys.
    exps = float(np.sum(2.0 * sb.T.astype(np.float64) * (sb.N + sb.R) * sb.H))
    kept = ds.out["kept_count"].cpu().numpy()
    out = {"workload": "%s mutual Stage I: B=%d, N in [%d, %d], all R+N tokens as anchor rows, "
                       "H=%d d=%d, hidden gather" % (name, sb.B, int(sb.N.min()), int(sb.N.max()),
                                                     sb.H, sb.d),
           "ms": round(ms, 4), "images_s": round(sb.B / (ms * 1e-3), 1),
           "mfma_tflops": round(flops / (ms * 1e-3) / 1e12, 1),
           "mfma_frac": round(flops / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
           "exp_per_s": round(exps / (ms * 1e-3) / 1e12, 2), "exp_unit": "T/s",
           "exp_frac": round(exps / (ms * 1e-3) / 1e12 / EXP_PEAK_TPS, 4),
           "lambda1": lam, "kept_mean": float(np.mean(kept))}
    if with_cpu:
        done, spent = 0, 0.0
        while done < 16 and spent < 10.0:
            one = synth.make_stage(name, "mut", samples=[done])
            t0 = time.perf_counter()
            scale = float(np.float32(1.0) / np.sqrt(np.float32(one.d)))
            res = oracle.prune(one.q, one.k, one.q_off, one.k_off, one.H, one.Hkv, one.d, one.R,
                               lam, dtype=one.dtype, scale=scale, row_reduce=oracle.ROWS_MEAN)
            oracle.gather(one.payload[0].rows, res["kept_idx"], res["kept_offsets"], one.k_off,
                          one.R)
            spent += time.perf_counter() - t0
            done += 1
        out["cpu_baseline"] = {"value": round(done / spent, 3), "unit": "images/s",
                               "cores": int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1)),
                               "kind": "oracle",
                               "sample": "first %d image(s) of %s, mutual scores, tau, survivors, "
                                         "gather, %.1f s" % (done, name, spent)}
    return out


def cls_f32_latency(torch, reps: int = 200) -> dict:
    """Latency of one fused prune of the LLaVA-1.5 CLS row in float32 (B = 1, 4 registers +
    576 visual keys, H = 16, d = 64, 1024-wide f32 hidden gather): HIP events around every
    call on the launch stream, the calls enqueued back to back."""
    from paper_2605_29657_amd import synth
    from paper_2605_29657_amd.runner import DeviceStage
    name = "llava15_cls_f32"
    with open(os.path.join(ROOT, "tests", "golden", "lambdas.json")) as f:
        lam = float(np.float32(json.load(f)[name]["vis"]["lam"]))
    sb = synth.make_stage(name, "vis")
    ds = DeviceStage(sb, ragged=sb.ragged)
    for _ in range(50):
        ds.prune(lam)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    # A GPU-side wait holds the stream while the host enqueues every call, so the events
    # time the device alone, not the host's enqueue rate.
    torch.cuda._sleep(int(5e7))
    for a, b in ev:
        a.record()
        ds.prune(lam)
        b.record()
    torch.cuda.synchronize()
    us = sorted(a.elapsed_time(b) * 1e3 for a, b in ev)
    return {"workload": "%s: B=%d, R=%d, N=%d, H=%d, d=%d, f32, %d-wide hidden gather" % (
                name, sb.B, sb.R, int(sb.N[0]), sb.H, sb.d, sb.payload[0].rows.shape[1]),
            "how": "HIP events around each call on the launch stream; the calls are enqueued "
                   "behind a GPU-side wait, so host enqueue time is excluded",
            "median_us": round(us[len(us) // 2], 2), "mean_us": round(float(np.mean(us)), 2),
            "min_us": round(us[0], 2), "calls": reps,
            "kept": int(ds.out["kept_count"][0].item())}


def register_redirect_bench(torch, reps: int = 20) -> dict:
    """Test-time register construction (Eq. register_redirect_appendix) at the LLaVA-NeXT
    vision shape: 32 images x (4 registers + 2880 patches) rows of a 4096-wide bf16 MLP
    activation, ten register channels.  Each channel element sits in its own 8 KB row,
    so the call is bound by latency and cache-line traffic, not by its few bytes."""
    from paper_2605_29657_amd import occam
    B, R, N, width = 32, 4, 2880, 4096
    h = torch.randn((B * (R + N), width), device="cuda").to(torch.bfloat16)
    chans = torch.tensor(np.random.default_rng(0).choice(width, 10, replace=False).astype(np.int32),
                         device="cuda")
    p = occam.Problem(B, 16, 16, 64, R, cands=N, dtype="bf16")
    occam.register_redirect(p, h, chans)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        occam.register_redirect(p, h, chans)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    alg = B * 10 * (2 * N * 2 + 2)           # read + zero each visual value, write the register
    lines = B * 10 * (R + N) * 128            # one 128-byte line per touched row and channel
    del h
    return {"workload": "B=%d, %d rows x %d bf16, 10 channels" % (B, R + N, width),
            "us": round(ms * 1e3, 2), "algorithmic_bytes": alg, "line_bytes": lines,
            "line_gbs": round(lines / (ms * 1e-3) / 1e9, 1)}


def budget_matching_bench(torch, reps: int = 20) -> dict:
    """Budget matching (Eq. lambda2_budget_matching_appendix) over a calibration set of 64
    LLaVA-NeXT samples (4 registers + 2880 candidates each, 184,320 ratios) at a target of
    576 kept per sample.  Scores are log-normal with a register score near the top, the
    shape the text scores take.  One workgroup runs the whole selection, so the call is
    bound by that workgroup's passes over the ratios, not by HBM."""
    from paper_2605_29657_amd import occam
    B, R, N = 64, 4, 2880
    g = torch.Generator(device="cuda").manual_seed(0)
    sc = torch.exp(torch.randn((B, R + N), device="cuda", generator=g) * 1.5) * 0.02
    sc[:, :R] = 0.3
    sc = sc.reshape(-1).contiguous()
    p = occam.Problem(B, 16, 16, 64, R, cands=N, dtype="bf16")
    ws = occam.workspace(p)
    out = torch.empty(2, dtype=torch.float32, device="cuda")
    occam.match_lambda(p, sc, 576.0, out[0:1], ws, mean_kept=out[1:2])
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        occam.match_lambda(p, sc, 576.0, out[0:1], ws, mean_kept=out[1:2])
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    lam, kept = out.cpu().tolist()
    return {"workload": "calibration set B=%d x %d candidates, K_tar=576" % (B, N),
            "us": round(ms * 1e3, 2), "lambda": lam, "mean_kept": kept,
            "ratios_per_us": round(B * N / (ms * 1e3), 1)}


def ablation_steps(torch, dvs, dts, k1: float, k2: float, steps: int) -> dict:
    """The component ablation's two threshold variants (Table
    tab:qwen_compact_component_ablation) on the headline batch, each at the register
    rule's mean budgets k1 / k2 (the paper compares variants at matched retention):

    * mean threshold: lambda matched on the device (occam_match_lambda with the mean
      visual score as reference) to k1 / k2, then the same fused prune of both stages;
    * fixed budget: occam_score, occam_select_topk with K = round(k1) / round(k2), and
      occam_gather of the same rows.

    Both steps cycle through the input copies dvs / dts (Stage I / Stage II).
    """
    from paper_2605_29657_amd import occam
    dv, dt = dvs[0], dts[0]
    lam = torch.empty(2, dtype=torch.float32, device="cuda")
    mk = torch.empty(2, dtype=torch.float32, device="cuda")
    for i, (ds, k) in enumerate(((dv, k1), (dt, k2))):
        occam.score(ds.problem, ds.q, ds.k, ds.out["scores"], ds.ws)
        occam.match_lambda(ds.problem, ds.out["scores"], k, lam[i:i + 1], ds.ws,
                           mean_kept=mk[i:i + 1], reduce=occam.REF_CAND_MEAN)
    lam1, lam2 = lam.cpu().tolist()
    K1, K2 = int(round(k1)), int(round(k2))

    mean_step = cycler([(lambda a=a, b=b: (a.prune(lam1, reduce=occam.REF_CAND_MEAN),
                                           b.prune(lam2, reduce=occam.REF_CAND_MEAN)))
                        for a, b in zip(dvs, dts)])

    def topk(ds, K):
        o = ds.out
        occam.score(ds.problem, ds.q, ds.k, o["scores"], ds.ws)
        occam.select_topk(ds.problem, o["scores"], K, o["kept_idx"], o["kept_count"],
                          o["kept_offsets"], ds.ws)
        occam.gather(ds.problem, ds.rows, o["kept_idx"], o["kept_offsets"])

    topk_step = cycler([(lambda a=a, b=b: (topk(a, K1), topk(b, K2))) for a, b in zip(dvs, dts)])

    def timed(fn, n):
        settle(torch, fn)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    B = dv.sb.B
    ms_mean = timed(mean_step, steps)
    kept_mean = (float(dv.out["kept_count"].float().mean()), float(dt.out["kept_count"].float().mean()))
    ms_topk = timed(topk_step, steps)
    sel_us = timed(lambda: occam.select_topk(dt.problem, dt.out["scores"], K2, dt.out["kept_idx"],
                                             dt.out["kept_count"], dt.out["kept_offsets"], dt.ws),
                   steps) * 1e3
    thr_us = timed(lambda: occam.select(dt.problem, dt.out["scores"], dt.out["tau"],
                                        dt.out["kept_idx"], dt.out["kept_count"],
                                        dt.out["kept_offsets"], dt.ws), steps) * 1e3
    return {"mean_threshold": {"lambda1": lam1, "lambda2": lam2,
                               "kept_stage1_mean": kept_mean[0], "kept_stage2_mean": kept_mean[1],
                               "ms_per_step": round(ms_mean, 4),
                               "images_s": round(B / (ms_mean * 1e-3), 1)},
            "fixed_budget": {"K1": K1, "K2": K2, "ms_per_step": round(ms_topk, 4),
                             "images_s": round(B / (ms_topk * 1e-3), 1),
                             "select_topk_stage2_us": round(sel_us, 2),
                             "select_threshold_stage2_us": round(thr_us, 2)}}


def chained_stage(txt, kept_idx, kept_offsets):
    """Stage II over the tokens Stage I kept: per sample the R register rows and the
    kept visual rows of the text-stage keys and payload, in Stage I's ascending order."""
    from paper_2605_29657_amd import synth
    B, R = txt.B, txt.R
    n1 = np.diff(kept_offsets).astype(np.int64)
    co = np.concatenate([[0], np.cumsum(txt.N)])
    krows, vis_rows = [], []
    for b in range(B):
        kept = kept_idx[kept_offsets[b]:kept_offsets[b + 1]].astype(np.int64)
        krows.append(txt.k_off[b] + np.arange(R))
        krows.append(txt.k_off[b] + R + kept)
        vis_rows.append((b, kept))
    krows = np.concatenate(krows)
    payload = []
    for pl in txt.payload:
        sel = []
        for b, kept in vis_rows:
            base = co[b] + b * pl.pad_rows
            if pl.pad_rows:
                sel.append(base + np.arange(pl.pad_rows))
            sel.append(base + pl.row0 + kept)
        payload.append(synth.Payload(pl.name, pl.rows[np.concatenate(sel)], pl.pad_rows, pl.row0))
    return synth.StageBatch(workload=txt.workload, stage=txt.stage, dtype=txt.dtype, B=B, R=R,
                            H=txt.H, Hkv=txt.Hkv, d=txt.d, T=txt.T, N=n1, q_off=txt.q_off,
                            k_off=np.concatenate([[0], np.cumsum(R + n1)]).astype(np.int64),
                            q=txt.q, k=txt.k[krows], payload=payload)


def stage_breakdown(torch, dvs, dts, txt, lam1: float, lam2: float, steps: int) -> dict:
    """Each stage alone, and the chained pipeline: Stage II over the R + N1 tokens that
    Stage I kept (its keys and payload rows staged untimed), index_map = Stage I's
    indices, so that Stage II reports original token indices.  Every timing cycles
    through input copies (dvs / dts for the two stages)."""
    from paper_2605_29657_amd.runner import DeviceStage
    from paper_2605_29657_amd import occam

    def timed(fn, n):
        settle(torch, fn)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    def input_bytes(ds):
        return (int(ds.q.numel() + ds.k.numel()) * ds.k.element_size() +
                sum(int(r.numel()) * r.element_size() for r in ds.row_src))

    dv, dt = dvs[0], dts[0]
    B = dv.sb.B
    ms1 = timed(cycler([(lambda d=d: d.prune(lam1)) for d in dvs]), steps)
    ms2 = timed(cycler([(lambda d=d: d.prune(lam2)) for d in dts]), steps)
    b1 = stage_bytes(dv.sb, dv.out["kept_count"].cpu().numpy())["total"]
    b2 = stage_bytes(dt.sb, dt.out["kept_count"].cpu().numpy())["total"]
    # Stage I scoring alone (occam_score: the one-row logits with online statistics, then
    # the scores): reads every key once, writes one score per key.
    scs = [torch.empty_like(dv.out["scores"]) for _ in dvs]
    ms1s = timed(cycler([(lambda d=d, o=o: occam.score(d.problem, d.q, d.k, o, d.ws))
                         for d, o in zip(dvs, scs)]), steps)
    del scs
    e1 = 2 if dv.sb.dtype == "bf16" else 4
    bs1 = int(dv.sb.k_off[-1]) * (dv.sb.Hkv * dv.sb.d * e1 + 4) + int(dv.sb.q_off[-1]) * dv.sb.H * dv.sb.d * e1
    kept_idx = dv.out["kept_idx"].cpu().numpy()
    kept_off = dv.out["kept_offsets"].cpu().numpy()
    ch = chained_stage(txt, kept_idx, kept_off)
    # Every sample keeps its T text rows; only the key counts are ragged.
    dcs = [DeviceStage(ch, ragged=True, row_offsets=not bool(np.all(ch.T == ch.T[0])))
           for _ in range(len(dts))]
    imap = dv.out["kept_idx"][:int(kept_off[-1])].clone()
    ms2c = timed(cycler([(lambda d=d: d.prune(lam2, index_map=imap)) for d in dcs]), steps)
    kept2c = dcs[0].out["kept_count"].float().mean().item()
    # The gathers alone (occam_gather over each copy's kept lists: the same pack_gather
    # kernel), next to a plain contiguous device copy of the same bytes, the copy's source
    # and destination cycling through enough buffers (>= 1.2 GB) that the memory-side
    # cache holds none of them.
    def gather_vs_copy(dss):
        sb = dss[0].sb
        kept = dss[0].out["kept_count"].cpu().numpy()
        nbytes = (stage_bytes(sb, kept)["gather"] - 4 * int(kept.sum())) // 2
        us = timed(cycler([(lambda d=d: occam.gather(d.problem, d.rows, d.out["kept_idx"],
                                                      d.out["kept_offsets"])) for d in dss]),
                   steps) * 1e3
        nb = max(3, -(-1200 * 10**6 // max(nbytes, 1)))
        bufs = [(torch.empty(nbytes, dtype=torch.uint8, device="cuda"),
                 torch.empty(nbytes, dtype=torch.uint8, device="cuda")) for _ in range(nb)]
        cus = timed(cycler([(lambda a=a, b=b: b.copy_(a)) for a, b in bufs]), steps) * 1e3
        del bufs
        return {"row_bytes_read": nbytes, "gather_us": round(us, 2), "copy_us": round(cus, 2),
                "gather_tbs": round(2 * nbytes / (us * 1e-6) / 1e12, 2),
                "copy_tbs": round(2 * nbytes / (cus * 1e-6) / 1e12, 2),
                "gather_vs_copy": round(cus / us, 3)}

    gathers = {"stage1": gather_vs_copy(dvs), "stage2": gather_vs_copy(dts),
               "how": "occam_gather alone (the pack_gather kernel) against a contiguous device "
                      "copy of the same bytes; TB/s count reads + writes"}
    rot = "each timing cycles through %d input copies (Stage I %d MB, Stage II %d MB, " \
          "chained Stage II %d MB of inputs in all)" % (
              len(dvs), sum(map(input_bytes, dvs)) // 10**6, sum(map(input_bytes, dts)) // 10**6,
              sum(map(input_bytes, dcs)) // 10**6)
    del dcs
    gbs = lambda nbytes, ms: nbytes / (ms * 1e-3) / 1e9
    return {"stage1_ms": round(ms1, 4), "stage2_ms": round(ms2, 4),
            "stage1_hbm_gbs": round(gbs(b1, ms1), 1),
            "stage1_hbm_frac": round(gbs(b1, ms1) / HBM_PEAK_GBS, 4),
            "stage2_hbm_gbs": round(gbs(b2, ms2), 1),
            "stage2_hbm_frac": round(gbs(b2, ms2) / HBM_PEAK_GBS, 4),
            "stage1_score": {"ms": round(ms1s, 4), "bytes": bs1,
                             "hbm_gbs": round(gbs(bs1, ms1s), 1),
                             "hbm_frac": round(gbs(bs1, ms1s) / HBM_PEAK_GBS, 4)},
            "rotation": rot,
            "gathers": gathers,
            "chained": {"stage2_keys_mean": float(np.mean(ch.N + ch.R)),
                        "stage2_ms": round(ms2c, 4), "step_ms": round(ms1 + ms2c, 4),
                        "images_s": round(B / ((ms1 + ms2c) * 1e-3), 1),
                        "kept_stage2_mean": kept2c}}


def workload_step(torch, name: str, steps: int) -> dict:
    """The headline step (Stage I prune + Stage II prune over all tokens) on another
    workload shape: images/s, the step's algorithmic bytes over its time, and the text
    stage's algorithmic MFMA rate (one Q K^T) over the step; then the text stage alone
    (its Q K^T rate, and with both passes' Q K^T), also for the samples with at least 312
    text rows when the batch mixes row counts.  Every timing cycles through NCOPY input
    copies."""
    from paper_2605_29657_amd import synth
    from paper_2605_29657_amd.runner import DeviceStage
    with open(os.path.join(ROOT, "tests", "golden", "lambdas.json")) as f:
        lams = json.load(f)[name]
    lam1 = float(np.float32(lams["vis"]["lam"]))
    lam2 = float(np.float32(lams["txt"]["lam"]))
    vis = synth.make_stage(name, "vis")
    txt = synth.make_stage(name, "txt")
    dvs = [DeviceStage(vis, ragged=vis.ragged) for _ in range(NCOPY)]
    dts = [DeviceStage(txt, ragged=txt.ragged) for _ in range(NCOPY)]
    dv, dt = dvs[0], dts[0]
    step = cycler([(lambda a=a, b=b: (a.prune(lam1), b.prune(lam2))) for a, b in zip(dvs, dts)])
    settle(torch, step)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    kept1 = dv.out["kept_count"].cpu().numpy()
    kept2 = dt.out["kept_count"].cpu().numpy()
    nbytes = stage_bytes(vis, kept1)["total"] + stage_bytes(txt, kept2)["total"]
    flops = float(np.sum(2.0 * txt.T.astype(np.float64) * (txt.N + txt.R) * txt.H * txt.d))
    out = {"workload": "%s: B=%d, N in [%d, %d], R=%d; Stage I H=%d d=%d %s; Stage II T in [%d, %d] "
                       "H=%d d=%d" % (name, vis.B, int(vis.N.min()), int(vis.N.max()), vis.R, vis.H,
                                      vis.d, vis.dtype, int(txt.T.min()), int(txt.T.max()), txt.H,
                                      txt.d),
           "ms_per_step": round(ms, 4), "images_s": round(vis.B / (ms * 1e-3), 1),
           "achieved_hbm_gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
           "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
           "text_mfma_frac": round(flops / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
           "kept_stage1_mean": float(np.mean(kept1)), "kept_stage2_mean": float(np.mean(kept2))}

    def text_stage(sb, dss):
        fn = cycler([(lambda d=d: d.prune(lam2)) for d in dss])
        settle(torch, fn)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / steps
        fl = float(np.sum(2.0 * sb.T.astype(np.float64) * (sb.N + sb.R) * sb.H * sb.d))
        tf = fl / (t * 1e-3) / 1e12
        return {"samples": int(sb.B), "ms": round(t, 4), "qk_tflops": round(tf, 1),
                "mfma_frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4),
                "two_pass_mfma_frac": round(2 * tf / MFMA_BF16_PEAK_TFLOPS, 4)}

    out["text_stage"] = text_stage(txt, dts)
    del dv, dt, dvs, dts
    big = [b for b in range(txt.B) if txt.T[b] >= 312]
    if big and len(big) < txt.B:
        sub = synth.make_stage(name, "txt", samples=big)
        dss = [DeviceStage(sub, ragged=sub.ragged) for _ in range(NCOPY)]
        out["text_stage"]["t_ge_312"] = text_stage(sub, dss)
        del dss
    torch.cuda.empty_cache()
    return out


def step_desc(name, vis, txt) -> str:
    """The headline step's workload in words, from the two stage batches (ranges for ragged
    sizes)."""
    def rng(a):
        lo, hi = int(np.min(a)), int(np.max(a))
        return "%d" % lo if lo == hi else "%d-%d" % (lo, hi)
    return ("%s: B=%d, R=%d, N=%s visual tokens; Stage I CLS row H=%d d=%d + %d-wide hidden gather; "
            "Stage II %s text rows H=%d d=%d over all %s tokens + hidden/K/V gather" % (
                name, vis.B, vis.R, rng(vis.N), vis.H, vis.d, vis.payload[0].rows.shape[1],
                rng(txt.T), txt.H, txt.d, rng(txt.N)))


def score_source_sha256() -> str:
    """sha256 of the sources the Stage II scoring kernel is built from."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2605_29657_amd", "csrc")
    h = hashlib.sha256()
    for f in ("anchor_text.hip", "occam_internal.hpp"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def traffic_from_counters(fetch_csv: str, write_csv: str, workload: str) -> dict:
    """profiles/traffic.json from two rocprofv3 --pmc runs of `bench.py --kernel-only`.

    FETCH_SIZE and WRITE_SIZE (KiB per dispatch) of every text_score dispatch are averaged
    and scaled by what the same counter reads for the run's last dispatch, the plain
    1 GiB device copy (__amd_rocclr_copyBuffer) that --kernel-only ends with.
    """
    import csv

    def read(path, kernel="text_score_kernel"):
        rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Dispatch_Id"]))
        score = [float(r["Counter_Value"]) for r in rows if kernel in r["Kernel_Name"]]
        copy = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
        if not score or not copy:
            raise SystemExit("%s: no %s or copy dispatch" % (path, kernel))
        return sum(score) / len(score), copy[-1], len(score)

    gib_kib = float(1 << 20)
    f_kib, f_copy, n_f = read(fetch_csv)
    w_kib, w_copy, n_w = read(write_csv)
    f_scale, w_scale = gib_kib / f_copy, gib_kib / w_copy
    fetch = f_kib * f_scale * 1024.0
    write = w_kib * w_scale * 1024.0
    extra = {}
    for key, kname in (("cls_stream", "cls_stream_kernel"), ("text_stats", "text_stats_kernel")):
        try:
            cf, _, n_c = read(fetch_csv, kname)
            cw, _, _ = read(write_csv, kname)
            extra[key] = {"fetch_bytes": int(round(cf * f_scale * 1024.0)),
                          "write_bytes": int(round(cw * w_scale * 1024.0)),
                          "dispatches": n_c}
        except SystemExit:
            pass
    return {**{"kernel": "text_score", "workload": workload,
            "bytes_per_launch": int(round(fetch + write)),
            "fetch_bytes": int(round(fetch)), "write_bytes": int(round(write)),
            "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
            "dispatches": [n_f, n_w],
            "source_sha256": score_source_sha256(),
            "note": "FETCH_SIZE and WRITE_SIZE (KiB per dispatch) of text_score, scaled by "
                    "what the same counters read for a 1 GiB device copy; the commands are in "
                    "scoring_traffic_llava_next_qwen3vl.md"}, **extra}


def fetch_summary(fetch_csv: str, write_csv: str) -> dict:
    """Mean FETCH_SIZE and WRITE_SIZE per dispatch of every kernel in two rocprofv3 --pmc
    runs of `bench.py --kernel-only`, in bytes, each scaled by what the same counter reads
    for the run's last dispatch, the plain 1 GiB device copy."""
    import csv
    import re

    def per_kernel(path):
        rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Dispatch_Id"]))
        copy = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
        if not copy:
            raise SystemExit("%s: no calibration copy" % path)
        scale = float(1 << 20) / copy[-1]
        acc = {}
        for r in rows:
            name = re.sub(r"\(.*", "", r["Kernel_Name"]).replace("void ", "").replace("occam::", "")
            if name.startswith(("at::", "__amd", "Cijk")):
                continue
            acc.setdefault(name, []).append(float(r["Counter_Value"]) * scale * 1024.0)
        return {k: (sum(v) / len(v), len(v)) for k, v in acc.items()}, scale

    f, fs = per_kernel(fetch_csv)
    w, ws = per_kernel(write_csv)
    return {"fetch_scale": round(fs, 4), "write_scale": round(ws, 4),
            "kernels": {k: {"fetch_bytes": int(round(f[k][0])),
                            "write_bytes": int(round(w.get(k, (0.0, 0))[0])),
                            "dispatches": f[k][1]} for k in sorted(f)}}


# Kernels of one headline step, in launch order: Stage I prune, then Stage II prune (three
# launches each; the threshold and the compaction run in the scoring kernels).
STEP_KERNELS = [
    ("cls_stream_kernel<true, 8, 2>", "cls_stream (Stage I logits + online statistics)"),
    ("cls_scores_kernel<true>", "cls_scores (Stage I scores, threshold, compaction)"),
    ("pack_gather_kernel", "pack_gather (Stage I: 1024-wide hidden rows)"),
    ("text_stats_kernel<8, false, false, 4, 1>", "text_stats (Stage II normalisers)"),
    ("text_score_kernel<8, false, true>", "text_score (Stage II scores, threshold, compaction)"),
    ("pack_gather_kernel", "pack_gather (Stage II: hidden, K and V rows)"),
]


def trace_summary(trace_csv: str, warmup: int = 5, steps: int = 20) -> dict:
    """Per-kernel durations of the headline step from a rocprofv3 --kernel-trace CSV of
    `bench.py --steps N` (N = steps).  The roofline measurement that follows the timed steps
    starts with the first long run of lone scoring launches (its settling calls and timed
    loop, at least `steps` in a row); the timed steps are the last `steps` occurrences of
    the step's kernel sequence before that run (the settling and warm-up steps come earlier;
    the steps on one input copy and the ablation steps, which launch the same sequence,
    later), and the lone scoring figure
    is the last `steps` launches of that run."""
    import csv
    import re
    import statistics as st

    rows = sorted(csv.DictReader(open(trace_csv)), key=lambda r: int(r["Start_Timestamp"]))
    short = [re.sub(r"\(.*", "", r["Kernel_Name"]).replace("void ", "").replace("occam::", "")
             for r in rows]
    dur = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in rows]
    names = [k for k, _ in STEP_KERNELS]
    ours = [i for i, n in enumerate(short) if not n.startswith(("at::", "__amd", "Cijk"))]
    lone = "text_score_kernel<8, false, true>"
    run, j = [], 0
    while j < len(ours):
        k = j
        while k < len(ours) and short[ours[k]] == lone:
            k += 1
        if k - j >= steps:
            run = ours[j:k]
            break
        j = k + 1
    if not run:
        raise SystemExit("%s: no run of %d lone scoring launches" % (trace_csv, steps))
    reps, j = [], 0
    while j + len(names) <= len(ours) and ours[j + len(names) - 1] < run[0]:
        if [short[i] for i in ours[j:j + len(names)]] == names:
            reps.append([dur[i] for i in ours[j:j + len(names)]])
            j += len(names)
        else:
            j += 1
    if len(reps) < warmup + steps:
        raise SystemExit("%s: found %d of %d steps" % (trace_csv, len(reps), warmup + steps))
    timed = reps[-steps:]
    per = [{"kernel": label, "avg_us": round(st.mean(r[k] for r in timed), 1),
            "min_us": round(min(r[k] for r in timed), 1),
            "max_us": round(max(r[k] for r in timed), 1)} for k, (_, label) in enumerate(STEP_KERNELS)]
    alone = [dur[i] for i in run[-steps:]]
    return {"steps": per, "step_sum_us": round(sum(x["avg_us"] for x in per), 1),
            "matched_steps": len(reps),
            "text_score_alone": {"n": len(alone), "avg_us": round(st.mean(alone), 1),
                                 "min_us": round(min(alone), 1), "max_us": round(max(alone), 1)}}


def reference_lse(torch, txt, dt):
    """Per-(row, head) natural log-sum-exp of a uniform text stage, float32 on the device.

    Set-up for timing the scoring kernel alone (occam_score with a caller normaliser);
    not part of any timed region.
    """
    B, S, T = txt.B, txt.R + int(txt.N[0]), int(txt.T[0])
    lse = torch.empty(int(txt.q_off[-1]) * txt.H, dtype=torch.float32, device="cuda")
    grp = txt.H // txt.Hkv
    with torch.no_grad():
        for b in range(B):
            qh = dt.q[b * T:(b + 1) * T].float().permute(1, 0, 2).contiguous()      # [H, T, d]
            kh = dt.k[b * S:(b + 1) * S].float().repeat_interleave(grp, dim=1)
            kh = kh.permute(1, 2, 0).contiguous()                                    # [H, d, S]
            lg = torch.matmul(qh, kh) / float(np.sqrt(np.float32(txt.d)))            # [H, T, S]
            lse.view(-1, txt.H)[b * T:(b + 1) * T] = torch.logsumexp(lg, dim=-1).transpose(0, 1)
    return lse


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llava_next")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-mutual", action="store_true",
                    help="skip the secondary mutual-scoring Stage I measurement")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the LLaVA-1.5, Qwen3-VL and video steps")
    ap.add_argument("--mutual-only", action="store_true",
                    help="run and print only the mutual-scoring Stage I measurement")
    ap.add_argument("--step-only", action="store_true",
                    help="time only the step of --workload and print a short JSON line (for a "
                         "kernel trace whose statistics cover the step's kernels alone)")
    ap.add_argument("--kernel-reps", type=int, default=20,
                    help="timed repetitions of the dominant kernel alone")
    ap.add_argument("--kernel-only", action="store_true",
                    help="run only the dominant kernel (and a plain 1 GiB device copy of known "
                         "size that calibrates byte counters), for counter collection")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write profiles/traffic.json from the counter_collection.csv files "
                         "of two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of --kernel-only")
    ap.add_argument("--fetch-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="per-kernel FETCH_SIZE / WRITE_SIZE bytes (scaled by the calibration "
                         "copy) from two rocprofv3 --pmc runs of --kernel-only")
    ap.add_argument("--trace-summary", metavar="TRACE_CSV",
                    help="per-kernel durations of the step from the kernel_trace.csv of a "
                         "rocprofv3 --kernel-trace run of `bench.py --steps K` (K = --steps)")
    args = ap.parse_args()
    if args.trace_summary:
        print(json.dumps(trace_summary(args.trace_summary, args.warmup, args.steps), indent=1))
        return
    if args.fetch_summary:
        print(json.dumps(fetch_summary(*args.fetch_summary), indent=1))
        return
    if args.traffic_from:
        tj = traffic_from_counters(args.traffic_from[0], args.traffic_from[1], args.workload)
        with open(os.path.join(ROOT, "profiles", "traffic.json"), "w") as f:
            json.dump(tj, f, indent=1)
            f.write("\n")
        print(json.dumps(tj))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: every sample is pruned independently, so a batch "
              "shards across GPUs with no exchange, and the figure per GPU is the one-GPU "
              "figure; run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2605_29657_amd import occam, synth
    from paper_2605_29657_amd.runner import DeviceStage
    from paper_2605_29657_amd.workloads import WORKLOADS

    occam.lib()   # fail loudly if the HIP library is missing
    torch.cuda.set_device(0)
    name = args.workload
    w = WORKLOADS[name]
    with open(os.path.join(ROOT, "tests", "golden", "lambdas.json")) as f:
        lams = json.load(f)[name]
    lam1 = float(np.float32(lams["vis"]["lam"]))
    lam2 = float(np.float32(lams["txt"]["lam"]))

    t0 = time.time()
    if args.mutual_only:
        rec = mutual_stage1(torch, args.steps, args.warmup, not args.no_cpu_baseline)
        print(json.dumps({"mutual_stage1": rec}), flush=True)
        return
    if args.kernel_only:
        txt = synth.make_stage(name, "txt", payload=False)
        dt = DeviceStage(txt, ragged=txt.ragged, payload=False)
        scores_buf = torch.empty_like(dt.out["scores"])
        if not txt.ragged:
            # The scoring kernel alone needs a normaliser; the set-up computes it for a
            # uniform batch only.
            lse = reference_lse(torch, txt, dt)
            for _ in range(args.kernel_reps):
                occam.score(dt.problem, dt.q, dt.k, scores_buf, dt.ws, row_lse=lse)
        for _ in range(args.kernel_reps):
            occam.score(dt.problem, dt.q, dt.k, scores_buf, dt.ws)     # statistics + scoring
        # Stage I scoring (the one-row logits with online statistics, then the scores).
        vis = synth.make_stage(name, "vis", payload=False)
        dv = DeviceStage(vis, ragged=vis.ragged, payload=False)
        vis_scores = torch.empty_like(dv.out["scores"])
        for _ in range(args.kernel_reps):
            occam.score(dv.problem, dv.q, dv.k, vis_scores, dv.ws)
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(1)
        dst.copy_(src)
        torch.cuda.synchronize()
        log("kernel-only: %d launches of text_score alone, %d of text_stats + text_score, "
            "%d of the Stage I scoring, one 1 GiB device copy" % ((args.kernel_reps,) * 3))
        return
    vis = synth.make_stage(name, "vis")
    txt = synth.make_stage(name, "txt")
    log("generated %s in %.1fs" % (name, time.time() - t0))
    # Consecutive steps cycle through NCOPY copies of both stages' inputs (the step of a
    # serving loop sees a new batch of images every time).
    dvs = [DeviceStage(vis, ragged=vis.ragged) for _ in range(NCOPY)]
    dts = [DeviceStage(txt, ragged=txt.ragged) for _ in range(NCOPY)]
    dv, dt = dvs[0], dts[0]
    torch.cuda.synchronize()
    B = vis.B
    step = cycler([(lambda a=a, b=b: (a.prune(lam1), b.prune(lam2))) for a, b in zip(dvs, dts)])

    # Device warm-up before the W warm-up steps: freshly staged buffers are touched for the
    # first time and the clocks leave their idle state; measured from a cold start, the
    # first 20 steps take ~1.8x the steady-state time and the next 20 ~5 % more.  Untimed
    # steps until ~100 ms of GPU work, then the W warm-up steps, then the timed steps.
    settle_steps, g0 = 0, time.perf_counter()
    while settle_steps < 400 and (settle_steps < 40 or time.perf_counter() - g0 < 0.1):
        for _ in range(10):
            step()
        torch.cuda.synchronize()
        settle_steps += 10
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    kept1 = dv.out["kept_count"].cpu().numpy()
    kept2 = dt.out["kept_count"].cpu().numpy()

    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = e0.elapsed_time(e1) / args.steps
    log("timed %d steps: %.3f ms/step (wall %.3f ms/step)" % (args.steps, ms,
                                                              wall * 1e3 / args.steps))
    if args.step_only:
        nbytes = stage_bytes(vis, kept1)["total"] + stage_bytes(txt, kept2)["total"]
        print(json.dumps({"workload": step_desc(name, vis, txt), "steps": args.steps,
                          "settle_steps": settle_steps, "ms_per_step": round(ms, 4),
                          "images_s": round(B / (ms * 1e-3), 1),
                          "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}),
              flush=True)
        return

    b1 = stage_bytes(vis, kept1)
    b2 = stage_bytes(txt, kept2)
    step_bytes = b1["total"] + b2["total"]
    images_s = B / (ms * 1e-3)
    step_gbs = step_bytes / (ms * 1e-3) / 1e9

    # Dominant kernel: the Stage II scoring kernel.  occam_score with a caller-supplied
    # normaliser launches exactly that one kernel, so HIP events around the call on the
    # launch stream time it alone.  The normaliser is the true per-(row, head) log-sum-exp
    # (float32 matmul on the device; setup only).
    # The calls cycle through the input copies; the normaliser (identical for all copies)
    # is one tensor.
    lse = reference_lse(torch, txt, dt)
    score_bufs = [torch.empty_like(d.out["scores"]) for d in dts]
    score_alone = cycler([(lambda d=d, o=o: occam.score(d.problem, d.q, d.k, o, d.ws, row_lse=lse))
                          for d, o in zip(dts, score_bufs)])
    settle(torch, score_alone)
    k0, k1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    k0.record()
    for _ in range(args.kernel_reps):
        score_alone()
    k1.record()
    torch.cuda.synchronize()
    score_ms = k0.elapsed_time(k1) / args.kernel_reps
    # Both Stage II passes (statistics + scoring) for reference.
    both = cycler([(lambda d=d, o=o: occam.score(d.problem, d.q, d.k, o, d.ws))
                   for d, o in zip(dts, score_bufs)])
    settle(torch, both)
    k0.record()
    for _ in range(args.kernel_reps):
        both()
    k1.record()
    torch.cuda.synchronize()
    both_ms = k0.elapsed_time(k1) / args.kernel_reps
    kern_bytes = b2["keys"] + b2["q"] + b2["scores"]
    achieved = kern_bytes / (score_ms * 1e-3) / 1e9
    flops = 2.0 * int(txt.q_off[-1]) * txt.H * (txt.R + int(txt.N[0])) * txt.d
    log("text_score alone %.3f ms (%.0f GB/s, %.0f TFLOP/s); stats+score %.3f ms" % (
        score_ms, achieved, flops / (score_ms * 1e-3) / 1e12, both_ms))

    # The same step when the caller supplies the Stage II row normalisers (the LLM's own
    # attention log-sum-exp, mode row_lse): Stage II is then the scoring pass alone.
    step_lse = cycler([(lambda a=a, b=b: (a.prune(lam1), b.prune(lam2, row_lse=lse)))
                       for a, b in zip(dvs, dts)])
    settle(torch, step_lse)
    k0.record()
    for _ in range(args.steps):
        step_lse()
    k1.record()
    torch.cuda.synchronize()
    ms_lse = k0.elapsed_time(k1) / args.steps
    single_pass = {"ms_per_step": round(ms_lse, 4), "images_s": round(B / (ms_lse * 1e-3), 1),
                   "achieved_hbm_gbs": round(step_bytes / (ms_lse * 1e-3) / 1e9, 1),
                   "hbm_frac": round(step_bytes / (ms_lse * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                   "kept_stage2_mean": float(dt.out["kept_count"].float().mean())}
    log("with a caller normaliser: %.3f ms/step (%.1f%% of HBM peak)" % (
        ms_lse, 100 * single_pass["hbm_frac"]))

    # The dominant kernel inside a step: the caller-normaliser step with its Stage II split
    # into occam_score (exactly text_score here), occam_threshold, occam_select and
    # occam_gather, HIP events on the launch stream around the scoring call of every step,
    # so that Stage I's traffic precedes it as in the step.
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    for i in range(-3, args.steps):
        a, d = dvs[i % NCOPY], dts[i % NCOPY]
        o = d.out
        a.prune(lam1)
        if i >= 0:
            ev[i][0].record()
        occam.score(d.problem, d.q, d.k, o["scores"], d.ws, row_lse=lse)
        if i >= 0:
            ev[i][1].record()
        occam.threshold(d.problem, o["scores"], lam2, occam.REG_MEAN, o["tau"])
        occam.select(d.problem, o["scores"], o["tau"], o["kept_idx"], o["kept_count"],
                     o["kept_offsets"], d.ws)
        occam.gather(d.problem, d.rows, o["kept_idx"], o["kept_offsets"])
    torch.cuda.synchronize()
    in_step_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    log("text_score inside the caller-normaliser step: %.3f ms" % in_step_ms)

    # For reference: the headline steps all on one copy, so that each step's statistics
    # pass can find keys that the previous step left in the memory-side cache.  (After the
    # lone scoring launches: a kernel trace finds the timed steps just before those.)
    def step_one_copy():
        dv.prune(lam1)
        dt.prune(lam2)

    settle(torch, step_one_copy)
    e0.record()
    for _ in range(args.steps):
        step_one_copy()
    e1.record()
    torch.cuda.synchronize()
    ms_one = e0.elapsed_time(e1) / args.steps
    log("the same steps on one input copy: %.3f ms/step" % ms_one)

    traffic = None
    tpath = os.path.join(ROOT, "profiles", "traffic.json")
    if os.path.exists(tpath):
        with open(tpath) as f:
            tj = json.load(f)
        # The counters describe the kernel source they were taken on: report them only
        # while that source is unchanged.
        if (tj.get("kernel") == "text_score" and tj.get("workload") == name and
                tj.get("source_sha256") == score_source_sha256()):
            traffic = tj.get("bytes_per_launch")

    rec = {
        "metric": "images/s for fused prune at 2880 visual tokens; achieved HBM GB/s % of peak",
        "value": round(images_s, 1),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": step_desc(name, vis, txt),
                   "global_batch": B, "lambda1": lam1, "lambda2": lam2,
                   "kept_stage1_mean": float(np.mean(kept1)),
                   "kept_stage2_mean": float(np.mean(kept2))},
        "achieved_hbm_gbs": round(step_gbs, 1),
        "hbm_frac": round(step_gbs / HBM_PEAK_GBS, 4),
        "step_bytes": step_bytes,
        "device_warmup_steps": settle_steps,
        "inputs": "each timed step (and every other timing below, unless stated) cycles through "
                  "%d copies of both stages' inputs, outputs and workspaces" % NCOPY,
        "one_copy_ms_per_step": round(ms_one, 4),
        "roofline": {"kernel": "text_score", "bound": "hbm", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "avg_ms": round(score_ms, 4),
                     "bytes_per_launch": kern_bytes,
                     "mfma_tflops": round(flops / (score_ms * 1e-3) / 1e12, 1),
                     "mfma_frac": round(flops / (score_ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
                     "stats_plus_score_ms": round(both_ms, 4),
                     "in_step": {"avg_ms": round(in_step_ms, 4),
                                 "achieved": round(kern_bytes / (in_step_ms * 1e-3) / 1e9, 1),
                                 "frac": round(kern_bytes / (in_step_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                                 "how": "HIP events around occam_score (text_score alone) inside "
                                        "every step of the caller-normaliser step"}},
    }
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(name, lam1, lam2)
    rec["caller_normaliser"] = single_pass
    rec["llava15_cls_f32_latency"] = cls_f32_latency(torch)
    log("LLaVA-1.5 f32 CLS-row prune (B=1): %.1f us median" % rec["llava15_cls_f32_latency"]["median_us"])
    rec["register_redirect"] = register_redirect_bench(torch)
    log("register redirect: %.1f us" % rec["register_redirect"]["us"])
    rec["budget_matching"] = budget_matching_bench(torch)
    log("budget matching: %.1f us" % rec["budget_matching"]["us"])
    rec["stages"] = stage_breakdown(torch, dvs, dts, txt, lam1, lam2, max(10, args.steps // 2))
    log("stage I alone %.3f ms (%.1f%% of HBM peak; its scoring %.1f%%), stage II alone %.3f ms "
        "(%.1f%%); chained step %.3f ms (%.0f keys)" % (
            rec["stages"]["stage1_ms"], 100 * rec["stages"]["stage1_hbm_frac"],
            100 * rec["stages"]["stage1_score"]["hbm_frac"], rec["stages"]["stage2_ms"],
            100 * rec["stages"]["stage2_hbm_frac"], rec["stages"]["chained"]["step_ms"],
            rec["stages"]["chained"]["stage2_keys_mean"]))
    g = rec["stages"]["gathers"]
    log("gathers alone: Stage I %.1f us (a plain copy of the bytes %.1f us), Stage II %.1f us (%.1f us)" % (
        g["stage1"]["gather_us"], g["stage1"]["copy_us"], g["stage2"]["gather_us"], g["stage2"]["copy_us"]))
    rec["ablation"] = ablation_steps(torch, dvs, dts, float(kept1.mean()), float(kept2.mean()),
                                     max(10, args.steps // 2))
    log("ablation: mean threshold %.3f ms/step, fixed budget %.3f ms/step" % (
        rec["ablation"]["mean_threshold"]["ms_per_step"],
        rec["ablation"]["fixed_budget"]["ms_per_step"]))
    del score_bufs, score_alone, both, step, step_lse, a, d, o
    if not args.no_workloads:
        del dv, dt, dvs, dts
        torch.cuda.empty_cache()
        rec["workloads"] = {}
        for wname in ("llava15", "qwen3vl_ragged", "video"):
            rec["workloads"][wname] = workload_step(torch, wname, 10)
            log("%s: %.3f ms/step, %.0f images/s, %.1f%% of HBM peak" % (
                wname, rec["workloads"][wname]["ms_per_step"], rec["workloads"][wname]["images_s"],
                100 * rec["workloads"][wname]["hbm_frac"]))
    if not args.no_mutual:
        dv = dt = dvs = dts = None
        torch.cuda.empty_cache()
        rec["mutual_stage1"] = mutual_stage1(torch, max(5, args.steps // 5), 2,
                                             not args.no_cpu_baseline)
        log("mutual Stage I: %.3f ms (%.0f TFLOP/s)" % (rec["mutual_stage1"]["ms"],
                                                       rec["mutual_stage1"]["mfma_tflops"]))
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
