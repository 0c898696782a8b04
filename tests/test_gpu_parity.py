"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Every workload shape is checked on seeded synthetic inputs: small batches element by
element, the headline LLaVA-NeXT batch at full size in the launch configuration the
benchmark times (sampled samples), plus edge cases (empty and ragged samples, all or
no survivors, several t-blocks, GQA, d % 16 == 8, other register reductions), the
unfused entry points, determinism, the caller-normaliser mode and index remapping.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2605_29657_amd import occam, synth
from paper_2605_29657_amd.runner import DeviceStage, to_device

from parity import (RTOL, check_bookkeeping, check_rows, check_scores, check_selection, custom_stage, f32_scale,
                    lam_for, oracle_prune)

pytestmark = pytest.mark.gpu


def run_and_check(sb, lam, reduce=oracle.REG_MEAN, ragged=None, rows=True, max_cands=None,
                  row_offsets=None):
    print("case: %s/%s B=%d R=%d H=%d Hkv=%d d=%d T=%s N=%s dtype=%s lam=%.6g ragged=%s" % (
        sb.workload, sb.stage, sb.B, sb.R, sb.H, sb.Hkv, sb.d, sb.T[:4], sb.N[:4], sb.dtype, lam,
        ragged), flush=True)
    ds = DeviceStage(sb, ragged=ragged, max_cands=max_cands, row_offsets=row_offsets)
    ds.prune(lam, reduce=reduce, with_rows=rows)
    g = ds.host(with_rows=rows)
    o = oracle_prune(sb, lam, reduce=reduce)
    rtol = RTOL[sb.dtype]
    err = check_scores(g["scores"], o["scores"], rtol)
    check_scores(g["tau"], o["tau"], rtol, "tau")
    sel = check_selection(g, o, sb, rtol)
    if rows:
        check_rows(g, sb)
    print("  max rel score err %.3g, kept %d, exempt %d" % (err, sel["kept"], sel["exempt"]),
          flush=True)
    return g, o


# ----------------------------------------------------------------------------- workloads
@pytest.mark.parametrize("ragged", [False, True])
def test_llava15_cls_f32(ragged):
    sb = synth.make_stage("llava15_cls_f32", "vis")
    run_and_check(sb, lam_for("llava15_cls_f32", "vis"), ragged=ragged)


@pytest.mark.parametrize("stage", ["vis", "txt"])
def test_llava15(stage):
    sb = synth.make_stage("llava15", stage, B=4)
    run_and_check(sb, lam_for("llava15", stage))


@pytest.mark.parametrize("stage", ["vis", "txt"])
def test_llava_next(stage):
    sb = synth.make_stage("llava_next", stage, B=2)
    run_and_check(sb, lam_for("llava_next", stage))


@pytest.mark.parametrize("stage", ["vis", "txt"])
def test_qwen3vl_ragged(stage):
    sb = synth.make_stage("qwen3vl_ragged", stage, B=5)
    assert sb.ragged
    run_and_check(sb, lam_for("qwen3vl_ragged", stage))


@pytest.mark.parametrize("stage", ["vis", "txt"])
def test_video_full_sample(stage):
    sb = synth.make_stage("video", stage, B=1)
    run_and_check(sb, lam_for("video", stage))


@pytest.mark.parametrize("stage", ["vis", "txt"])
def test_headline_full_batch_sampled(stage):
    # The LLaVA-NeXT batch at full size (B=32), uniform launch as the benchmark runs it;
    # three samples are recomputed by the oracle (a sample's bytes do not depend on B).
    name = "llava_next"
    lam = lam_for(name, stage)
    sb = synth.make_stage(name, stage)
    ds = DeviceStage(sb, ragged=False)
    ds.prune(lam)
    g = ds.host()
    pick = [0, 17, 31]
    sub = synth.make_stage(name, stage, samples=pick)
    o = oracle_prune(sub, lam)
    rtol = RTOL[sb.dtype]
    for j, b in enumerate(pick):
        gs = g["scores"][sb.k_off[b]:sb.k_off[b + 1]]
        check_scores(gs, o["scores"][sub.k_off[j]:sub.k_off[j + 1]], rtol)
        check_scores(g["tau"][b:b + 1], o["tau"][j:j + 1], rtol, "tau")
        gsel = dict(kept_idx=g["kept_idx"][g["kept_offsets"][b]:g["kept_offsets"][b + 1]],
                    kept_count=g["kept_count"][b:b + 1],
                    kept_offsets=np.array([0, g["kept_count"][b]]))
        one = synth.make_stage(name, stage, samples=[b], payload=False)
        oj = dict(scores=o["scores"][sub.k_off[j]:sub.k_off[j + 1]], tau=o["tau"][j:j + 1],
                  kept_idx=o["kept_idx"][o["kept_offsets"][j]:o["kept_offsets"][j + 1]],
                  kept_offsets=np.array([0, o["kept_count"][j]]))
        check_selection(gsel, oj, one, rtol)
    # Whole-batch properties at full size: bookkeeping and byte-exact rows.
    check_bookkeeping(g, sb)
    check_rows(g, sb)


def replicate(one: synth.StageBatch, n: int) -> synth.StageBatch:
    """A batch of n copies of a one-sample batch (same shapes, offsets of a batch of n)."""
    assert one.B == 1
    T, N = np.repeat(one.T, n), np.repeat(one.N, n)
    sb = synth.StageBatch(workload=one.workload, stage=one.stage, dtype=one.dtype, B=n, R=one.R,
                          H=one.H, Hkv=one.Hkv, d=one.d, T=T, N=N,
                          q_off=np.concatenate([[0], np.cumsum(T)]).astype(np.int64),
                          k_off=np.concatenate([[0], np.cumsum(N + one.R)]).astype(np.int64),
                          q=np.concatenate([one.q] * n, axis=0), k=np.concatenate([one.k] * n, axis=0))
    for pl in one.payload:
        rows = sb.k.reshape(sb.k.shape[0], -1) if pl.name == "k_rows" else np.concatenate([pl.rows] * n, 0)
        sb.payload.append(synth.Payload(pl.name, rows, pl.pad_rows, pl.row0))
    return sb


def full_batch_sampled(name, stage, pick, ragged, sb=None, sub=None, oracle_of=None):
    """The whole batch in the benchmark's launch configuration; the picked samples are
    recomputed by the oracle (sample pick[j] against oracle sample oracle_of[j] of `sub`),
    every sample's bookkeeping and rows are checked."""
    lam = lam_for(name, stage)
    sb = synth.make_stage(name, stage) if sb is None else sb
    print("case: full batch %s/%s B=%d ragged=%s oracle samples %s" % (name, stage, sb.B, ragged,
                                                                       pick), flush=True)
    ds = DeviceStage(sb, ragged=ragged)
    ds.prune(lam)
    g = ds.host()
    sub = synth.make_stage(name, stage, samples=pick) if sub is None else sub
    oracle_of = list(range(len(pick))) if oracle_of is None else oracle_of
    o = oracle_prune(sub, lam)
    rtol = RTOL[sb.dtype]
    worst = 0.0
    for b, j in zip(pick, oracle_of):
        gs = g["scores"][sb.k_off[b]:sb.k_off[b + 1]]
        worst = max(worst, check_scores(gs, o["scores"][sub.k_off[j]:sub.k_off[j + 1]], rtol))
        check_scores(g["tau"][b:b + 1], o["tau"][j:j + 1], rtol, "tau")
        gsel = dict(kept_idx=g["kept_idx"][g["kept_offsets"][b]:g["kept_offsets"][b + 1]],
                    kept_count=g["kept_count"][b:b + 1],
                    kept_offsets=np.array([0, g["kept_count"][b]]))
        one = synth.StageBatch(workload=name, stage=stage, dtype=sb.dtype, B=1, R=sb.R, H=sb.H,
                               Hkv=sb.Hkv, d=sb.d, T=sb.T[b:b + 1], N=sb.N[b:b + 1],
                               q_off=np.array([0, sb.T[b]]), k_off=np.array([0, sb.N[b] + sb.R]),
                               q=None, k=None)
        oj = dict(scores=o["scores"][sub.k_off[j]:sub.k_off[j + 1]], tau=o["tau"][j:j + 1],
                  kept_idx=o["kept_idx"][o["kept_offsets"][j]:o["kept_offsets"][j + 1]],
                  kept_offsets=np.array([0, o["kept_count"][j]]))
        check_selection(gsel, oj, one, rtol)
    check_bookkeeping(g, sb)
    check_rows(g, sb)
    print("  max rel score err %.3g over samples %s" % (worst, pick), flush=True)


@pytest.mark.parametrize("stage", ["vis", "txt"])
def test_qwen3vl_full_batch_sampled(stage):
    # B = 64 ragged, as the benchmark launches it; the oracle recomputes the first and last
    # samples and sample 13, which has 512 text rows (four row blocks).
    sb = synth.make_stage("qwen3vl_ragged", stage)
    if stage == "txt":
        assert sb.T[13] == 512
    full_batch_sampled("qwen3vl_ragged", stage, [0, 13, 63], ragged=True, sb=sb)


@pytest.mark.parametrize("stage", ["vis", "txt"])
def test_video_full_batch_sampled(stage):
    # B = 8 uniform at full size (16384 visual tokens and 8 registers per sample; 256 text
    # rows = two row blocks), launched as the benchmark launches it.  Every slot holds the
    # bytes of sample 7 (drawing all eight samples takes minutes on the host), so the
    # oracle's one result must be reproduced by every sample, at every base offset.
    one = synth.make_stage("video", stage, samples=[7])
    full_batch_sampled("video", stage, list(range(8)), ragged=False, sb=replicate(one, 8),
                       sub=one, oracle_of=[0] * 8)


# ----------------------------------------------------------------------------- mutual scoring
# Stage I without a CLS row (Eq. mutual_scoring): every register and visual token is
# an anchor row and each key is scored by the mean attention it receives.
def test_mutual_llava15():
    sb = synth.make_stage("llava15", "mut", B=3)
    run_and_check(sb, lam_for("llava15", "mut"))


def small_qwen_samples(n=3, limit=1500):
    """Sample numbers of the Qwen3-VL-shaped batch whose N stays below ``limit``."""
    out = []
    for b in range(64):
        sb = synth.make_stage("qwen3vl_ragged", "vis", samples=[b], payload=False)
        if int(sb.N[0]) < limit:
            out.append(b)
        if len(out) == n:
            break
    return out


def test_mutual_qwen3vl_ragged_d72():
    sb = synth.make_stage("qwen3vl_ragged", "mut", samples=small_qwen_samples())
    run_and_check(sb, lam_for("qwen3vl_ragged", "mut"))


def test_mutual_ragged_with_an_empty_sample():
    N = np.array([0, 37, 130])
    sb = custom_stage(B=3, R=4, H=4, Hkv=4, d=64, T=N + 4, N=N, stage="mut", seed=11)
    run_and_check(sb, 1.0)


def test_mutual_at_one_row_matches_the_max_form():
    # One anchor row: mean and max over rows are the same number.
    sb = custom_stage(B=2, R=4, H=8, Hkv=8, d=64, T=[1, 1], N=[100, 50], seed=12)
    a = DeviceStage(sb, ragged=True)
    a.prune(1.2)
    sb.stage = "mut"
    m = DeviceStage(sb, ragged=True)
    m.prune(1.2)
    assert torch.equal(a.out["scores"], m.out["scores"])


def test_mutual_headline_shape_sampled():
    # LLaVA-NeXT-shaped encoder without a CLS row at full size: B=32 samples of 2884
    # anchor rows x 2884 keys; two samples recomputed by the oracle.
    name = "llava_next"
    lam = lam_for(name, "mut")
    sb = synth.make_stage(name, "mut")
    ds = DeviceStage(sb, ragged=False)
    ds.prune(lam)
    g = ds.host()
    pick = [3, 30]
    sub = synth.make_stage(name, "mut", samples=pick)
    o = oracle_prune(sub, lam)
    rtol = RTOL[sb.dtype]
    for j, b in enumerate(pick):
        gs = g["scores"][sb.k_off[b]:sb.k_off[b + 1]]
        check_scores(gs, o["scores"][sub.k_off[j]:sub.k_off[j + 1]], rtol)
        check_scores(g["tau"][b:b + 1], o["tau"][j:j + 1], rtol, "tau")
        gsel = dict(kept_idx=g["kept_idx"][g["kept_offsets"][b]:g["kept_offsets"][b + 1]],
                    kept_count=g["kept_count"][b:b + 1],
                    kept_offsets=np.array([0, g["kept_count"][b]]))
        one = synth.make_stage(name, "mut", samples=[b], payload=False)
        oj = dict(scores=o["scores"][sub.k_off[j]:sub.k_off[j + 1]], tau=o["tau"][j:j + 1],
                  kept_idx=o["kept_idx"][o["kept_offsets"][j]:o["kept_offsets"][j + 1]],
                  kept_offsets=np.array([0, o["kept_count"][j]]))
        check_selection(gsel, oj, one, rtol)
    # Every key's mutual score is a mean of probabilities: each sample's scores sum to 1.
    sums = np.add.reduceat(g["scores"].astype(np.float64), sb.k_off[:-1])
    np.testing.assert_allclose(sums, 1.0, rtol=1e-4)
    check_bookkeeping(g, sb)
    check_rows(g, sb)


# ----------------------------------------------------------------------------- edge cases
def test_ragged_with_empty_samples():
    sb = custom_stage(B=5, R=3, H=4, Hkv=4, d=64, T=[1] * 5, N=[0, 37, 0, 300, 1])
    run_and_check(sb, 0.8)


def test_ragged_text_with_empty_and_long_samples():
    sb = custom_stage(B=4, R=4, H=8, Hkv=8, d=128, T=[3, 200, 33, 129], N=[0, 70, 257, 5])
    run_and_check(sb, 1.5)


def test_statistics_row_block_groups():
    # Three and four 128-row blocks at most: the statistics pass takes four row blocks per
    # workgroup, so a group holds row blocks past a sample's rows (idle waves that still copy
    # their share of every key block).  d = 72 gives a key block of five copies for the 16
    # waves of a group (some waves copy nothing).
    for T, d in (([300, 50, 129, 1], 128), ([500, 257, 3], 72)):
        sb = custom_stage(B=len(T), R=4, H=8, Hkv=8, d=d, T=T, N=[400, 90, 0, 33][:len(T)],
                          seed=len(T))
        run_and_check(sb, 1.2)


def test_statistics_key_ranges():
    # Few (sample, head) tasks with many keys: the statistics pass splits each task's keys
    # into ranges (here 5 and 3, one of them with two row blocks per workgroup), and the
    # scoring pass merges the ranges' normalisers.
    for T, N, H in (([128, 70], [3000, 1500], 8), ([200, 129], [1900, 2100], 16)):
        sb = custom_stage(B=2, R=4, H=H, Hkv=H, d=128, T=T, N=N, seed=H)
        run_and_check(sb, 1.3)


def test_cls_row_odd_head_chunks():
    # One anchor row, 16 heads of 5, 6, 7 or 9 sixteen-byte chunks (d = 40, 48, 56, 72):
    # the key rows stream as contiguous runs of four rows; ragged, with an empty sample and
    # a chunk that ends after one key.
    for d in (40, 48, 56, 72):
        sb = custom_stage(B=4, R=4, H=16, Hkv=16, d=d, T=[1] * 4, N=[300, 0, 1021, 125], seed=d)
        run_and_check(sb, 0.9)


def test_lambda_zero_keeps_everything_and_huge_keeps_nothing():
    sb = custom_stage(B=3, R=2, H=4, Hkv=2, d=64, T=[40] * 3, N=[100] * 3)
    g, _ = run_and_check(sb, 0.0)
    assert np.array_equal(g["kept_count"], sb.N)
    g, _ = run_and_check(sb, 1e30)
    assert np.all(g["kept_count"] == 0) and np.all(g["kept_offsets"] == 0)


def test_uniform_rows_with_ragged_keys():
    # Ragged key counts, every sample 128 or 256 text rows, passed without row offsets:
    # the scoring pass's full-row-block form meets the ragged task mapping (and, at 256
    # rows, the combine over two row blocks).
    for T in (128, 256):
        sb = custom_stage(B=4, R=4, H=8, Hkv=8, d=128, T=[T] * 4, N=[700, 30, 0, 260], seed=T)
        run_and_check(sb, 1.0, ragged=True, row_offsets=False)


def test_ragged_text_with_many_samples():
    # 130 ragged samples: each lane of the task-decoding wave counts three samples, some
    # samples have no candidates, some rows span two 128-row blocks.
    rng = np.random.default_rng(11)
    B = 130
    T = rng.integers(1, 200, size=B)
    N = rng.integers(0, 300, size=B)
    N[::17] = 0
    sb = custom_stage(B=B, R=4, H=4, Hkv=4, d=64, T=list(T), N=list(N), seed=5)
    run_and_check(sb, 1.0)


def test_late_keys_far_above_the_early_ones():
    # Sinks scaled x25 and x60 put some (row, head) logits 2^64 .. 2^128 and more than
    # 2^128 (in base-2 units) above the largest logit among the sample's first 32 keys:
    # sums against an early reference would overflow float32, so the statistics pass
    # must re-reference those rows.
    for scale, seed in ((25.0, 3), (60.0, 4)):
        sb = custom_stage(B=2, R=4, H=8, Hkv=8, d=128, T=[128, 60], N=[700, 300], sinks=6,
                          sink_scale=scale, seed=seed)
        q, k = synth.bf16_bits_to_f32(sb.q), synth.bf16_bits_to_f32(sb.k)
        gaps = []
        for b in range(sb.B):
            qb = q[sb.q_off[b]:sb.q_off[b + 1]].astype(np.float64)
            kb = k[sb.k_off[b]:sb.k_off[b + 1]].astype(np.float64)
            x = np.einsum("thd,shd->hts", qb, kb) / np.sqrt(sb.d) * np.log2(np.e)
            gaps.append((x.max(axis=2) - x[:, :, :32].max(axis=2)).ravel())
        gaps = np.concatenate(gaps)
        assert np.any((gaps > 64) & (gaps < 128)) and np.any(gaps > 128), (scale, gaps.max())
        run_and_check(sb, 1.0)


@pytest.mark.parametrize("reduce", [oracle.REG_MAX, oracle.REG_SUM])
def test_other_register_reductions(reduce):
    sb = custom_stage(B=2, R=8, H=8, Hkv=8, d=64, T=[1, 1], N=[500, 333])
    run_and_check(sb, 0.9, reduce=reduce)


def test_gqa_and_d72_text_rows():
    sb = custom_stage(B=2, R=4, H=8, Hkv=2, d=72, T=[64, 17], N=[250, 90])
    run_and_check(sb, 1.2)


def test_f32_cls_d72_and_d256():
    run_and_check(custom_stage(B=2, R=1, H=16, Hkv=16, d=72, T=[1, 1], N=[200, 31], dtype="f32"),
                  1.0)
    run_and_check(custom_stage(B=1, R=2, H=4, Hkv=1, d=256, T=[1], N=[100], dtype="f32"), 1.0)


def test_text_path_at_one_row_matches_the_cls_path():
    # A ragged problem whose rows are all 1 but whose row bound is 2 runs the MFMA path;
    # the same problem with row bound 1 runs the VALU path.  Two independent codes, one
    # answer.
    sb = custom_stage(B=3, R=4, H=16, Hkv=16, d=64, T=[1, 1, 1], N=[576, 100, 31])
    a = DeviceStage(sb, ragged=True)
    a.prune(1.0)
    ga = a.host()
    b = DeviceStage(sb, ragged=True)
    b.problem = occam.Problem(sb.B, sb.H, sb.Hkv, sb.d, sb.R, q_offsets=b.q_off,
                              key_offsets=b.k_off, max_rows=2, max_cands=int(sb.N.max()),
                              dtype=sb.dtype)
    b.ws = occam.workspace(b.problem)
    b.prune(1.0)
    gb = b.host()
    check_scores(gb["scores"], ga["scores"].astype(np.float64), 1e-4, "mfma vs valu")


# ----------------------------------------------------------------------------- API variants
def test_unfused_calls_equal_the_fused_call():
    sb = synth.make_stage("llava15", "txt", B=3)
    lam = lam_for("llava15", "txt")
    ds = DeviceStage(sb)
    ds.prune(lam)
    fused = ds.host()
    p, dev = ds.problem, "cuda"
    scores = torch.empty(ds.total_keys, dtype=torch.float32, device=dev)
    tau = torch.empty(sb.B, dtype=torch.float32, device=dev)
    kept = torch.empty(ds.total_cands, dtype=torch.int32, device=dev)
    cnt = torch.empty(sb.B, dtype=torch.int32, device=dev)
    offs = torch.empty(sb.B + 1, dtype=torch.int32, device=dev)
    occam.score(p, ds.q, ds.k, scores, ds.ws)
    occam.threshold(p, scores, lam, occam.REG_MEAN, tau)
    occam.select(p, scores, tau, kept, cnt, offs, ds.ws)
    dsts = [torch.zeros_like(d) for d in ds.row_dst]
    rows = [occam.Rows(s, d_, src_pad_rows=pl.pad_rows, src_row0=pl.row0)
            for s, d_, pl in zip(ds.row_src, dsts, sb.payload)]
    occam.gather(p, rows, kept, offs)
    torch.cuda.synchronize()
    total = int(offs[-1])
    assert np.array_equal(scores.cpu().numpy(), fused["scores"])
    assert np.array_equal(tau.cpu().numpy(), fused["tau"])
    assert np.array_equal(kept[:total].cpu().numpy(), fused["kept_idx"])
    assert np.array_equal(offs.cpu().numpy(), fused["kept_offsets"])
    for d_, want in zip(dsts, fused["rows"]):
        got = d_[:total].cpu()
        got = got.view(torch.int16).numpy().view(np.uint16) if got.dtype == torch.bfloat16 else got.numpy()
        assert np.array_equal(got.view(np.uint8), want.view(np.uint8))


@pytest.mark.parametrize("name,stage", [("llava_next", "vis"), ("llava_next", "txt"),
                                        ("qwen3vl_ragged", "txt")])
def test_run_to_run_bitwise_determinism(name, stage):
    sb = synth.make_stage(name, stage, B=4)
    lam = lam_for(name, stage)
    ds = DeviceStage(sb)
    ds.prune(lam)
    a = ds.host()
    for v in ds.out.values():
        v.fill_(-7)
    ds.prune(lam)
    b = ds.host()
    for key in ("scores", "tau", "kept_idx", "kept_count", "kept_offsets"):
        assert np.array_equal(a[key].view(np.uint8), b[key].view(np.uint8)), key


def test_caller_normaliser_over_a_larger_key_set():
    # row_lse from the caller (here: the log-sum-exp over the keys plus 24 extra keys that
    # are not scored, computed on the host in float64) replaces the per-row softmax sum.
    sb = custom_stage(B=2, R=4, H=8, Hkv=8, d=64, T=[20, 20], N=[150, 150], dtype="bf16")
    rng = np.random.default_rng(5)
    qf = synth.bf16_bits_to_f32(sb.q).reshape(-1, sb.H, sb.d).astype(np.float64)
    kf = synth.bf16_bits_to_f32(sb.k).reshape(-1, sb.Hkv, sb.d).astype(np.float64)
    scale = f32_scale(sb.d)
    lse = np.empty((int(sb.q_off[-1]), sb.H))
    for b in range(sb.B):
        extra = rng.standard_normal((24, sb.Hkv, sb.d))
        keys = np.concatenate([kf[sb.k_off[b]:sb.k_off[b + 1]], extra])
        for t in range(sb.q_off[b], sb.q_off[b + 1]):
            for h in range(sb.H):
                lg = keys[:, h] @ qf[t, h] * scale
                m = lg.max()
                lse[t, h] = m + np.log(np.exp(lg - m).sum())
    lse32 = lse.astype(np.float32)
    ds = DeviceStage(sb)
    ds.prune(0.7, row_lse=torch.from_numpy(lse32.reshape(-1)).cuda())
    g = ds.host()
    o = oracle_prune(sb, 0.7, row_lse=lse32.reshape(-1).astype(np.float64))
    check_scores(g["scores"], o["scores"], RTOL["bf16"])
    check_selection(g, o, sb, RTOL["bf16"])
    check_rows(g, sb)


def test_index_map_remaps_the_list_but_not_the_gather():
    sb = custom_stage(B=3, R=2, H=4, Hkv=4, d=64, T=[9, 9, 9], N=[60, 0, 45])
    rng = np.random.default_rng(8)
    imap = rng.permutation(100000)[:int(sb.N.sum())].astype(np.int32)
    ds = DeviceStage(sb, ragged=True)
    ds.prune(1.1, index_map=torch.from_numpy(imap).cuda())
    g = ds.host()
    o = oracle_prune(sb, 1.1, index_map=imap)
    check_scores(g["scores"], o["scores"], RTOL["bf16"])
    check_selection(g, o, sb, RTOL["bf16"], index_map=imap)
    # Rows are gathered at the local indices: recover them through the inverse map.
    co = np.concatenate([[0], np.cumsum(sb.N)])
    local = np.empty_like(g["kept_idx"])
    for b in range(sb.B):
        inv = {int(imap[co[b] + v]): v for v in range(sb.N[b])}
        s, e = g["kept_offsets"][b], g["kept_offsets"][b + 1]
        local[s:e] = [inv[int(x)] for x in g["kept_idx"][s:e]]
    check_rows(dict(g, kept_idx=local), sb)
