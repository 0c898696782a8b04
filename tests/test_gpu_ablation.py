"""GPU parity of the component ablation's threshold variants (Appendix, Table
tab:qwen_compact_component_ablation): the mean-based threshold (occam_threshold,
occam_prune and occam_match_lambda with OCCAM_REF_CAND_MEAN) and the fixed budget
(occam_select_topk), against the oracle.

occam_select_topk is compared bit for bit on score vectors both sides read as the same
float32 values (ties included); on scores computed by the GPU, the kept sets may differ
only at tokens whose oracle score lies within the score tolerance of the K-th score."""
import numpy as np
import pytest
import torch

import oracle
from paper_2605_29657_amd import occam, synth
from paper_2605_29657_amd.runner import DeviceStage

from parity import RTOL, check_bookkeeping, check_rows, check_scores, check_selection, \
    custom_stage, oracle_prune

pytestmark = pytest.mark.gpu


def problem_for(N, R, ragged=True):
    N = np.asarray(N, dtype=np.int64)
    k_off = np.concatenate([[0], np.cumsum(N + R)]).astype(np.int64)
    if ragged:
        p = occam.Problem(len(N), 16, 16, 64, R, key_offsets=torch.tensor(
            k_off.astype(np.int32), device="cuda"), max_cands=max(1, int(N.max())))
    else:
        p = occam.Problem(len(N), 16, 16, 64, R, cands=int(N[0]))
    return p, k_off


def gpu_topk(p, sc, B, K, index_map=None):
    ncand = max(1, sc.numel())
    kept = torch.full((ncand,), -1, dtype=torch.int32, device="cuda")
    cnt = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    offs = torch.full((B + 1,), -1, dtype=torch.int32, device="cuda")
    occam.select_topk(p, sc, K, kept, cnt, offs, occam.workspace(p), index_map=index_map)
    torch.cuda.synchronize()
    offs_h = offs.cpu().numpy()
    return kept[:int(offs_h[-1])].cpu().numpy(), cnt.cpu().numpy(), offs_h


def run_topk(N, R, K, seed, quant=0, zeros=0, ragged=True, with_map=False):
    print("case: topk B=%d N=%s R=%d K=%d seed=%d quant=%d zeros=%d ragged=%s map=%s" % (
        len(N), list(N)[:6], R, K, seed, quant, zeros, ragged, with_map), flush=True)
    rng = np.random.default_rng(seed)
    p, k_off = problem_for(N, R, ragged)
    sc = rng.random(int(k_off[-1])).astype(np.float32) * 0.01
    if quant:
        sc = (np.round(sc * quant) / quant).astype(np.float32)
    if zeros:
        sc[rng.integers(0, sc.size, zeros)] = 0.0
    im = None
    if with_map:
        im = rng.permutation(int(np.sum(N)) * 3)[:int(np.sum(N))].astype(np.int32)
    got = gpu_topk(p, torch.from_numpy(sc).cuda(), len(N), K,
                   None if im is None else torch.from_numpy(im).cuda())
    want = oracle.select_topk(sc.astype(np.float64), k_off, R, K, index_map=im)
    for g, w, what in zip(got, want, ("kept_idx", "kept_count", "kept_offsets")):
        assert np.array_equal(g, w), what


def test_topk_ragged_with_empty_samples_and_ties():
    run_topk([300, 0, 577, 1, 64, 2], R=4, K=50, seed=1, quant=64, zeros=30)


@pytest.mark.parametrize("K", [0, 1, 63, 64, 255, 256, 10000])
def test_topk_budgets(K):
    run_topk([256, 1000, 17], R=2, K=K, seed=2, quant=1000)


def test_topk_all_equal_scores_keep_the_first_indices():
    run_topk([500, 500], R=1, K=123, seed=3, quant=1)        # scores in {0, 0.01}: mostly 0


def test_topk_index_map_uniform():
    run_topk([2880] * 4, R=4, K=576, seed=4, ragged=False, with_map=True)


def test_topk_full_size_batch():
    run_topk([2880] * 32, R=4, K=192, seed=5, ragged=False)


def test_topk_video_sample():
    run_topk([16384], R=1, K=4096, seed=6, quant=100000)


def test_topk_on_gpu_scores_then_gather():
    # The ablation's pipeline: occam_score, occam_select_topk, occam_gather.
    sb = synth.make_stage("llava_next", "txt", B=2)
    ds = DeviceStage(sb)
    ds.prune(1.0)                                     # scores (and an unrelated selection)
    g = ds.host(with_rows=False)
    K = 288
    o_sc = oracle_prune(sb, 1.0)["scores"]
    kept, cnt, offs = gpu_topk(ds.problem, ds.out["scores"][:ds.total_keys], sb.B, K)
    okept, ocnt, ooffs = oracle.select_topk(o_sc, sb.k_off, sb.R, K)
    assert np.array_equal(cnt, ocnt) and np.array_equal(offs, ooffs)
    rtol = RTOL[sb.dtype]
    for b in range(sb.B):
        sv = o_sc[sb.k_off[b] + sb.R:sb.k_off[b + 1]]
        kth = np.sort(sv)[::-1][K - 1]
        diff = set(kept[offs[b]:offs[b + 1]].tolist()) ^ set(okept[ooffs[b]:ooffs[b + 1]].tolist())
        for v in diff:
            assert abs(sv[v] - kth) <= rtol * kth, (b, v, sv[v], kth)
    # Gather of the top-K survivors: byte copies of their rows.
    res = dict(kept_idx=kept, kept_offsets=offs, kept_count=cnt)
    check_bookkeeping(res, sb)
    dsts = [torch.zeros_like(d) for d in ds.row_dst]
    rows = [occam.Rows(s, d_, src_pad_rows=pl.pad_rows, src_row0=pl.row0)
            for s, d_, pl in zip(ds.row_src, dsts, sb.payload)]
    occam.gather(ds.problem, rows, torch.from_numpy(kept).cuda(), torch.from_numpy(offs).cuda())
    torch.cuda.synchronize()
    total = int(offs[-1])
    out = []
    for d_ in dsts:
        a = d_[:total].cpu()
        out.append(a.view(torch.int16).numpy().view(np.uint16) if a.dtype == torch.bfloat16
                   else a.numpy())
    res["rows"] = out
    check_rows(res, sb)


# ----------------------------------------------------------------------------- mean threshold
def sum_rtol(N, threads=256):
    """Relative error bound of the GPU's float32 candidate mean of non-negative scores:
    a strided per-thread sum, a 64-lane tree, the waves in order and one division."""
    depth = -(-int(N) // threads) + 6 + threads // 64 + 1
    return depth * 2.0 ** -24 * 1.01


def test_mean_threshold_values():
    rng = np.random.default_rng(7)
    N = [300, 0, 2880, 1, 16384]
    R = 2
    p, k_off = problem_for(N, R)
    sc = (rng.random(int(k_off[-1])) ** 4).astype(np.float32)
    tau = torch.empty(len(N), dtype=torch.float32, device="cuda")
    occam.threshold(p, torch.from_numpy(sc).cuda(), 1.7, occam.REF_CAND_MEAN, tau)
    torch.cuda.synchronize()
    got = tau.cpu().numpy().astype(np.float64)
    want = oracle.threshold(sc.astype(np.float64), k_off, R, np.float32(1.7), oracle.CAND_MEAN)
    for b in range(len(N)):
        assert abs(got[b] - want[b]) <= (sum_rtol(N[b]) + 2 ** -24) * want[b] + 0.0, b
    assert got[1] == 0.0


@pytest.mark.parametrize("name,stage", [("llava_next", "vis"), ("llava_next", "txt"),
                                        ("qwen3vl_ragged", "txt")])
def test_mean_threshold_prune(name, stage):
    sb = synth.make_stage(name, stage, B=2)
    for lam in (1.0, 3.0):
        print("case: %s/%s mean threshold lam=%g" % (name, stage, lam), flush=True)
        ds = DeviceStage(sb)
        ds.prune(lam, reduce=occam.REF_CAND_MEAN)
        g = ds.host()
        o = oracle_prune(sb, lam, reduce=oracle.CAND_MEAN)
        rtol = RTOL[sb.dtype]
        check_scores(g["scores"], o["scores"], rtol)
        check_scores(g["tau"], o["tau"], rtol, "tau")
        check_selection(g, o, sb, rtol)
        check_rows(g, sb)
        # The unfused threshold gives the same bits as the one fused into the selection.
        tau = torch.empty(sb.B, dtype=torch.float32, device="cuda")
        occam.threshold(ds.problem, ds.out["scores"], lam, occam.REF_CAND_MEAN, tau)
        torch.cuda.synchronize()
        assert np.array_equal(tau.cpu().numpy(), g["tau"])


def test_mean_threshold_ragged_with_an_empty_sample():
    sb = custom_stage(B=3, R=2, H=4, Hkv=2, d=64, T=[5, 1, 9], N=[200, 0, 333], seed=8)
    ds = DeviceStage(sb)
    ds.prune(1.2, reduce=occam.REF_CAND_MEAN)
    g = ds.host()
    o = oracle_prune(sb, 1.2, reduce=oracle.CAND_MEAN)
    check_scores(g["tau"], o["tau"], RTOL[sb.dtype], "tau")
    check_selection(g, o, sb, RTOL[sb.dtype])
    assert g["tau"][1] == 0.0 and g["kept_count"][1] == 0


def test_budget_matching_with_the_mean_reference():
    # Dyadic visual scores and a power-of-two N: the candidate mean is exact in float32
    # whatever the order, so the ratios are the same float32 values on both sides.
    rng = np.random.default_rng(9)
    N, R, B = 512, 2, 6
    p, k_off = problem_for([N] * B, R, ragged=False)
    sc = (rng.integers(0, 4096, int(k_off[-1])) / 4096.0).astype(np.float32)
    ws = occam.workspace(p)
    out = torch.empty(2, dtype=torch.float32, device="cuda")
    occam.match_lambda(p, torch.from_numpy(sc).cuda(), 100.0, out[0:1], ws, mean_kept=out[1:2],
                       reduce=occam.REF_CAND_MEAN)
    torch.cuda.synchronize()
    lam, mk = out.cpu().numpy()
    ref = oracle.threshold(sc.astype(np.float64), k_off, R, 1.0, oracle.CAND_MEAN)
    assert np.array_equal(ref, ref.astype(np.float32))
    rat = [(sc[k_off[b] + R:k_off[b + 1]] / np.float32(ref[b])).astype(np.float64)
           for b in range(B)]
    want = np.float32(oracle.match_lambda(rat, 100.0))
    assert lam.view(np.uint32) == want.view(np.uint32), (lam, want)
    kept = sum(int(np.count_nonzero(r >= np.float64(lam))) for r in rat)
    assert mk == np.float32(kept / B)
