"""GPU parity of budget matching (Appendix Eq. lambda2_budget_matching_appendix):
occam_match_lambda against the oracle's match_lambda on the same score vectors.

The count decision is taken in float32 on both sides: the expected ratios are the
float32 quotients s(v) / s(r) (register scores are chosen dyadic, so s(r) is exact in
float32 whatever the summation order), and the oracle picks the level from them.  The
returned lambda and the mean kept count must then agree bit for bit."""
import numpy as np
import pytest
import torch

import oracle
from paper_2605_29657_amd import occam

pytestmark = pytest.mark.gpu


def make_scores(N, R, seed, ties=0, zeros=0):
    rng = np.random.default_rng(seed)
    N = np.asarray(N, dtype=np.int64)
    k_off = np.concatenate([[0], np.cumsum(N + R)]).astype(np.int64)
    sc = np.empty(int(k_off[-1]), dtype=np.float32)
    for b in range(len(N)):
        kb = int(k_off[b])
        sc[kb:kb + R] = rng.integers(16, 257, R) / 256.0            # dyadic register scores
        v = np.exp(rng.standard_normal(int(N[b])) * 1.5) * 0.02
        if ties and N[b]:
            v = np.round(v * ties) / ties                            # many equal ratios
        if zeros and N[b]:
            v[rng.integers(0, N[b], zeros)] = 0.0
        sc[kb + R:kb + R + N[b]] = v.astype(np.float32)
    return sc, k_off


def expected(sc, k_off, R, reduce, k_target):
    sr = oracle.register_reference(sc.astype(np.float64), k_off, R, reduce)
    assert np.array_equal(sr, sr.astype(np.float32))                 # exact in float32
    rat = [(sc[k_off[b] + R:k_off[b + 1]] / np.float32(sr[b])).astype(np.float64)
           for b in range(len(k_off) - 1)]
    lam = oracle.match_lambda(rat, np.float64(np.float32(k_target)))
    kept = sum(int(np.count_nonzero(r >= lam)) for r in rat)
    return np.float32(lam), np.float32(kept / (len(k_off) - 1)), rat


def run_case(N, R, k_target, reduce=oracle.REG_MEAN, seed=0, ties=0, zeros=0, ragged=True,
             ws=None):
    print("case: B=%d N=%s R=%d k=%s reduce=%d seed=%d ties=%d zeros=%d" % (
        len(N), list(N)[:6], R, k_target, reduce, seed, ties, zeros), flush=True)
    sc, k_off = make_scores(N, R, seed, ties, zeros)
    B = len(N)
    if ragged:
        p = occam.Problem(B, 16, 16, 64, R, key_offsets=torch.tensor(k_off.astype(np.int32),
                                                                      device="cuda"),
                          max_cands=max(1, int(max(N))))
    else:
        p = occam.Problem(B, 16, 16, 64, R, cands=int(N[0]))
    d_sc = torch.from_numpy(sc).cuda()
    if ws is None:
        ws = occam.workspace(p)
    assert ws.numel() >= occam.workspace_size(p)
    out = torch.full((2,), -7.0, dtype=torch.float32, device="cuda")
    occam.match_lambda(p, d_sc, k_target, out[0:1], ws, mean_kept=out[1:2], reduce=reduce)
    torch.cuda.synchronize()
    got_lam, got_mk = out.cpu().numpy()
    want_lam, want_mk, rat = expected(sc, k_off, R, reduce, k_target)
    assert got_lam.view(np.uint32) == want_lam.view(np.uint32), (got_lam, want_lam)
    assert got_mk == want_mk, (got_mk, want_mk)
    # The float32 lambda keeps exactly the matched count.
    kept = sum(int(np.count_nonzero(r >= np.float64(got_lam))) for r in rat)
    assert np.float32(kept / B) == want_mk
    return got_lam, got_mk


def test_ragged_with_an_empty_sample():
    run_case([300, 0, 577, 1, 64], R=4, k_target=50.0, seed=1)


@pytest.mark.parametrize("k_target", [0.0, 0.4, 1.0, 17.25, 99.5, 250.0, 1e6])
def test_targets_from_none_to_all(k_target):
    run_case([200, 131, 256], R=2, k_target=k_target, seed=2)


@pytest.mark.parametrize("reduce", [oracle.REG_MEAN, oracle.REG_MAX, oracle.REG_SUM])
def test_register_reductions(reduce):
    run_case([576] * 6, R=8 if reduce == oracle.REG_MEAN else 3, k_target=64.0, reduce=reduce,
             seed=3, ragged=False)


def test_many_equal_ratios_and_zeros():
    # Few distinct levels: the matched count is a level, not the target itself.
    lam, mk = run_case([1000, 999, 17], R=1, k_target=333.3, seed=4, ties=64, zeros=40)
    assert lam > 0


def test_half_way_target_takes_the_smaller_count():
    # Two samples, distinct ratios: 2 * 4.25 = 8.5 kept over the batch lies half way
    # between the levels of 8 and 9, and the tie goes to 8 (the larger lambda).
    run_case([40, 40], R=1, k_target=4.25, seed=5)


def test_all_ratios_zero_or_equal():
    run_case([50, 50], R=1, k_target=10.0, seed=6, ties=1)   # ratios in {0, 1/256 multiples}


def test_no_candidates_gives_one():
    lam, mk = run_case([0, 0, 0], R=2, k_target=5.0, seed=7)
    assert lam == 1.0 and mk == 0.0


def test_full_size_batch():
    # 64 samples of 2880 candidates: about 184k ratios through all four radix passes.
    run_case([2880] * 64, R=4, k_target=576.0, seed=8, ragged=False)


def test_many_small_samples():
    # 1000 samples of 0..50 candidates: one chunk each, many workgroups per pass.
    N = np.random.default_rng(9).integers(0, 51, 1000)
    run_case(list(N), R=2, k_target=12.5, seed=9)


def test_repeated_calls_reuse_the_workspace():
    # The selection state lives in the workspace and is cleared by every call.
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    for seed, k, N in ((10, 3.0, [700, 300, 1500]), (11, 40.0, [1500, 2]), (12, 0.0, [5])):
        run_case(N, R=4, k_target=k, seed=seed, ws=ws)
