"""Pins of the fp64 oracle against things other than itself.

Each test ties one part of the oracle to a closed form, a library routine, an
invariant the paper's definitions imply, or a brute-force / high-precision
recomputation, so that a plausible slip in the oracle (a dropped 1/H, a max
where a mean belongs, a wrong key-head mapping, a strict comparison, an offset
error) fails at least one of them.  CPU only.
"""
import json
import os

import mpmath
import numpy as np
import pytest
import scipy.special as sps
import torch

import oracle
from paper_2605_29657_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------- helpers
def f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def one_sample(q, k, R, H, Hkv, d, dtype="f32", **kw):
    """Oracle scores of a single sample; q [T,H,d], k [S,Hkv,d] float32."""
    T, S = q.shape[0], k.shape[0]
    return oracle.scores(f32(q), f32(k), [0, T], [0, S], H, Hkv, d, R, dtype=dtype, **kw)


def softmax_row(qv, kmat, scale):
    """Textbook softmax (scipy) of scale * k @ q over all keys."""
    return sps.softmax(scale * (kmat.astype(np.float64) @ qv.astype(np.float64)))


# ----------------------------------------------------------------------------- decoding
def test_bf16_decode_matches_torch():
    rng = np.random.default_rng(1)
    bits = rng.integers(0, 1 << 16, size=4000, dtype=np.uint32).astype(np.uint16)
    exp_field = (bits.astype(np.uint32) >> 7) & 0xFF
    bits = bits[exp_field != 0xFF]                                 # no inf / NaN
    bits = np.concatenate([bits, np.array([0x0000, 0x8000, 0x0001, 0x3F80, 0xBF80, 0x7F7F],
                                          dtype=np.uint16)])
    want = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).double().numpy()
    got = np.array([oracle.bf16_to_double(int(b)) for b in bits])
    assert np.array_equal(got, want)


def test_generator_bf16_rounding_matches_torch():
    rng = np.random.default_rng(2)
    x = (rng.standard_normal(20000) * 10.0 ** rng.integers(-20, 20, 20000)).astype(np.float32)
    mine = synth.to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(mine, ref)


# ----------------------------------------------------------------------------- steps 1-2
@pytest.mark.parametrize("d", [4, 64, 72])
def test_single_head_single_row_is_scipy_softmax(d):
    rng = np.random.default_rng(d)
    S, R = 37, 3
    q = rng.standard_normal((1, 1, d)).astype(np.float32)
    k = rng.standard_normal((S, 1, d)).astype(np.float32)
    got = one_sample(q, k, R, 1, 1, d)
    want = softmax_row(q[0, 0], k[:, 0], 1.0 / np.sqrt(d))
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=0)


def test_scale_parameter_is_the_temperature():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((1, 1, 8)).astype(np.float32)
    k = rng.standard_normal((20, 1, 8)).astype(np.float32)
    got = one_sample(q, k, 2, 1, 1, 8, scale=0.37)
    np.testing.assert_allclose(got, softmax_row(q[0, 0], k[:, 0], 0.37), rtol=1e-13)


def test_head_mean_with_a_uniform_head():
    # Head 1 has q = 0, so its softmax is uniform 1/S; the score is the mean of the two heads.
    rng = np.random.default_rng(4)
    S, d = 25, 16
    q = np.zeros((1, 2, d), np.float32)
    q[0, 0] = rng.standard_normal(d)
    k = rng.standard_normal((S, 2, d)).astype(np.float32)
    got = one_sample(q, k, 2, 2, 2, d)
    want = 0.5 * (softmax_row(q[0, 0], k[:, 0], 1 / np.sqrt(d)) + 1.0 / S)
    np.testing.assert_allclose(got, want, rtol=1e-13)


def test_grouped_query_heads_read_their_key_head():
    # H=4, Hkv=2: heads 0,1 -> key head 0, heads 2,3 -> key head 1 (h // (H/Hkv)).
    rng = np.random.default_rng(5)
    S, d = 30, 8
    q = np.zeros((1, 4, d), np.float32)
    qs = rng.standard_normal(d).astype(np.float32)
    q[0, 2] = qs
    q[0, 3] = qs
    k = rng.standard_normal((S, 2, d)).astype(np.float32)
    got = one_sample(q, k, 1, 4, 2, d)
    p = softmax_row(qs, k[:, 1], 1 / np.sqrt(d))
    want = (2.0 / S + 2.0 * p) / 4.0
    np.testing.assert_allclose(got, want, rtol=1e-13)


def test_visual_max_and_register_mean_over_rows():
    # Row 0 has q = 0 (uniform); row 1 is a real query.  Visual: max; register: mean.
    rng = np.random.default_rng(6)
    S, d, R = 40, 8, 3
    q = np.zeros((2, 1, d), np.float32)
    q[1, 0] = 3.0 * rng.standard_normal(d)
    k = rng.standard_normal((S, 1, d)).astype(np.float32)
    got = one_sample(q, k, R, 1, 1, d)
    p = softmax_row(q[1, 0], k[:, 0], 1 / np.sqrt(d))
    want = np.maximum(p, 1.0 / S)
    want[:R] = 0.5 * (p[:R] + 1.0 / S)
    np.testing.assert_allclose(got, want, rtol=1e-13)


def test_head_mean_is_taken_before_the_row_max():
    # head 0: row 0 = q*, row 1 = 0; head 1: row 0 = 0, row 1 = q*.
    # max_t mean_h = (p + 1/S)/2, whereas mean_h max_t would give p for the peaked keys.
    rng = np.random.default_rng(7)
    S, d, R = 33, 8, 1
    qs = 4.0 * rng.standard_normal(d).astype(np.float32)
    q = np.zeros((2, 2, d), np.float32)
    q[0, 0] = qs
    q[1, 1] = qs
    k = np.repeat(rng.standard_normal((S, 1, d)).astype(np.float32), 2, axis=1)
    got = one_sample(q, k, R, 2, 2, d)
    p = softmax_row(qs, k[:, 0], 1 / np.sqrt(d))
    want = 0.5 * (p + 1.0 / S)
    np.testing.assert_allclose(got, want, rtol=1e-13)
    assert not np.allclose(got[R:], np.maximum(p, 1.0 / S)[R:])


def test_identical_rows_collapse_to_one_row():
    # T copies of one row: max and mean over rows both return that row (Stage II at T=1
    # is Stage I).
    rng = np.random.default_rng(8)
    S, d, H = 50, 16, 3
    q1 = rng.standard_normal((1, H, d)).astype(np.float32)
    k = rng.standard_normal((S, H, d)).astype(np.float32)
    a = one_sample(q1, k, 4, H, H, d)
    b = one_sample(np.repeat(q1, 5, axis=0), k, 4, H, H, d)
    np.testing.assert_allclose(b, a, rtol=1e-14)


@pytest.mark.parametrize("H,T", [(1, 1), (4, 1), (16, 1)])
def test_cls_scores_sum_to_one(H, T):
    rng = np.random.default_rng(H)
    B, R, d = 3, 4, 32
    N = np.array([10, 0, 57])
    k_off = np.concatenate([[0], np.cumsum(N + R)])
    q = synth.to_bf16_bits(rng.standard_normal((B, H, d)).astype(np.float32))
    k = synth.to_bf16_bits(rng.standard_normal((k_off[-1], H, d)).astype(np.float32))
    sc = oracle.scores(q, k, np.arange(B + 1), k_off, H, H, d, R, dtype="bf16")
    for b in range(B):
        assert abs(sc[k_off[b]:k_off[b + 1]].sum() - 1.0) < 1e-12


def test_row_lse_of_the_given_keys_reproduces_the_softmax():
    rng = np.random.default_rng(9)
    S, d, H, T = 31, 8, 2, 3
    q = rng.standard_normal((T, H, d)).astype(np.float32)
    k = rng.standard_normal((S, H, d)).astype(np.float32)
    lse = np.empty((T, H))
    for t in range(T):
        for h in range(H):
            lse[t, h] = sps.logsumexp(k[:, h].astype(np.float64) @ q[t, h].astype(np.float64)
                                      / np.sqrt(d))
    a = one_sample(q, k, 2, H, H, d)
    b = one_sample(q, k, 2, H, H, d, row_lse=lse.reshape(-1))
    np.testing.assert_allclose(b, a, rtol=1e-12)


def test_row_lse_of_a_superset_equals_the_superset_softmax():
    # Normalising over extra keys that are not scored (e.g. the LLM's text tokens) gives
    # the same scores as scoring the superset and reading the original keys.
    rng = np.random.default_rng(10)
    S, extra, d, H, T, R = 20, 9, 8, 2, 2, 2
    q = rng.standard_normal((T, H, d)).astype(np.float32)
    kall = rng.standard_normal((S + extra, H, d)).astype(np.float32)
    lse = np.empty((T, H))
    for t in range(T):
        for h in range(H):
            lse[t, h] = sps.logsumexp(kall[:, h].astype(np.float64) @ q[t, h].astype(np.float64)
                                      / np.sqrt(d))
    sub = one_sample(q, kall[:S], R, H, H, d, row_lse=lse.reshape(-1))
    full = one_sample(q, kall, R, H, H, d)
    np.testing.assert_allclose(sub, full[:S], rtol=1e-12)


def test_ragged_batch_equals_samplewise_calls():
    rng = np.random.default_rng(11)
    H, Hkv, d, R = 4, 2, 16, 3
    T = np.array([1, 5, 2, 7])
    N = np.array([9, 0, 31, 4])
    q_off = np.concatenate([[0], np.cumsum(T)])
    k_off = np.concatenate([[0], np.cumsum(N + R)])
    q = rng.standard_normal((q_off[-1], H, d)).astype(np.float32)
    k = rng.standard_normal((k_off[-1], Hkv, d)).astype(np.float32)
    batch = oracle.scores(q, k, q_off, k_off, H, Hkv, d, R, dtype="f32")
    for b in range(len(T)):
        one = one_sample(q[q_off[b]:q_off[b + 1]], k[k_off[b]:k_off[b + 1]], R, H, Hkv, d)
        np.testing.assert_array_equal(batch[k_off[b]:k_off[b + 1]], one)


def test_visual_permutation_permutes_scores():
    rng = np.random.default_rng(12)
    S, d, H, T, R = 45, 8, 2, 3, 4
    q = rng.standard_normal((T, H, d)).astype(np.float32)
    k = rng.standard_normal((S, H, d)).astype(np.float32)
    perm = rng.permutation(S - R)
    kp = k.copy()
    kp[R:] = k[R:][perm]
    a = one_sample(q, k, R, H, H, d)
    b = one_sample(q, kp, R, H, H, d)
    np.testing.assert_allclose(b[:R], a[:R], rtol=1e-13)
    np.testing.assert_allclose(b[R:], a[R:][perm], rtol=1e-13)


def test_fp64_error_is_below_1e13_against_50_digit_arithmetic():
    # Tiny integer inputs; scores recomputed in mpmath at 50 digits bound the oracle's error.
    mpmath.mp.dps = 50
    rng = np.random.default_rng(13)
    for trial in range(20):
        H, Hkv, T, R, d = int(rng.integers(1, 3)), 1, int(rng.integers(1, 4)), int(rng.integers(1, 3)), 4
        Hkv = H if rng.integers(0, 2) else 1
        N = int(rng.integers(0, 11))
        S = R + N
        q = rng.integers(-2, 3, (T, H, d)).astype(np.float32)
        k = rng.integers(-2, 3, (S, Hkv, d)).astype(np.float32)
        got = one_sample(q, k, R, H, Hkv, d)
        scale = mpmath.mpf(1) / mpmath.sqrt(d)
        abar = [[mpmath.mpf(0)] * S for _ in range(T)]
        for h in range(H):
            g = h // (H // Hkv)
            for t in range(T):
                lg = [scale * sum(mpmath.mpf(float(q[t, h, e])) * float(k[s, g, e]) for e in range(d))
                      for s in range(S)]
                z = sum(mpmath.exp(x) for x in lg)
                for s in range(S):
                    abar[t][s] += mpmath.exp(lg[s]) / z / H
        for s in range(S):
            col = [abar[t][s] for t in range(T)]
            want = (sum(col) / T) if s < R else max(col)
            assert abs(got[s] - float(want)) <= 1e-13 * float(want)


# ----------------------------------------------------------------------------- mutual scoring
def mutual_sample(T_extra=0, S=40, H=3, Hkv=3, d=16, R=2, seed=30):
    """A self-attention sample: the anchor rows are the R + N tokens themselves (plus
    T_extra further rows), Eq. mutual_scoring."""
    rng = np.random.default_rng(seed)
    T = S + T_extra
    q = rng.standard_normal((T, H, d)).astype(np.float32)
    k = rng.standard_normal((S, Hkv, d)).astype(np.float32)
    return q, k


@pytest.mark.parametrize("H,Hkv", [(1, 1), (3, 3), (4, 2)])
def test_mutual_scores_sum_to_one(H, Hkv):
    # Every anchor row's head-mean map sums to 1 over the keys, so the mean over rows
    # does too; a max in place of the mean, a dropped 1/T or 1/H breaks it.
    q, k = mutual_sample(H=H, Hkv=Hkv, seed=31 + H)
    sc = one_sample(q, k, 2, H, Hkv, 16, row_reduce=oracle.ROWS_MEAN)
    assert abs(sc.sum() - 1.0) < 1e-12


def test_mutual_with_one_row_is_the_cls_score():
    q, k = mutual_sample(seed=32)
    a = one_sample(q[:1], k, 2, 3, 3, 16, row_reduce=oracle.ROWS_MEAN)
    b = one_sample(q[:1], k, 2, 3, 3, 16)
    assert np.array_equal(a, b)


def test_mutual_uniform_attention_gives_one_over_s():
    # q = 0: every row attends uniformly, so every key receives 1/S on average.
    q, k = mutual_sample(seed=33)
    sc = one_sample(np.zeros_like(q), k, 2, 3, 3, 16, row_reduce=oracle.ROWS_MEAN)
    np.testing.assert_allclose(sc, 1.0 / k.shape[0], rtol=1e-14)


def test_mutual_is_below_the_row_max_and_keeps_the_register_mean():
    q, k = mutual_sample(seed=34)
    mean = one_sample(q, k, 2, 3, 3, 16, row_reduce=oracle.ROWS_MEAN)
    mx = one_sample(q, k, 2, 3, 3, 16)
    assert np.all(mean <= mx + 1e-15)
    assert np.array_equal(mean[:2], mx[:2])          # registers take the mean either way
    assert np.any(mean[2:] < mx[2:] * 0.999)


def test_mutual_is_invariant_to_the_order_of_the_anchor_rows():
    q, k = mutual_sample(T_extra=5, seed=35)
    perm = np.random.default_rng(35).permutation(q.shape[0])
    a = one_sample(q, k, 2, 3, 3, 16, row_reduce=oracle.ROWS_MEAN)
    b = one_sample(q[perm], k, 2, 3, 3, 16, row_reduce=oracle.ROWS_MEAN)
    np.testing.assert_allclose(b, a, rtol=1e-13)


def test_mutual_equals_the_column_mean_of_a_50_digit_attention_map():
    mpmath.mp.dps = 50
    rng = np.random.default_rng(36)
    for trial in range(8):
        H, d, R, N = int(rng.integers(1, 3)), 4, int(rng.integers(1, 3)), int(rng.integers(0, 7))
        S = R + N
        q = rng.integers(-2, 3, (S, H, d)).astype(np.float32)
        k = rng.integers(-2, 3, (S, H, d)).astype(np.float32)
        got = one_sample(q, k, R, H, H, d, row_reduce=oracle.ROWS_MEAN)
        scale = mpmath.mpf(1) / mpmath.sqrt(d)
        for s in range(S):
            acc = mpmath.mpf(0)
            for u in range(S):
                for h in range(H):
                    lg = [scale * sum(mpmath.mpf(float(q[u, h, e])) * float(k[j, h, e]) for e in range(d))
                          for j in range(S)]
                    acc += mpmath.exp(lg[s]) / sum(mpmath.exp(x) for x in lg) / H
            want = acc / S
            assert abs(got[s] - float(want)) <= 1e-13 * float(want)


def test_oracle_rejects_an_unknown_row_reduction():
    q, k = mutual_sample(seed=37)
    with pytest.raises(ValueError):
        one_sample(q, k, 2, 3, 3, 16, row_reduce=2)


# ----------------------------------------------------------------------------- step 3
@pytest.mark.parametrize("reduce,fn", [(oracle.REG_MEAN, np.mean), (oracle.REG_MAX, np.max),
                                       (oracle.REG_SUM, np.sum)])
def test_threshold_reductions(reduce, fn):
    rng = np.random.default_rng(14)
    R, N, B = 4, 6, 3
    k_off = np.arange(B + 1) * (R + N)
    sc = rng.random(k_off[-1])
    tau = oracle.threshold(sc, k_off, R, 0.3, reduce)
    for b in range(B):
        assert tau[b] == pytest.approx(0.3 * fn(sc[k_off[b]:k_off[b] + R]), rel=1e-15)


def test_threshold_rejects_bad_lambda():
    with pytest.raises(ValueError):
        oracle.threshold(np.ones(5), [0, 5], 1, -0.1)
    with pytest.raises(ValueError):
        oracle.threshold(np.ones(5), [0, 5], 1, float("nan"))


# ----------------------------------------------------------------------------- steps 4-5
def test_closed_form_single_head_mean_register():
    # H = T = 1, MEAN over R registers: keep(v) <=> l_v - (logsumexp_r l_r - ln R) >= ln lambda.
    # The softmax denominator cancels, so the decision needs no normaliser.
    rng = np.random.default_rng(15)
    d, R, N = 16, 3, 200
    for trial in range(10):
        q = rng.standard_normal((1, 1, d)).astype(np.float32)
        k = rng.standard_normal((R + N, 1, d)).astype(np.float32)
        lam = float(np.float32(rng.uniform(0.05, 3.0)))
        res = oracle.prune(f32(q), f32(k), [0, 1], [0, R + N], 1, 1, d, R, lam, dtype="f32")
        lg = (k[:, 0].astype(np.float64) @ q[0, 0].astype(np.float64)) / np.sqrt(d)
        margin = lg[R:] - (sps.logsumexp(lg[:R]) - np.log(R)) - np.log(lam)
        clear = np.abs(margin) > 1e-9
        want = np.flatnonzero(margin >= 0)
        got = res["kept_idx"]
        assert set(got[np.isin(got, np.flatnonzero(clear))]) == set(want[clear[want]])


def test_adding_a_key_changes_no_other_decision():
    # Same closed form: planting any extra key (a sink) leaves every other decision as it was.
    rng = np.random.default_rng(16)
    d, R, N = 16, 2, 120
    q = rng.standard_normal((1, 1, d)).astype(np.float32)
    k = rng.standard_normal((R + N, 1, d)).astype(np.float32)
    sink = 8.0 * rng.standard_normal((1, 1, d)).astype(np.float32)
    k2 = np.concatenate([k, sink])
    a = oracle.prune(k=k, q=q, q_off=[0, 1], k_off=[0, R + N], H=1, Hkv=1, d=d, R=R, lam=0.7,
                     dtype="f32")
    b = oracle.prune(k=k2, q=q, q_off=[0, 1], k_off=[0, R + N + 1], H=1, Hkv=1, d=d, R=R, lam=0.7,
                     dtype="f32")
    assert list(b["kept_idx"][b["kept_idx"] < N]) == list(a["kept_idx"])


def test_ties_at_the_threshold_are_kept():
    # A visual key equal to the (single) register scores exactly s(r): kept at lambda = 1
    # (the rule is >=), dropped just above.
    rng = np.random.default_rng(17)
    d = 8
    q = rng.standard_normal((1, 2, d)).astype(np.float32)
    k = rng.standard_normal((12, 2, d)).astype(np.float32)
    k[5] = k[0]                                   # visual token 4 == register
    at = oracle.prune(q, k, [0, 1], [0, 12], 2, 2, d, 1, 1.0, dtype="f32")
    above = oracle.prune(q, k, [0, 1], [0, 12], 2, 2, d, 1, float(np.nextafter(np.float32(1), 2)),
                         dtype="f32")
    assert at["scores"][5] == at["scores"][0]
    assert 4 in set(at["kept_idx"]) and 4 not in set(above["kept_idx"])


def test_lambda_zero_keeps_all_and_sets_nest():
    rng = np.random.default_rng(18)
    B, R, N, H, d = 3, 4, 80, 4, 16
    k_off = np.arange(B + 1) * (R + N)
    q = rng.standard_normal((B, H, d)).astype(np.float32)
    k = rng.standard_normal((k_off[-1], H, d)).astype(np.float32)
    sc = oracle.scores(q, k, np.arange(B + 1), k_off, H, H, d, R, dtype="f32")
    prev = None
    for lam in [0.0, 0.05, 0.2, 0.5, 1.0, 2.0, 5.0, 1e6]:
        tau = oracle.threshold(sc, k_off, R, lam)
        kept, cnt, offs = oracle.select(sc, tau, k_off, R)
        sets = [set(kept[offs[b]:offs[b + 1]]) for b in range(B)]
        if lam == 0.0:
            assert all(c == N for c in cnt)
        if lam == 1e6:
            assert all(c == 0 for c in cnt)
        if prev is not None:
            assert all(s <= p for s, p in zip(sets, prev))
        prev = sets


def test_selection_is_top_k_by_score():
    # Any lambda selects exactly the K highest-scoring visual tokens, K = |S_lambda|
    # (argsort, Sec. 3.2 top-K rule): the relative test is a score threshold.
    rng = np.random.default_rng(19)
    R, N, H, d = 2, 300, 3, 16
    q = rng.standard_normal((1, H, d)).astype(np.float32)
    k = rng.standard_normal((R + N, H, d)).astype(np.float32)
    for lam in [0.1, 0.6, 1.0, 1.7]:
        res = oracle.prune(q, k, [0, 1], [0, R + N], H, H, d, R, lam, dtype="f32")
        K = int(res["kept_count"][0])
        top = np.argsort(-res["scores"][R:], kind="stable")[:K]
        assert set(top) == set(res["kept_idx"])


def test_bookkeeping_and_index_map():
    rng = np.random.default_rng(20)
    B, R = 4, 2
    N = np.array([7, 0, 13, 5])
    k_off = np.concatenate([[0], np.cumsum(N + R)])
    sc = rng.random(k_off[-1])
    tau = rng.random(B) * 0.8
    imap = rng.permutation(10000)[:N.sum()].astype(np.int32)
    kept, cnt, offs = oracle.select(sc, tau, k_off, R)
    kept_m, cnt_m, offs_m = oracle.select(sc, tau, k_off, R, index_map=imap)
    assert offs[0] == 0 and np.array_equal(np.diff(offs), cnt)
    co = np.concatenate([[0], np.cumsum(N)])
    for b in range(B):
        seg = kept[offs[b]:offs[b + 1]]
        want = np.flatnonzero(sc[k_off[b] + R:k_off[b + 1]] >= tau[b])
        assert np.array_equal(seg, want)
        assert np.all(np.diff(seg) > 0) and np.all((seg >= 0) & (seg < N[b]))
        assert np.array_equal(kept_m[offs[b]:offs[b + 1]], imap[co[b] + seg])
    assert np.array_equal(cnt, cnt_m)


def test_brute_force_subset_and_breakpoint_sweep():
    # Tiny inputs: the kept set is the only subset consistent with the predicate, and
    # sweeping lambda across every ratio breakpoint moves the count by exactly the
    # number of tokens that share that ratio (exact ties made with duplicated keys).
    rng = np.random.default_rng(21)
    d, R, H = 4, 1, 2
    for trial in range(8):
        N = int(rng.integers(3, 10))
        base = rng.integers(-2, 3, (N, H, d)).astype(np.float32)
        base[rng.integers(0, N)] = base[0]                      # at least one exact tie
        k = np.concatenate([rng.integers(-2, 3, (R, H, d)).astype(np.float32), base])
        q = rng.integers(-2, 3, (1, H, d)).astype(np.float32)
        sc = oracle.scores(q, k, [0, 1], [0, R + N], H, H, d, R, dtype="f32")
        ratio = sc[R:] / sc[:R].mean()
        uniq, mult = np.unique(ratio, return_counts=True)
        for lam, m in zip(uniq, mult):
            below = oracle.select(sc, oracle.threshold(sc, [0, R + N], R, lam * (1 - 1e-9)),
                                  [0, R + N], R)[1][0]
            at = oracle.select(sc, oracle.threshold(sc, [0, R + N], R, lam * (1 + 1e-9)),
                               [0, R + N], R)[1][0]
            assert below - at == m
        lam = float(np.median(ratio)) * 1.000001
        kept = set(oracle.prune(q, k, [0, 1], [0, R + N], H, H, d, R, lam, dtype="f32")["kept_idx"])
        consistent = []
        for mask in range(1 << N):
            S = {v for v in range(N) if mask >> v & 1}
            if all((ratio[v] >= lam) == (v in S) for v in range(N)):
                consistent.append(S)
        assert consistent == [kept]


def test_gather_is_a_row_copy():
    rng = np.random.default_rng(22)
    B, R = 3, 2
    N = np.array([6, 3, 9])
    k_off = np.concatenate([[0], np.cumsum(N + R)])
    co = np.concatenate([[0], np.cumsum(N)])
    hidden = rng.integers(0, 1 << 16, (N.sum(), 24), dtype=np.int64).astype(np.uint16)
    krows = rng.standard_normal((k_off[-1], 8)).astype(np.float32)
    sc = rng.random(k_off[-1])
    kept, cnt, offs = oracle.select(sc, np.full(B, 0.5), k_off, R)
    g1 = oracle.gather(hidden, kept, offs, k_off, R, src_pad_rows=0, src_row0=0)
    g2 = oracle.gather(krows, kept, offs, k_off, R, src_pad_rows=R, src_row0=R)
    for b in range(B):
        seg = kept[offs[b]:offs[b + 1]]
        assert np.array_equal(g1[offs[b]:offs[b + 1]], np.take(hidden, co[b] + seg, axis=0))
        assert np.array_equal(g2[offs[b]:offs[b + 1]], np.take(krows, k_off[b] + R + seg, axis=0))


# ----------------------------------------------------------------------------- sinks (A13)
def test_register_absorption_suppresses_a_planted_sink():
    # Register construction (Algorithm 1; Eq. register_redirect_appendix) moves the sink's
    # high-norm component into the register.  In key space: a sink k_i = a * k0 becomes k0
    # and the register gains (a - 1) * k0.  On raw keys the sink is kept; after absorption
    # it falls below the register anchor while the planted informative keys stay, and the
    # visual attention spreads out (n_eff rises, Sec. 3.2 Obs. 1).
    H, d, N, alpha, n_inf, lam = 16, 64, 576, 8.0, 20, 0.045
    raw_kept = abs_kept = 0
    inf_kept = inf_total = 0
    neff_raw, neff_abs = [], []
    seeds = range(40)
    for seed in seeds:
        rng = np.random.default_rng(1000 + seed)
        q = rng.standard_normal((1, H, d)).astype(np.float32)
        k = rng.standard_normal((1 + N, H, d)).astype(np.float32)
        perm = rng.permutation(N)
        sink, inf = perm[0], perm[1:1 + n_inf]
        qh = q[0] / np.linalg.norm(q[0], axis=-1, keepdims=True)
        for v in inf:
            u = rng.standard_normal((H, d))
            u -= np.sum(u * qh, -1, keepdims=True) * qh
            u /= np.linalg.norm(u, axis=-1, keepdims=True)
            nrm = np.linalg.norm(k[1 + v], axis=-1, keepdims=True)
            k[1 + v] = nrm * (0.6 * qh + 0.8 * u)
        k0 = k[1 + sink].copy()
        raw = k.copy()
        raw[1 + sink] = alpha * k0
        absd = k.copy()
        absd[0] = k[0] + (alpha - 1.0) * k0
        r = oracle.prune(q, raw, [0, 1], [0, 1 + N], H, H, d, 1, lam, dtype="f32")
        a = oracle.prune(q, absd, [0, 1], [0, 1 + N], H, H, d, 1, lam, dtype="f32")
        raw_kept += sink in set(r["kept_idx"])
        abs_kept += sink in set(a["kept_idx"])
        inf_kept += len(set(inf) & set(a["kept_idx"]))
        inf_total += n_inf
        vr, va = r["scores"][1:], a["scores"][1:]
        neff_raw.append(oracle.neff(vr / vr.sum()))
        neff_abs.append(oracle.neff(va / va.sum()))
    assert raw_kept == len(seeds)
    assert abs_kept <= 0.05 * len(seeds)
    assert inf_kept == inf_total
    assert np.mean(neff_abs) > np.mean(neff_raw)


# ----------------------------------------------------------------------------- helpers of the paper
def test_neff_closed_forms():
    assert oracle.neff(np.full(37, 1 / 37)) == pytest.approx(37, rel=1e-12)
    assert oracle.neff(np.eye(1, 9)[0]) == pytest.approx(1.0, rel=1e-15)
    p = 0.3
    assert oracle.neff([p, 1 - p]) == pytest.approx(np.exp(-(p * np.log(p) + (1 - p) * np.log(1 - p))))


def test_budget_matching_hits_the_best_level():
    rng = np.random.default_rng(23)
    for trial in range(10):
        D = int(rng.integers(1, 6))
        lists = [np.round(rng.random(int(rng.integers(0, 30))) * 4, 1) for _ in range(D)]
        target = float(rng.uniform(0, 20))
        lam = oracle.match_lambda(lists, target)
        mean_count = lambda l: np.mean([np.sum(x >= l) for x in lists])
        grid = np.concatenate([np.unique(np.concatenate(lists + [np.zeros(0)])), [0.0, 1e9]])
        best = min(abs(mean_count(g) - target) for g in grid)
        assert abs(mean_count(lam) - target) == pytest.approx(best)
        assert abs(mean_count(np.float32(lam)) - target) == pytest.approx(best)


def test_paper_stage1_table_lambda_zero_keeps_all_and_counts_fall():
    # The paper's lambda_1 sweep on LLaVA-NeXT (Table tab:lamda1cc): lambda_1 = 0 keeps all
    # 2880 tokens and N_1 falls as lambda_1 rises.  Real-data counts are not reproducible
    # here; the zero point and the monotone trend are.
    with open(os.path.join(GOLDEN, "paper_stage1_lambda_sweep.json")) as f:
        table = json.load(f)
    lams = [row["lambda1"] for row in table["rows"]]
    n1 = [row["N1"] for row in table["rows"]]
    assert lams[0] == 0 and n1[0] == table["visual_tokens"] == 2880
    order = np.argsort(lams)
    assert all(np.diff(np.array(n1)[order]) <= 0)
    sb = synth.make_stage("llava_next", "vis", B=1, payload=False)
    sc = oracle.scores(sb.q, sb.k, sb.q_off, sb.k_off, sb.H, sb.Hkv, sb.d, sb.R, dtype="bf16")
    counts = []
    for lam in sorted(lams):
        tau = oracle.threshold(sc, sb.k_off, sb.R, lam)
        counts.append(int(oracle.select(sc, tau, sb.k_off, sb.R)[1][0]))
    assert counts[0] == 2880
    assert all(np.diff(counts) <= 0)


# ----------------------------------------------------------------------------- register construction
def redirect_case(seed=40, B=3, R=2, N=(7, 0, 12), width=9):
    rng = np.random.default_rng(seed)
    N = np.asarray(N)
    k_off = np.concatenate([[0], np.cumsum(N + R)]).astype(np.int64)
    h = rng.standard_normal((int(k_off[-1]), width)).astype(np.float32)
    return h, k_off, R


def test_register_redirect_moves_the_channel_max_and_zeroes_the_visual_rows():
    h, k_off, R = redirect_case()
    chans = [5, 1]
    out = oracle.register_redirect(h, k_off, R, chans, reg_slot=1, dtype="f32")
    for b in range(len(k_off) - 1):
        lo, hi = k_off[b], k_off[b + 1]
        vis = slice(lo + R, hi)
        for c in range(h.shape[1]):
            if c in chans and hi - lo > R:
                assert out[lo + 1, c] == np.max(h[vis, c])     # numpy's max, to the bit
                assert np.all(out[vis, c] == 0.0)
                assert out[lo, c] == h[lo, c]                 # the other register row
            else:
                assert np.array_equal(out[lo:hi, c], h[lo:hi, c])


def test_register_redirect_leaves_an_empty_sample_alone():
    h, k_off, R = redirect_case(seed=41)
    out = oracle.register_redirect(h, k_off, R, [0, 3], dtype="f32")
    assert np.array_equal(out[k_off[1]:k_off[2]], h[k_off[1]:k_off[2]])


def test_register_redirect_ignores_repeats_and_out_of_range_channels():
    h, k_off, R = redirect_case(seed=42)
    a = oracle.register_redirect(h, k_off, R, [2, 7, 2, -1, 9, 100], dtype="f32")
    b = oracle.register_redirect(h, k_off, R, [2, 7], dtype="f32")
    assert np.array_equal(a, b)


def test_register_redirect_bf16_keeps_the_bits_and_writes_plus_zero():
    h, k_off, R = redirect_case(seed=43)
    h[k_off[0] + R:k_off[1], 4] = -np.abs(h[k_off[0] + R:k_off[1], 4])   # all <= 0 ...
    h[k_off[0] + R + 3, 4] = -0.0                                       # ... max is -0
    bits = synth.to_bf16_bits(h)
    out = oracle.register_redirect(bits, k_off, R, [4, 6], dtype="bf16")
    assert out[k_off[0], 4] == 0x0000                                   # +0, not 0x8000
    vis = slice(k_off[2] + R, k_off[3])
    want = bits[vis, 6][np.argmax(h[vis, 6])]
    assert out[k_off[2], 6] == want
    assert np.all(out[vis, 6] == 0)


def test_register_redirect_absorbs_a_sink_channel():
    # A planted high-activation channel of one patch (the sink pattern the register
    # construction targets) ends up in the register, and no visual row keeps it.
    h, k_off, R = redirect_case(seed=44, B=1, N=(30,), width=16)
    h[R + 11, 9] = 80.0
    out = oracle.register_redirect(h, k_off, R, [9], dtype="f32")
    assert out[0, 9] == 80.0 and np.max(np.abs(out[R:, 9])) == 0.0
    assert np.linalg.norm(out[R + 11]) < 0.5 * np.linalg.norm(h[R + 11])


def test_budget_matching_tie_rule_and_interval_ends():
    # Ratios 1..4 of one sample: counts 4, 3, 2, 1 at 1, 2, 3, 4.  A target of 2.5 is
    # equally far from 2 and 3: the smaller count wins, lambda = sqrt(3 * 2).
    assert oracle.match_lambda([np.array([1.0, 2.0, 3.0, 4.0])], 2.5) == pytest.approx(np.sqrt(6))
    # Beyond every candidate: the lowest level, half its ratio (no ratio below it).
    assert oracle.match_lambda([np.array([1.0, 2.0, 3.0, 4.0])], 100.0) == 0.5
    # Two samples: the mean count is halved; target 1 = count 2 over the batch.
    lam = oracle.match_lambda([np.array([4.0, 1.0]), np.array([3.0, 2.0])], 1.0)
    assert lam == pytest.approx(np.sqrt(3 * 2))
    assert oracle.match_lambda([np.zeros(0)], 3.0) == 1.0


# ----------------------------------------------------------------------------- ablation
def test_mean_threshold_hand_example_and_invariants():
    # Table tab:qwen_compact_component_ablation, mean-based threshold: tau = lambda * mean
    # of the visual scores; the register scores do not enter.
    sc = np.array([0.1, 0.2, 0.3, 0.1, 0.3, 0.05, 0.9, 0.4, 0.4, 0.4])
    k_off = [0, 6, 10]
    tau = oracle.threshold(sc, k_off, 2, 1.0, oracle.CAND_MEAN)
    assert tau[0] == pytest.approx(0.75 / 4) and tau[1] == pytest.approx(0.4)
    rng = np.random.default_rng(41)
    R, N = 3, 200
    s = rng.random(R + N)
    t1 = oracle.threshold(s, [0, R + N], R, 1.3, oracle.CAND_MEAN)
    s2 = s.copy()
    s2[:R] = rng.random(R) * 50                        # registers changed: same threshold
    assert oracle.threshold(s2, [0, R + N], R, 1.3, oracle.CAND_MEAN)[0] == t1[0]
    # Scale invariance of the decisions, and lambda = 1 keeps some but not all tokens.
    kept1 = oracle.select(s, t1, [0, R + N], R)[0]
    t3 = oracle.threshold(s * 8.0, [0, R + N], R, 1.3, oracle.CAND_MEAN)
    assert np.array_equal(oracle.select(s * 8.0, t3, [0, R + N], R)[0], kept1)
    t_one = oracle.threshold(s, [0, R + N], R, 1.0, oracle.CAND_MEAN)
    n_one = len(oracle.select(s, t_one, [0, R + N], R)[0])
    assert 0 < n_one < N
    # Uniform visual scores: lambda = 1 keeps all, anything above keeps none.
    u = np.concatenate([s[:R], np.full(N, 0.125)])
    for lam, want in ((1.0, N), (1.0 + 1e-12, 0)):
        t = oracle.threshold(u, [0, R + N], R, lam, oracle.CAND_MEAN)
        assert len(oracle.select(u, t, [0, R + N], R)[0]) == want
    # No visual tokens: tau = 0, nothing to keep.
    assert oracle.threshold(s[:R], [0, R], R, 2.0, oracle.CAND_MEAN)[0] == 0.0


def test_topk_is_the_sorted_prefix():
    # Fixed budget: the K best by (score desc, index asc), i.e. numpy's stable lexsort.
    rng = np.random.default_rng(43)
    R = 2
    N = np.array([0, 1, 7, 40, 300])
    k_off = np.concatenate([[0], np.cumsum(N + R)])
    sc = np.round(rng.random(int(k_off[-1])) * 16) / 16   # many ties
    for K in (0, 1, 5, 40, 1000):
        kept, cnt, offs = oracle.select_topk(sc, k_off, R, K)
        for b in range(len(N)):
            sv = sc[k_off[b] + R:k_off[b + 1]]
            order = np.lexsort((np.arange(N[b]), -sv))       # last key sorts first
            want = np.sort(order[:K])
            got = kept[offs[b]:offs[b + 1]]
            assert np.array_equal(got, want), (b, K)
            assert cnt[b] == min(K, N[b])
            # Every kept token beats every dropped one (or ties with a lower index).
            drop = np.setdiff1d(np.arange(N[b]), got)
            for v in got:
                assert np.all((sv[v] > sv[drop]) | ((sv[v] == sv[drop]) & (v < drop)))


def test_topk_matches_the_threshold_rule_without_ties_and_maps_indices():
    # With distinct scores, keeping the K best equals the threshold rule at the K-th
    # largest score; index_map entries replace the local indices.
    rng = np.random.default_rng(47)
    R, N = 1, 500
    sc = rng.random(R + N)
    for K in (1, 17, 250, 499):
        kth = np.sort(sc[R:])[::-1][K - 1]
        kept_t = oracle.select(sc, np.array([kth]), [0, R + N], R)[0]
        assert np.array_equal(oracle.select_topk(sc, [0, R + N], R, K)[0], kept_t)
    im = (np.arange(N) * 7 + 3).astype(np.int32)
    kept, _, _ = oracle.select_topk(sc, [0, R + N], R, 10)
    kept_m, _, _ = oracle.select_topk(sc, [0, R + N], R, 10, index_map=im)
    assert np.array_equal(kept_m, im[kept])
