"""GPU parity over seeded random shapes: head counts, grouped-query ratios, head dimensions,
register counts, ragged row and key counts and lambdas drawn from a fixed generator, on the
three scoring forms (one anchor row: VALU; several rows, max over rows: MFMA; mutual
scoring, every token an anchor row and the mean over rows: MFMA), against the fp64 oracle.

The shapes stay inside what the library accepts (bf16 head dimensions a multiple of 8,
float32 a multiple of 4; the MFMA path takes bf16 with d <= 128; one-row queries of at most
24 KB, inside the LDS bound of the one-row kernel), so every case must pass the same
acceptance rules as the workload tests.
"""
import numpy as np
import pytest

from paper_2605_29657_amd.runner import DeviceStage
from parity import RTOL, check_rows, check_scores, check_selection, custom_stage, oracle_prune

pytestmark = pytest.mark.gpu


def _cases(n=48, seed=2605):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        form = ("vis", "txt", "mut")[i % 3]
        text = form != "vis"
        dtype = "bf16" if text or rng.random() < 0.6 else "f32"
        step = 8 if dtype == "bf16" else 4
        d = int(rng.integers(1, (128 if text else 256) // step + 1)) * step
        heads = [1, 2, 3, 4, 6, 8, 12, 16, 24, 32] + ([] if text else [48, 64])
        if not text:
            heads = [h for h in heads if h * d * (2 if dtype == "bf16" else 4) <= 24576]
        H = int(rng.choice(heads))
        Hkv = int(rng.choice([g for g in range(1, H + 1) if H % g == 0]))
        R = int(rng.choice([1, 1, 2, 4, 8, 32]))
        B = int(rng.integers(1, 5))
        N = [int(x) for x in rng.integers(0, 400 if form == "mut" else 700, size=B)]
        if form == "mut":
            T = [n_ + R for n_ in N]
        else:
            T = [int(x) for x in rng.integers(2, 300, size=B)] if text else [1] * B
        lam = float(rng.choice([0.5, 1.0, 2.0]))
        out.append((i, form, dtype, B, R, H, Hkv, d, T, N, lam))
    return out


@pytest.mark.parametrize("case", _cases(), ids=lambda c: "case%d" % c[0])
def test_random_shape(case):
    i, form, dtype, B, R, H, Hkv, d, T, N, lam = case
    print("case%d: %s dtype=%s B=%d R=%d H=%d Hkv=%d d=%d T=%s N=%s lam=%g" % (
        i, form, dtype, B, R, H, Hkv, d, T, N, lam), flush=True)
    sb = custom_stage(B=B, R=R, H=H, Hkv=Hkv, d=d, T=T, N=N, dtype=dtype, seed=1000 + i,
                      stage=form)
    ds = DeviceStage(sb, ragged=True)
    ds.prune(lam)
    g = ds.host()
    o = oracle_prune(sb, lam)
    rtol = RTOL[dtype]
    check_scores(g["scores"], o["scores"], rtol)
    check_scores(g["tau"], o["tau"], rtol, "tau")
    check_selection(g, o, sb, rtol)
    check_rows(g, sb)


@pytest.mark.parametrize("case", _cases()[:24], ids=lambda c: "case%d" % c[0])
def test_random_shape_unfused_equals_fused(case):
    # occam_score, occam_threshold, occam_select and occam_gather in turn give the fused
    # prune's scores, tau, survivors and rows bit for bit (the fused kernels run the same
    # arithmetic in the same order).
    import torch
    from paper_2605_29657_amd import occam
    i, form, dtype, B, R, H, Hkv, d, T, N, lam = case
    print("case%d: %s dtype=%s B=%d R=%d H=%d Hkv=%d d=%d T=%s N=%s lam=%g" % (
        i, form, dtype, B, R, H, Hkv, d, T, N, lam), flush=True)
    sb = custom_stage(B=B, R=R, H=H, Hkv=Hkv, d=d, T=T, N=N, dtype=dtype, seed=1000 + i,
                      stage=form)
    ds = DeviceStage(sb, ragged=True)
    ds.prune(lam)
    fused = ds.host()
    p, dev = ds.problem, "cuda"
    scores = torch.empty(ds.total_keys, dtype=torch.float32, device=dev)
    tau = torch.empty(sb.B, dtype=torch.float32, device=dev)
    kept = torch.empty(max(ds.total_cands, 1), dtype=torch.int32, device=dev)
    cnt = torch.empty(sb.B, dtype=torch.int32, device=dev)
    offs = torch.empty(sb.B + 1, dtype=torch.int32, device=dev)
    occam.score(p, ds.q, ds.k, scores, ds.ws)
    occam.threshold(p, scores, lam, occam.REG_MEAN, tau)
    occam.select(p, scores, tau, kept, cnt, offs, ds.ws)
    dsts = [torch.zeros_like(x) for x in ds.row_dst]
    rows = [occam.Rows(s, x, src_pad_rows=pl.pad_rows, src_row0=pl.row0)
            for s, x, pl in zip(ds.row_src, dsts, sb.payload)]
    occam.gather(p, rows, kept, offs)
    torch.cuda.synchronize()
    total = int(offs[-1])
    assert np.array_equal(scores.cpu().numpy(), fused["scores"])
    assert np.array_equal(tau.cpu().numpy(), fused["tau"])
    assert np.array_equal(kept[:total].cpu().numpy(), fused["kept_idx"])
    assert np.array_equal(offs.cpu().numpy(), fused["kept_offsets"])
    for x, want in zip(dsts, fused["rows"]):
        got = x[:total].cpu()
        got = got.view(torch.int16).numpy().view(np.uint16) if got.dtype == torch.bfloat16 else got.numpy()
        assert np.array_equal(got.view(np.uint8), want.view(np.uint8))
