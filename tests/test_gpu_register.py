"""GPU parity of the test-time register construction (Algorithm 1; Appendix Eq.
register_redirect_appendix): the activation tensor after occam_register_redirect must
equal the oracle's, bit for bit (a maximum and zeros are exact)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2605_29657_amd import occam, synth

pytestmark = pytest.mark.gpu


def run_case(N, R, width, channels, reg_slot, dtype, seed, pad=0, ragged=True):
    print("case: N=%s R=%d width=%d channels=%s reg_slot=%d dtype=%s pad=%d ragged=%s" % (
        list(N)[:6], R, width, list(channels)[:12], reg_slot, dtype, pad, ragged), flush=True)
    rng = np.random.default_rng(seed)
    N = np.asarray(N, dtype=np.int64)
    B = len(N)
    k_off = np.concatenate([[0], np.cumsum(N + R)]).astype(np.int64)
    rows = int(k_off[-1])
    h32 = rng.standard_normal((rows, width + pad)).astype(np.float32)
    h32[rng.integers(0, rows, 5), rng.integers(0, width, 5)] *= 40.0     # a few sink-like values
    if dtype == "bf16":
        host = synth.to_bf16_bits(h32)
        dev = torch.from_numpy(host.view(np.int16)).cuda().view(torch.bfloat16)
    else:
        host = h32
        dev = torch.from_numpy(host).cuda()
    view = dev[:, :width]                                   # rows `width + pad` elements apart
    ch = torch.tensor(np.asarray(channels, dtype=np.int32), device="cuda")
    if ragged:
        p = occam.Problem(B, 16, 16, 64, R, key_offsets=torch.tensor(k_off.astype(np.int32),
                                                                      device="cuda"),
                          max_cands=int(N.max()), dtype=dtype)
    else:
        p = occam.Problem(B, 16, 16, 64, R, cands=int(N[0]), dtype=dtype)
    occam.register_redirect(p, view, ch, reg_slot=reg_slot)
    torch.cuda.synchronize()
    if dtype == "bf16":
        got = dev.view(torch.int16).cpu().numpy().view(np.uint16)
    else:
        got = dev.cpu().numpy()
    want = oracle.register_redirect(host[:, :width], k_off, R, channels, reg_slot=reg_slot,
                                    dtype=dtype)
    assert np.array_equal(got[:, :width].view(np.uint32 if dtype == "f32" else np.uint16),
                          want.view(np.uint32 if dtype == "f32" else np.uint16))
    assert np.array_equal(got[:, width:], host[:, width:])  # the padding is never touched


def test_bf16_ragged_with_an_empty_sample_repeats_and_bad_indices():
    run_case([300, 0, 1, 577], R=4, width=4096, channels=[11, 4095, 7, 11, -3, 4096, 0, 2048],
             reg_slot=2, dtype="bf16", seed=1)


def test_f32_uniform_padded_rows():
    run_case([576] * 3, R=1, width=1024, channels=list(range(3, 1024, 97)), reg_slot=0,
             dtype="f32", seed=2, pad=8, ragged=False)


def test_llava_next_shape_ten_channels():
    # 32 images x (4 registers + 2880 patches), a 1024-wide activation, the paper's ten
    # register neurons (indices drawn at random here).
    chans = np.random.default_rng(3).choice(1024, 10, replace=False)
    run_case([2880] * 32, R=4, width=1024, channels=chans, reg_slot=0, dtype="bf16", seed=3,
             ragged=False)


def test_no_channels_is_a_no_op():
    run_case([10, 20], R=2, width=64, channels=[], reg_slot=1, dtype="bf16", seed=4)
