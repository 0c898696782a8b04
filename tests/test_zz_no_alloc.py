"""occam_prune_noalloc (the library's built-in workspace) against occam_prune (a workspace
of the caller's): both run the same kernels, so every output must be bit-identical.

Two calls in a row per stage, the second on a smaller batch than the first, so that the
second call reads nothing the first one left in the shared built-in workspace.
"""
import numpy as np
import pytest
import torch

from paper_2605_29657_amd import occam, synth
from paper_2605_29657_amd.runner import DeviceStage

from parity import lam_for

pytestmark = pytest.mark.gpu


def both(sb, lam, ragged=None):
    """occam_prune on a workspace of its own, then occam_prune_noalloc into fresh outputs;
    returns the host copies of both."""
    ds = DeviceStage(sb, ragged=ragged)
    ds.prune(lam)
    ref = ds.host()
    o = occam.prune_outputs(sb.B, ds.total_cands, ds.total_keys)
    dst = [torch.full_like(d, 0) for d in ds.row_dst]
    rows = [occam.Rows(r.src, d, src_pad_rows=r.c.src_pad_rows, src_row0=r.c.src_row0)
            for r, d in zip(ds.rows, dst)]
    occam.prune_noalloc(ds.problem, ds.q, ds.k, lam, o["kept_idx"], o["kept_count"],
                        o["kept_offsets"], rows=rows, scores=o["scores"], tau=o["tau"])
    torch.cuda.synchronize()
    total = int(o["kept_offsets"][-1].item())
    got = dict(scores=o["scores"][:ds.total_keys].cpu().numpy(), tau=o["tau"].cpu().numpy(),
               kept_count=o["kept_count"].cpu().numpy(),
               kept_offsets=o["kept_offsets"].cpu().numpy(),
               kept_idx=o["kept_idx"][:total].cpu().numpy(),
               rows=[d[:total].cpu().view(torch.int16).numpy() if d.dtype == torch.bfloat16
                     else d[:total].cpu().numpy() for d in dst])
    return ref, got


def same(ref, got, what):
    for key in ("scores", "tau", "kept_count", "kept_offsets", "kept_idx"):
        a, b = np.asarray(ref[key]), np.asarray(got[key])
        assert a.shape == b.shape, (what, key)
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), (what, key)
    for i, (a, b) in enumerate(zip(ref["rows"], got["rows"])):
        assert np.array_equal(np.asarray(a).view(np.uint8), np.asarray(b).view(np.uint8)), \
            (what, "rows", i)


@pytest.mark.parametrize("stage", ["txt", "vis"])
def test_noalloc_matches_prune_twice_shrinking(stage):
    # First the LLaVA-NeXT shape (4 samples of 2884 keys), then a smaller LLaVA-1.5 batch.
    for name, B in (("llava_next", 4), ("llava15", 2)):
        sb = synth.make_stage(name, stage, B=B)
        print("case: noalloc %s/%s B=%d" % (name, stage, B), flush=True)
        ref, got = both(sb, lam_for(name, stage))
        same(ref, got, "%s/%s" % (name, stage))


def test_noalloc_ragged_after_uniform():
    # A ragged Qwen3-VL text batch (several row blocks, d = 128), then two of its samples.
    for B in (4, 2):
        sb = synth.make_stage("qwen3vl_ragged", "txt", B=B)
        print("case: noalloc qwen3vl_ragged/txt B=%d" % B, flush=True)
        ref, got = both(sb, lam_for("qwen3vl_ragged", "txt"), ragged=True)
        same(ref, got, "qwen3vl_ragged B=%d" % B)
