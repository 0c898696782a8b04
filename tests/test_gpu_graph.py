"""The library under HIP graph capture: every call enqueues kernels on the caller's stream
only (no allocation, no host synchronisation, no memset nodes), so a fused prune can be
captured once and replayed.  Each replay is checked bit for bit against the eager result,
with eager work and synchronisations between the replays."""
import numpy as np
import pytest
import torch

from paper_2605_29657_amd import occam, synth
from paper_2605_29657_amd.runner import DeviceStage

from parity import custom_stage, lam_for

pytestmark = pytest.mark.gpu


def snapshot(ds):
    torch.cuda.synchronize()
    return {k: v.clone() for k, v in ds.out.items()}, [d.clone() for d in ds.row_dst]


def assert_same(a, b):
    outs_a, rows_a = a
    outs_b, rows_b = b
    total = int(outs_b["kept_offsets"][-1])
    for k in outs_a:
        x, y = outs_a[k], outs_b[k]
        if k == "kept_idx":                 # entries past the packed total are not written
            x, y = x[:total], y[:total]
        assert torch.equal(x, y), k
    for x, y in zip(rows_a, rows_b):
        assert torch.equal(x.view(torch.uint8) if x.dtype != torch.uint8 else x,
                           y.view(torch.uint8) if y.dtype != torch.uint8 else y)


@pytest.mark.parametrize("name,stage", [("llava15", "vis"), ("llava15", "txt"),
                                        ("llava15", "mut"), ("qwen3vl_ragged", "txt")])
def test_captured_prune_replays_bitwise(name, stage):
    print("case: graph %s/%s" % (name, stage), flush=True)
    if name == "qwen3vl_ragged":
        sb = synth.make_stage(name, stage, samples=[0, 1, 2])
    else:
        sb = synth.make_stage(name, stage, B=3)
    lam = lam_for(name, stage)
    ds = DeviceStage(sb)
    for v in ds.out.values():
        v.zero_()
    ds.prune(lam)
    eager = snapshot(ds)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ds.prune(lam)                       # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ds.prune(lam)
    for rep in range(3):
        for v in ds.out.values():
            v.fill_(-1)                     # eager work between replays
        for d in ds.row_dst:
            d.zero_()
        torch.cuda.synchronize()
        g.replay()
        assert_same(snapshot(ds), eager)


def test_captured_budget_matching_and_topk_replay():
    print("case: graph budget matching + top-K", flush=True)
    sb = custom_stage(B=3, R=4, H=4, Hkv=4, d=64, T=[1, 1, 1], N=[300, 0, 577], seed=31)
    ds = DeviceStage(sb, ragged=True)
    ds.prune(1.0)
    torch.cuda.synchronize()
    sc = ds.out["scores"]
    lam = torch.zeros(2, dtype=torch.float32, device="cuda")
    kept = torch.zeros_like(ds.out["kept_idx"])
    cnt = torch.zeros_like(ds.out["kept_count"])
    offs = torch.zeros_like(ds.out["kept_offsets"])

    def work():
        occam.match_lambda(ds.problem, sc, 50.0, lam[0:1], ds.ws, mean_kept=lam[1:2])
        occam.select_topk(ds.problem, sc, 64, kept, cnt, offs, ds.ws)

    work()
    torch.cuda.synchronize()
    want = (lam.clone(), kept.clone(), cnt.clone(), offs.clone())
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        work()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        work()
    for rep in range(3):
        for t in (lam, kept, cnt, offs):
            t.fill_(-3)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        total = int(want[3][-1])
        assert torch.equal(lam, want[0]) and torch.equal(cnt, want[2])
        assert torch.equal(offs, want[3])
        assert torch.equal(kept[:total], want[1][:total])
