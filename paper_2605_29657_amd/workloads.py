"""Workload shapes of the pruning path (data only, no arithmetic).

Five synthetic workloads stand in for the visual sequences the paper prunes
(LLaVA-1.5's 576 tokens, LLaVA-NeXT's 2880, Qwen3-VL's ragged merged patches and
multi-frame video; Sec. 4 and Appendix "Architecture-specific
instantiations").  Each has a vision stage (one CLS anchor row, Stage I) and,
except the first, a text stage (text anchor rows inside the LLM, Stage II).

Field meanings:
  B            samples in the batch
  R            register keys per sample (laid out first)
  N            visual candidates per sample (int, or (lo, hi, step) for ragged)
  vis / txt    dict(H=query heads, Hkv=key heads, d=head dim, T=anchor rows
               (int or (lo, hi) ragged), hidden=row width of the payload
               gathered with the survivors)
  dtype        "f32" or "bf16" for every tensor of the workload
  sinks        planted sink keys per sample (int or (lo, hi)) and their norm
               factor ``sink_scale``
  informative  keys aligned with the CLS query (cos 0.6), counted per 576
               visual tokens (scaled with N)
  relevant     (lo, hi) keys per sample aligned with one text row (cos 0.6)
  dup          near-duplicate structure: None, ("clusters", frac, lo, hi, cos) or
               ("temporal", frame_len, frac, cos)
  keep1/keep2  calibration targets for the mean kept count of each stage:
               an absolute count, or a fraction of N when below 1
"""

WORKLOADS = {
    # LLaVA-1.5 vision tower, CLS stage only, single image, fp32.
    "llava15_cls_f32": dict(
        id=0, B=1, R=4, N=576, dtype="f32",
        vis=dict(H=16, Hkv=16, d=64, T=1, hidden=1024),
        txt=None,
        sinks=3, sink_scale=8.0, informative=20, relevant=None, dup=None,
        keep1=250, keep2=None),
    # LLaVA-1.5 shaped, both stages, bf16.
    "llava15": dict(
        id=1, B=64, R=4, N=576, dtype="bf16",
        vis=dict(H=16, Hkv=16, d=64, T=1, hidden=1024),
        txt=dict(H=32, Hkv=32, d=128, T=64, hidden=4096),
        sinks=3, sink_scale=8.0, informative=20, relevant=(5, 40), dup=None,
        keep1=250, keep2=64),
    # LLaVA-NeXT shaped: 5 tiles x 576 = 2880 visual tokens, 30 % near-duplicates.
    "llava_next": dict(
        id=2, B=32, R=4, N=2880, dtype="bf16",
        vis=dict(H=16, Hkv=16, d=64, T=1, hidden=1024),
        txt=dict(H=32, Hkv=32, d=128, T=128, hidden=4096),
        sinks=3, sink_scale=8.0, informative=20, relevant=(5, 40),
        dup=("clusters", 0.30, 4, 16, 0.99),
        keep1=523, keep2=40),
    # Qwen3-VL shaped ragged batch: N in [256, 4096] step 4, T in [16, 512], d_vis = 72.
    "qwen3vl_ragged": dict(
        id=3, B=64, R=4, N=(256, 4096, 4), dtype="bf16",
        vis=dict(H=16, Hkv=16, d=72, T=1, hidden=1152),
        txt=dict(H=32, Hkv=32, d=128, T=(16, 512), hidden=4096),
        sinks=(0, 6), sink_scale=8.0, informative=20, relevant=(5, 40), dup=None,
        keep1=0.18, keep2=0.111),
    # Multi-frame video: 8 frames x 2048 tokens, 50 % temporal near-duplicates.
    "video": dict(
        id=4, B=8, R=8, N=16384, dtype="bf16",
        vis=dict(H=16, Hkv=16, d=64, T=1, hidden=1024),
        txt=dict(H=32, Hkv=32, d=128, T=256, hidden=4096),
        sinks=3, sink_scale=10.0, informative=20, relevant=(5, 40),
        dup=("temporal", 2048, 0.50, 0.98),
        keep1=0.18, keep2=0.02),
}

# The workload the throughput figure is quoted on: LLaVA-NeXT's 2880 visual tokens.
HEADLINE = "llava_next"


def by_id(i: int) -> str:
    for name, w in WORKLOADS.items():
        if w["id"] == i:
            return name
    raise KeyError(i)
