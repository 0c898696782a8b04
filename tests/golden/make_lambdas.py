"""Write tests/golden/lambdas.json: per workload and stage, the coefficient lambda whose
mean kept count on a calibration split matches the stage's target budget.

This is the paper's budget-matching protocol (Appendix, Eq.
lambda2_budget_matching_appendix; 50-100 calibration samples, "Parameter settings")
run on the fp64 oracle over the synthetic calibration split (split 1), so the
stored values come from the oracle alone.  Targets (workloads.py keep1/keep2):
Stage I keeps about 200-300 of 576 tokens on LLaVA-1.5 and 523 of 2880 on
LLaVA-NeXT (Appendix, "Parameter settings"; Table tab:lamda1cc); Stage II matches
64 tokens (LLaVA-1.5) and 40 tokens (LLaVA-NeXT, the 1.4 % budget of Table
tab:llavanext).  The mutual-scoring Stage I (Eq. mutual_scoring) takes the Stage I
targets.  Usage: python tests/golden/make_lambdas.py
"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from paper_2605_29657_amd import synth  # noqa: E402
from paper_2605_29657_amd.workloads import WORKLOADS  # noqa: E402

# Calibration samples per workload (fewer where one sample is large).
CALIB = {"llava15_cls_f32": 64, "llava15": 64, "llava_next": 64, "qwen3vl_ragged": 16, "video": 4}
# The mutual-scoring Stage I (every token an anchor row: (R+N)^2 work per sample).
CALIB_MUT = {"llava15": 64, "llava_next": 8, "qwen3vl_ragged": 16}


def calibrate(name, stage):
    n = CALIB_MUT[name] if stage == "mut" else CALIB[name]
    sb = synth.make_stage(name, stage, split=1, B=n, payload=False)
    rr = oracle.ROWS_MEAN if stage == "mut" else oracle.ROWS_MAX
    sc = oracle.scores(sb.q, sb.k, sb.q_off, sb.k_off, sb.H, sb.Hkv, sb.d, sb.R, dtype=sb.dtype,
                       row_reduce=rr)
    rat = oracle.ratios(sc, sb.k_off, sb.R)
    target = synth.keep_target(name, "vis" if stage == "mut" else stage, float(np.mean(sb.N)))
    lam = oracle.match_lambda(rat, target)
    lam32 = float(np.float32(lam))
    mean_kept = float(np.mean([np.sum(r >= lam32) for r in rat]))
    return dict(lam=lam32, target=target, mean_kept=mean_kept, samples=n)


def main():
    """Compute every missing entry (``--all`` recomputes the stored ones too)."""
    path = os.path.join(HERE, "lambdas.json")
    out = {}
    if os.path.exists(path) and "--all" not in sys.argv:
        with open(path) as f:
            out = json.load(f)
    for name, w in WORKLOADS.items():
        out.setdefault(name, {})
        stages = [st for st in ("vis", "txt") if w[st] is not None]
        if name in CALIB_MUT:
            stages.append("mut")
        for stage in stages:
            if stage in out[name]:
                continue
            t0 = time.time()
            out[name][stage] = calibrate(name, stage)
            print(name, stage, out[name][stage], "%.1fs" % (time.time() - t0), flush=True)
    with open(path, "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)


if __name__ == "__main__":
    main()
