"""MI355X (gfx950) register-anchored relative evidence test of OccamToken (arXiv 2605.29657).

The compute path is ``liboccam.so`` (hand-written HIP kernels behind the C ABI of
``include/occam.h``); :mod:`paper_2605_29657_amd.occam` is its thin Python binding.
Importing this package loads nothing; the binding loads the library on first use
and raises if it is missing.
"""
__all__ = ["occam", "synth", "workloads"]
