"""One GPU's share of a GPT pipeline stage (forward, recompute, backward) on MI355X.

The compute lives in the HIP library ``libmerak_stage.so`` behind the C ABI of
``include/merak_stage.h``; ``paper_2206_04959_amd.binding`` marshals arguments
to it.  Importing the package loads nothing: ``synth`` (seeded workloads) and
``flops`` (algorithmic work counts) are plain Python.
"""
__all__ = ["synth", "flops", "binding"]
