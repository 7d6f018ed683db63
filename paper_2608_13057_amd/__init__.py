"""MI355X (gfx950) implementation of one GPU's share of TEMPO's expert-parallel
MoE block: stage-1 dispatch (counts, plan split, M-tile padded permute),
stage-2 grouped expert FFN (bf16 / fp8 e4m3 MFMA), stage-3 combine, and the
stage-4 profiling harness and max-affine cost fit.

The compute path is the HIP library ``libtempo_moe.so`` (C ABI in
``include/tempo_moe.h``); :mod:`paper_2608_13057_amd.moe` is its Python
binding, :mod:`paper_2608_13057_amd.synth` the seeded workload generator,
:mod:`paper_2608_13057_amd.fit` the cost-model fit.
"""
__all__ = ["moe", "synth", "fit", "build"]
