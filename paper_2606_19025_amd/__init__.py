"""Resident-expert MoE layer for MI355X (gfx950).

One worker's local training step through an MoE layer in which the worker holds
only its resident subset of experts: top-k routing, skip-token masking of
routes to non-resident ("ghost") experts, dispatch grouped by resident expert,
the per-expert SwiGLU FFN as a grouped bf16 MFMA GEMM, the weighted combine,
the backward of all of these, and the expert-wise pseudo-gradient delta of the
round boundary.  The arithmetic lives in hand-written HIP kernels behind the
C ABI declared in include/moe_resident.h; ``paper_2606_19025_amd.binding`` is
a thin ctypes layer over it.  Importing this package does not load the native
library.
"""
__all__ = ["binding", "layer", "inputs"]
