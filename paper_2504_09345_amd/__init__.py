"""MI355X (gfx950) paged-KV grouped-query attention: decode rows and causal
prefill chunks over a block-table-addressed KV page pool (the hot path of
MoE-Lens, arXiv 2504.09345), as hand-written HIP kernels behind a C ABI.

Importing the package loads nothing; ``paper_2504_09345_amd.binding`` loads
``libpagedattn.so`` on first use and raises if it is missing.
"""
__all__ = ["workloads", "binding"]
