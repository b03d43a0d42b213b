"""QuadTree attention forward (Tang et al., ICLR 2022) on AMD Instinct MI355X (gfx950).

The computation lives in hand-written HIP kernels behind the C ABI of ``include/qta.h``
(``libqta.so``, built by ``paper_2201_02767_amd.build``). ``paper_2201_02767_amd.qta`` is the thin
torch binding; ``paper_2201_02767_amd.inputs`` draws the seeded synthetic workloads.
"""
from .qta import (NOALLOC_WORKSPACE_BYTES, Options, Plan, QtaError, attention, build_pyramid, coarse_attn, fine_attn,
                  finest_attn, forward, forward_noalloc, k_levels, level_dims, lib, topk, workspace_bytes,
                  workspace_layout)

__all__ = ["NOALLOC_WORKSPACE_BYTES", "Options", "Plan", "QtaError", "attention", "build_pyramid", "coarse_attn",
           "fine_attn", "finest_attn", "forward", "forward_noalloc", "k_levels", "level_dims", "lib", "topk",
           "workspace_bytes", "workspace_layout"]
