"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws random numbers and arranges them: it holds none of the method's arithmetic
(no pooling, no attention, no selection). Both the GPU tests/benchmark and the CPU oracle take their
inputs from here.

Workloads (stand-ins for the feature maps of the paper's experiments; the datasets themselves are
not used):
  tiny     - 16x16 self-attention, 1 head x 32, fp32, 3 levels, K=4, QuadTree-A.
  matching - 60x80 (640x480 image at 1/8, coarsest 15x20 as in the feature-matching setting),
             8 heads x 32, fp32, 3 levels, K=8, QuadTree-B; keys are the queries shifted by one
             random offset of at most 8 tokens plus N(0, 0.3^2) noise.
  stereo   - 2 x 120x160, 8 heads x 32, bf16, 4 levels, K=8, QuadTree-B; keys are the queries
             shifted along x by a per-pixel disparity in [0, 24] plus N(0, 0.2^2) noise.
  backbone - 32 x 56x56 (224^2 image, stage 1), 1 head x 64, bf16, 3 levels, K=8, QuadTree-B;
             q, k, v are random linear maps of Gaussian-blurred (sigma 2 tokens) N(0,1) features.
  highres  - 2 x 200x336 (800x1333 image at 1/4), 2 heads x 32, bf16, 5 levels, K=16, QuadTree-B;
             generated like backbone. Its coarsest level (13x21) comes from ceil pooling.
  detection - 2 x 200x334 (an 800x1333 detection input at stride 4: the first stage of a PVTv2-b0
             backbone), 1 head x 32, bf16, 5 levels (coarsest 13x21), K=32 as the paper's detection
             backbones use (Sec. 4.2, Table 4), QuadTree-B; generated like backbone. With 4K = 128
             candidates per sibling group it takes the wide fine-level path.
  matching_ksched - matching with the paper's K schedule for feature matching (Sec. 4.1.1): K = 8
             at the finest selecting level, doubled at each coarser level (16 at the coarsest).
  backbone_vgiven - backbone with V's coarser levels given as inputs, as in self-attention where a
             stride-2 conv-norm-act layer builds them (Sec. 3.2); each level is an independent
             N(0,1) map standing in for that layer's normalised output.
  backbone_pe - backbone with the multiscale position encoding (Sec. 3.2): 3x3 depth-wise kernels
             N(0, 0.3^2) and biases N(0, 0.1^2) per level and channel (random-init weights).
  stereo_epipolar - stereo with attention along the epipolar lines only (Sec. 4.1.2): each of the
             2 x 120 rows of 160 tokens is its own binary tree of 4 levels.

Seeds: numpy PCG64 with seed = 1000 * config_number + tensor id (q=1, k=2, v=3, w=4, aux=5,
10 + l for the given V level l, 20 and 21 for the position-encoding weights and biases, 30 for the
upstream gradient of the backward pass).
All arrays are float32 ``[B, H, W, heads, d]``; for bf16 workloads the values are rounded to the
nearest bfloat16 (ties to even), so they are exactly representable in bf16.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    number: int       # config number, used in the seeds
    B: int
    H: int
    W: int
    heads: int
    d: int
    levels: int
    K: object         # one count for every level, or a tuple with one entry per level (entry 0 unused)
    variant: str      # "A" or "B"
    dtype: str        # "f32" or "bf16"
    kind: str         # generator: "iid_scaled", "shift", "disparity", "smooth"
    v_given: bool = False   # V's coarser levels are inputs (make_v_levels) instead of pooled
    pe: bool = False        # multiscale position encoding (make_pe)
    epipolar: bool = False  # attention along rows only

    @property
    def tokens(self) -> int:
        return self.B * self.H * self.W

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS = {
    "tiny": Workload("tiny", 1, 1, 16, 16, 1, 32, 3, 4, "A", "f32", "iid_scaled"),
    "matching": Workload("matching", 2, 1, 60, 80, 8, 32, 3, 8, "B", "f32", "shift"),
    "stereo": Workload("stereo", 3, 2, 120, 160, 8, 32, 4, 8, "B", "bf16", "disparity"),
    "backbone": Workload("backbone", 4, 32, 56, 56, 1, 64, 3, 8, "B", "bf16", "smooth"),
    "highres": Workload("highres", 5, 2, 200, 336, 2, 32, 5, 16, "B", "bf16", "smooth"),
    "detection": Workload("detection", 6, 2, 200, 334, 1, 32, 5, 32, "B", "bf16", "smooth"),
    "matching_ksched": Workload("matching_ksched", 2, 1, 60, 80, 8, 32, 3, (0, 8, 16), "B", "f32", "shift"),
    "backbone_vgiven": Workload("backbone_vgiven", 4, 32, 56, 56, 1, 64, 3, 8, "B", "bf16", "smooth", True),
    "backbone_pe": Workload("backbone_pe", 4, 32, 56, 56, 1, 64, 3, 8, "B", "bf16", "smooth", False, True),
    "stereo_epipolar": Workload("stereo_epipolar", 3, 2, 120, 160, 8, 32, 4, 8, "B", "bf16", "disparity",
                                epipolar=True),
}


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 value (ties to even) of each float32 element, returned as float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def _rng(wl: Workload, tensor_id: int, seed_offset: int = 0) -> np.random.Generator:
    return np.random.default_rng(1000 * wl.number + tensor_id + 100000 * seed_offset)


def _gaussian_blur(x: np.ndarray, sigma: float = 2.0, radius: int = 6) -> np.ndarray:
    """Separable Gaussian blur over the two spatial axes of [B, H, W, C], reflect border."""
    t = np.arange(-radius, radius + 1, dtype=np.float64)
    g = np.exp(-0.5 * (t / sigma) ** 2)
    g = (g / g.sum()).astype(np.float32)
    B, H, W, C = x.shape
    pad = np.pad(x, ((0, 0), (radius, radius), (0, 0), (0, 0)), mode="reflect")
    y = np.zeros_like(x)
    for i, gi in enumerate(g):
        y += gi * pad[:, i:i + H]
    pad = np.pad(y, ((0, 0), (0, 0), (radius, radius), (0, 0)), mode="reflect")
    z = np.zeros_like(x)
    for i, gi in enumerate(g):
        z += gi * pad[:, :, i:i + W]
    return z


def make_qkv(wl: Workload, seed_offset: int = 0):
    """Return (q, k, v) float32 [B, H, W, heads, d] for a workload."""
    B, H, W, C = wl.B, wl.H, wl.W, wl.heads * wl.d
    shape = (B, H, W, C)
    if wl.kind == "iid_scaled":
        s = np.float32(1.0 / np.sqrt(wl.d))
        q = _rng(wl, 1, seed_offset).standard_normal(shape, dtype=np.float32) * s
        k = _rng(wl, 2, seed_offset).standard_normal(shape, dtype=np.float32) * s
        v = _rng(wl, 3, seed_offset).standard_normal(shape, dtype=np.float32) * s
    elif wl.kind == "shift":
        q = _rng(wl, 1, seed_offset).standard_normal(shape, dtype=np.float32)
        aux = _rng(wl, 5, seed_offset)
        k = np.empty_like(q)
        for b in range(B):
            dy, dx = aux.integers(-8, 9, size=2)
            k[b] = np.roll(q[b], shift=(-int(dy), -int(dx)), axis=(0, 1))
        k += 0.3 * _rng(wl, 2, seed_offset).standard_normal(shape, dtype=np.float32)
        v = _rng(wl, 3, seed_offset).standard_normal(shape, dtype=np.float32)
    elif wl.kind == "disparity":
        q = _rng(wl, 1, seed_offset).standard_normal(shape, dtype=np.float32)
        disp = _rng(wl, 5, seed_offset).integers(0, 25, size=(B, H, W))
        xs = np.minimum(np.arange(W)[None, None, :] + disp, W - 1)
        bs = np.arange(B)[:, None, None]
        ys = np.arange(H)[None, :, None]
        k = q[bs, ys, xs] + 0.2 * _rng(wl, 2, seed_offset).standard_normal(shape, dtype=np.float32)
        v = _rng(wl, 3, seed_offset).standard_normal(shape, dtype=np.float32)
    elif wl.kind == "smooth":
        feat_c = 64
        x = _rng(wl, 5, seed_offset).standard_normal((B, H, W, feat_c), dtype=np.float32)
        x = _gaussian_blur(x)
        x = (x - x.mean(axis=(0, 1, 2))) / x.std(axis=(0, 1, 2))
        outs = []
        for tid in (1, 2, 3):
            m = _rng(wl, tid, seed_offset).standard_normal((feat_c, C), dtype=np.float32) / np.float32(8.0)
            outs.append((x.reshape(-1, feat_c) @ m).reshape(shape))
        q, k, v = outs
    else:
        raise ValueError(wl.kind)
    res = []
    for t in (q, k, v):
        t = np.ascontiguousarray(t, dtype=np.float32)
        if wl.dtype == "bf16":
            t = round_bf16(t)
        res.append(t.reshape(B, H, W, wl.heads, wl.d))
    return tuple(res)


def make_level_weights(wl: Workload, seed_offset: int = 0) -> np.ndarray:
    """QuadTree-B level weights [B, H*W, heads, L]: a softmax over levels of N(0,1) logits."""
    g = _rng(wl, 4, seed_offset).standard_normal((wl.B, wl.H * wl.W, wl.heads, wl.levels))
    e = np.exp(g - g.max(axis=-1, keepdims=True))
    return (e / e.sum(axis=-1, keepdims=True)).astype(np.float32)


def make_v_levels(wl: Workload, seed_offset: int = 0) -> list:
    """Given V levels for a workload with ``v_given``: entry l (1 <= l < levels) is float32
    ``[B, H_l, W_l, heads, d]`` with H_l, W_l by ceil halving; entry 0 is None (level 0 is v)."""
    out = [None]
    H, W = wl.H, wl.W
    for l in range(1, wl.levels):
        H, W = (H + 1) // 2, (W + 1) // 2
        x = _rng(wl, 10 + l, seed_offset).standard_normal((wl.B, H, W, wl.heads, wl.d), dtype=np.float32)
        out.append(round_bf16(x) if wl.dtype == "bf16" else x)
    return out


def make_pe(wl: Workload, seed_offset: int = 0):
    """Position-encoding weights fp32 [levels, heads*d, 3, 3] and biases fp32 [levels, heads*d]."""
    C = wl.heads * wl.d
    wgt = (_rng(wl, 20, seed_offset).standard_normal((wl.levels, C, 3, 3)) * 0.3).astype(np.float32)
    bias = (_rng(wl, 21, seed_offset).standard_normal((wl.levels, C)) * 0.1).astype(np.float32)
    return wgt, bias


def make_dout(wl: Workload, seed_offset: int = 0) -> np.ndarray:
    """Upstream gradient of the layer output for the backward pass: N(0,1) float32
    ``[B, H, W, heads, d]`` (rounded to bf16 for bf16 workloads)."""
    g = _rng(wl, 30, seed_offset).standard_normal((wl.B, wl.H, wl.W, wl.heads, wl.d), dtype=np.float32)
    return round_bf16(g) if wl.dtype == "bf16" else g
