"""GPU parity of the backward pass (gradients of q, k, v and w with the kept keys held fixed)
against the CPU oracle's backward, teacher-forced with the GPU forward's selections.

Error measure for dq, dk, dv: the forward's per-row measure (tests/parity.py ``rel_err``): for
every row (batch, token, head), max |gpu - oracle| over the d channels divided by max(max |oracle|
over the row, 1e-3 * RMS of the whole tensor). Every such gradient is computed in fp32 from inputs
that are exact in the storage type (bf16 inputs are bf16 values), with sums of at most a few thousand
terms (the coarse level's 1024 keys), so 1e-4 leaves an order of magnitude over fp32 accumulation;
the same bound holds for bf16 inputs because nothing is rounded to bf16 on the way.

dw is the exception: dw_{i,l} = <dout_i, m^l> is a dot product with the forward's stored message of
the query's level-l ancestor, and for bf16 inputs that message carries the forward's bf16 rounding of
the attention weights (the forward's messages are held to 2e-2 of max |m| per row). The dot product
can cancel to nearly zero, so a bound relative to |dw| itself does not follow from the message bar;
what follows is |dw_gpu - dw_ref| <= tol * sum_c |dout_ic| * max_c |m^l_c| (the message error summed
against dout). dw is checked element by element against that bound, tol being the forward's message
tolerance (1e-4 fp32, 2e-2 bf16), with the oracle's messages in the bound.
The tensor-wide measure max |gpu - oracle| / max |oracle| is printed beside both.
"""
import sys

import numpy as np
import pytest
import torch

import paper_2201_02767_amd as P
from paper_2201_02767_amd.inputs import (WORKLOADS, make_dout, make_level_weights, make_pe, make_qkv, make_v_levels,
                                         round_bf16)
from oracle import oracle as O
from tests.parity import TOL, rel_err, to_np

pytestmark = pytest.mark.gpu

TDT = {"f32": torch.float32, "bf16": torch.bfloat16}
TOL_GRAD = 1e-4


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    P.lib()
    return torch.device("cuda:0")


def announce(msg: str) -> None:
    print(f"[gpu case] {msg}", file=sys.stderr, flush=True)


def dev_t(x, dtype, dev):
    return torch.from_numpy(np.ascontiguousarray(x)).to(dev).to(TDT[dtype])


def rand(seed, shape, dtype):
    x = np.random.default_rng(seed).standard_normal(shape).astype(np.float32)
    return round_bf16(x) if dtype == "bf16" else x


def grad_err(g, r):
    return float(np.abs(g - r).max() / max(np.abs(r).max(), 1e-30))


def dw_err(g, r, dout, msgs):
    """max over (map, token, head, level) of |g - r| / (sum_c |dout_c| * max_c |m^l_c| of the token's
    level-l ancestor); g, r [B, H*W, heads, L], dout [B, H, W, heads, d], msgs[l] [B, N_l, heads, d]."""
    B, H, W, heads, d = dout.shape
    L = r.shape[-1]
    l1 = np.abs(np.asarray(dout, np.float64)).sum(-1).reshape(B, H * W, heads)
    yy, xx = np.divmod(np.arange(H * W), W)
    norm = np.empty(r.shape)
    for l in range(L):
        Wl = -(-W // (1 << l))
        anc = (yy >> l) * Wl + (xx >> l)
        norm[..., l] = l1 * np.abs(msgs[l]).max(-1)[:, anc, :]
    return float((np.abs(np.asarray(g, np.float64) - r) / np.maximum(norm, 1e-30)).max())


def run_backward(dev, q, k, v, g, *, levels, K, variant, dtype, w=None, scale=None, epipolar=False, label="",
                 v_levels=None, pe_weight=None, pe_bias=None):
    """GPU backward against the oracle's, teacher-forced. ``v_levels`` (numpy list, entry l >= 1, in the
    library's map layout: B*H one-row maps for epipolar attention), ``pe_weight``, ``pe_bias``: the
    forward's given V levels and position encoding, whose gradients are compared too."""
    B, H, W, heads, d = q.shape
    announce(f"backward {label} B={B} H={H} W={W} heads={heads} d={d} L={levels} K={K} {variant} {dtype}"
             f"{' epipolar' if epipolar else ''}{' V levels given' if v_levels is not None else ''}"
             f"{' position encoding' if pe_weight is not None else ''}")
    plan = P.Plan(B, H, W, heads, d, levels=levels, K=K, variant=variant, dtype=TDT[dtype], device=dev, scale=scale,
                  epipolar=epipolar, v_supplied=v_levels is not None, pe=pe_weight is not None)
    tq, tk, tv, tg = (dev_t(x, dtype, dev) for x in (q, k, v, g))
    tw = None if w is None else torch.from_numpy(w).to(dev)
    tvl = None if v_levels is None else [None] + [dev_t(v_levels[l], dtype, dev) for l in range(1, levels)]
    tpw = None if pe_weight is None else torch.from_numpy(np.ascontiguousarray(pe_weight)).to(dev)
    tpb = None if pe_bias is None else torch.from_numpy(np.ascontiguousarray(pe_bias)).to(dev)
    plan.run(tq, tk, tv, tw, v_levels=tvl, pe_weight=tpw, pe_bias=tpb)
    dq, dk, dv, dw = plan.backward(tq, tk, tv, tg, tw, v_levels=tvl, pe_weight=tpw, pe_bias=tpb)
    torch.cuda.synchronize()
    sel = [None] + [to_np(plan.selection(l)[0]) for l in range(1, levels)]
    if epipolar:
        q, k, v, g = (x.reshape(B * H, 1, W, heads, d) for x in (q, k, v, g))
        w = None if w is None else w.reshape(B * H, W, heads, levels)
    ref = O.backward(q, k, v, g, levels=levels, K=K, variant=variant, dtype=dtype, w=w, scale=scale, forced=sel,
                     v_levels=v_levels, pe_weight=pe_weight, pe_bias=pe_bias)
    errs, wide = {}, {}
    for name, t in (("dq", dq), ("dk", dk), ("dv", dv), ("dw", dw)):
        if ref[name] is None:
            assert t is None
            continue
        g_ = to_np(t).reshape(ref[name].shape)
        if name == "dw":
            fwd = O.forward(q, k, v, levels=levels, K=K, variant=variant, dtype=dtype, w=w, scale=scale, forced=sel,
                            v_levels=v_levels, pe_weight=pe_weight, pe_bias=pe_bias)
            errs[name] = dw_err(g_, ref[name], g, fwd["msg"])
        else:
            errs[name] = rel_err(g_, ref[name])
        wide[name] = grad_err(g_, ref[name])
    # the position encoding's kernels (rows of 9 taps) and bias (rows of one level's channels), and the
    # given V levels (rows of d channels), per row like dq, dk, dv
    if pe_weight is not None:
        L_, C_ = pe_weight.shape[:2]
        errs["dpe_weight"] = rel_err(to_np(plan.grad_extra["dpe_weight"]).reshape(L_, C_, 9),
                                     ref["dpe_weight"].reshape(L_, C_, 9))
        if pe_bias is not None:
            errs["dpe_bias"] = rel_err(to_np(plan.grad_extra["dpe_bias"]), ref["dpe_bias"])
    if v_levels is not None:
        errs["dv_levels"] = max(rel_err(to_np(plan.grad_extra["dv_levels"][l]).reshape(ref["dv_levels"][l].shape),
                                        ref["dv_levels"][l]) for l in range(1, levels))
    announce(f"  gradient errors per row (dw: per element against the message bound) {errs}, tensor-wide {wide}")
    for name, e in errs.items():
        assert e <= (TOL[dtype] if name == "dw" else TOL_GRAD), f"{name} error {e}"
    return plan, (dq, dk, dv, dw), errs


@pytest.mark.parametrize("variant,dtype,B,H,W,heads,d,L,K,with_w", [
    ("A", "f32", 1, 16, 16, 1, 32, 3, 4, False),        # the tiny workload's shape
    ("B", "f32", 1, 16, 16, 1, 32, 3, 4, True),
    ("B", "f32", 2, 13, 11, 2, 32, 3, 3, False),       # ragged maps, w = 1/L
    ("A", "bf16", 2, 25, 19, 2, 32, 4, 4, False),      # ragged over four levels
    ("B", "bf16", 1, 31, 22, 3, 64, 3, 8, True),       # d = 64, odd head count
    ("A", "f32", 1, 20, 24, 2, 64, 3, 16, False),      # 64 candidates per sibling group
    ("B", "bf16", 1, 9, 7, 1, 32, 2, 2, True),         # two levels: the finest parents are coarse
    ("A", "f32", 2, 7, 9, 2, 32, 1, 4, False),         # one level: dense attention
    ("B", "bf16", 1, 5, 40, 2, 32, 1, 4, True),
    ("B", "f32", 1, 40, 41, 1, 32, 2, 4, True),        # 420 coarse tokens: 7 key chunks per lane
    ("A", "bf16", 1, 50, 37, 1, 32, 6, 3, False),      # six levels (the unpooling's 8-level kernel)
    ("B", "f32", 1, 257, 200, 1, 32, 9, 2, True),      # nine levels, coarsest 2x1 (its 16-level kernel)
    ("A", "bf16", 1, 27, 33, 2, 32, 3, [0, 2, 16], False),   # K schedule, blocked level 1
    ("B", "f32", 1, 33, 29, 2, 32, 4, [0, 8, 4, 2], True),
])
def test_backward_matches_oracle(dev, variant, dtype, B, H, W, heads, d, L, K, with_w):
    seed = 300 + H * W + L
    q, k, v, g = (rand(seed + i, (B, H, W, heads, d), dtype) for i in range(4))
    w = np.random.default_rng(seed).random((B, H * W, heads, L)).astype(np.float32) if with_w else None
    run_backward(dev, q, k, v, g, levels=L, K=K, variant=variant, dtype=dtype, w=w, label="case")


@pytest.mark.parametrize("variant,dtype", [("A", "bf16"), ("B", "f32")])
def test_backward_epipolar(dev, variant, dtype):
    q, k, v, g = (rand(400 + i, (2, 5, 37, 2, 32), dtype) for i in range(4))
    w = np.random.default_rng(4).random((2, 5 * 37, 2, 4)).astype(np.float32) if variant == "B" else None
    run_backward(dev, q, k, v, g, levels=4, K=3, variant=variant, dtype=dtype, w=w, epipolar=True, label="rows")


@pytest.mark.parametrize("name", ["tiny", "matching", "matching_ksched", "stereo", "backbone", "highres",
                                  "stereo_epipolar"])
def test_backward_workload_full_size(dev, name):
    wl = WORKLOADS[name]
    q, k, v = make_qkv(wl)
    g = make_dout(wl)
    w = make_level_weights(wl) if wl.variant == "B" else None
    run_backward(dev, q, k, v, g, levels=wl.levels, K=wl.K, variant=wl.variant, dtype=wl.dtype, w=w,
                 epipolar=wl.epipolar, label=name)


@pytest.mark.parametrize("variant,dtype,B,H,W,heads,d,L,K,with_w,pe,vgiven", [
    ("B", "f32", 1, 13, 11, 2, 32, 3, 3, True, True, False),
    ("A", "bf16", 2, 25, 19, 2, 32, 4, 4, False, True, False),      # ragged, four levels, blocked levels
    ("B", "bf16", 1, 31, 22, 3, 64, 3, 8, True, False, True),       # d = 64, given V levels
    ("A", "f32", 1, 20, 24, 2, 32, 3, [0, 2, 16], False, True, True),
    ("B", "bf16", 1, 9, 7, 1, 32, 2, 2, True, True, True),          # two levels
    ("B", "f32", 2, 7, 9, 2, 32, 1, 4, True, True, False),          # one level
    ("B", "f32", 1, 20, 21, 1, 32, 3, 4, False, True, False),       # B with w = 1/L
])
def test_backward_position_encoding_and_given_v(dev, variant, dtype, B, H, W, heads, d, L, K, with_w, pe, vgiven):
    """Gradients of the multiscale position encoding's kernels and bias and of caller-supplied V levels,
    with q, k, v, w, against the oracle's backward."""
    seed = 500 + H * W + L
    q, k, v, g = (rand(seed + i, (B, H, W, heads, d), dtype) for i in range(4))
    rng = np.random.default_rng(seed)
    w = rng.random((B, H * W, heads, L)).astype(np.float32) if with_w else None
    dims = O.level_dims(H, W, L)
    vl = [None] + [rand(seed + 10 + l, (B, dims[l][0], dims[l][1], heads, d), dtype) for l in range(1, L)] \
        if vgiven else None
    pw = (rng.standard_normal((L, heads * d, 3, 3)) * 0.3).astype(np.float32) if pe else None
    pb = (rng.standard_normal((L, heads * d)) * 0.1).astype(np.float32) if pe else None
    run_backward(dev, q, k, v, g, levels=L, K=K, variant=variant, dtype=dtype, w=w, label="pe/vgiven", v_levels=vl,
                 pe_weight=pw, pe_bias=pb)


@pytest.mark.parametrize("variant", ["A", "B"])
def test_backward_position_encoding_epipolar(dev, variant):
    """Attention along rows with the encoding (every level's pass runs separately on one-row maps)."""
    q, k, v, g = (rand(600 + i, (2, 5, 37, 2, 32), "bf16") for i in range(4))
    rng = np.random.default_rng(6)
    w = rng.random((2, 5 * 37, 2, 4)).astype(np.float32) if variant == "B" else None
    pw = (rng.standard_normal((4, 64, 3, 3)) * 0.3).astype(np.float32)
    pb = (rng.standard_normal((4, 64)) * 0.1).astype(np.float32)
    run_backward(dev, q, k, v, g, levels=4, K=3, variant=variant, dtype="bf16", w=w, epipolar=True, label="rows pe",
                 pe_weight=pw, pe_bias=pb)


@pytest.mark.parametrize("name", ["backbone_pe", "backbone_vgiven"])
def test_backward_pe_and_vgiven_workloads_full_size(dev, name):
    wl = WORKLOADS[name]
    q, k, v = make_qkv(wl)
    g = make_dout(wl)
    w = make_level_weights(wl) if wl.variant == "B" else None
    vl = make_v_levels(wl) if wl.v_given else None
    pw, pb = make_pe(wl) if wl.pe else (None, None)
    run_backward(dev, q, k, v, g, levels=wl.levels, K=wl.K, variant=wl.variant, dtype=wl.dtype, w=w, label=name,
                 v_levels=vl, pe_weight=pw, pe_bias=pb)


def test_backward_repeated_calls(dev):
    """Repeated calls agree: dw has one writer per element (identical bits); dk, dv and the
    messages' gradients at levels >= 2 (hence dq too) are summed with atomics, so only the order of
    their additions may change."""
    wl = WORKLOADS["matching"]
    announce("backward repeated calls, matching")
    q, k, v = (dev_t(x, "f32", dev) for x in make_qkv(wl))
    g = dev_t(make_dout(wl), "f32", dev)
    w = torch.from_numpy(make_level_weights(wl)).to(dev)
    plan = P.Plan(wl.B, wl.H, wl.W, wl.heads, wl.d, levels=wl.levels, K=wl.K, variant="B", dtype=torch.float32,
                  device=dev)
    plan.run(q, k, v, w)
    first = [t.clone() for t in plan.backward(q, k, v, g, w)]
    for _ in range(2):
        again = plan.backward(q, k, v, g, w)
        torch.cuda.synchronize()
        assert torch.equal(again[3], first[3])
        for a, b in zip(again[:3], first[:3]):
            assert grad_err(to_np(a), to_np(b)) <= 1e-6


@pytest.mark.parametrize("variant,dtype,name", [("B", "f32", "matching"), ("A", "bf16", "backbone"),
                                                ("B", "bf16", "backbone"), ("A", "bf16", "highres"),
                                                ("B", "bf16", "stereo_epipolar")])
def test_backward_overlap_matches_one_stream(dev, variant, dtype, name):
    """The three-stream schedule (the finest level's sort and key pass on a second stream, the
    coarser levels' on a third; with QuadTree-B, one intermediate level and a coarse level that fills
    the chip, as for backbone, that level's query pass on the third stream too) gives the one-stream
    gradients, up to the order of the atomic sums."""
    wl = WORKLOADS[name].with_(variant=variant, dtype=dtype)
    announce(f"backward overlap vs one stream, {name} {variant} {dtype}")
    q, k, v = (dev_t(x, dtype, dev) for x in make_qkv(wl))
    g = dev_t(make_dout(wl), dtype, dev)
    w = torch.from_numpy(make_level_weights(wl)).to(dev) if variant == "B" else None
    plan = P.Plan(wl.B, wl.H, wl.W, wl.heads, wl.d, levels=wl.levels, K=wl.K, variant=variant, dtype=TDT[dtype],
                  device=dev, epipolar=wl.epipolar)
    plan.run(q, k, v, w)
    one = [None if t is None else t.clone() for t in plan.backward(q, k, v, g, w, overlap=False)]
    two = plan.backward(q, k, v, g, w, overlap=True)
    torch.cuda.synchronize()
    for a, b in zip(one, two):
        if a is None:
            assert b is None
            continue
        assert grad_err(to_np(b), to_np(a)) <= 1e-6


def test_autograd_function(dev):
    """attention() under autograd gives the gradients of the plan's backward, in q's dtype. dw has
    one writer per element (identical bits); dq, dk and dv take sums made with atomics (the
    message gradients at levels >= 2, the key lists' order), so they are compared to the bf16
    rounding of the plan's gradients."""
    announce("autograd function, 2 x 24 x 20, bf16, B")
    B, H, W, heads, d, L = 2, 24, 20, 2, 32, 3
    q, k, v = (dev_t(rand(500 + i, (B, H, W, heads, d), "bf16"), "bf16", dev).requires_grad_() for i in range(3))
    w = torch.rand((B, H * W, heads, L), device=dev).requires_grad_()
    out = P.attention(q, k, v, levels=L, K=4, variant="B", w=w)
    g = dev_t(rand(504, (B, H, W, heads, d), "bf16"), "bf16", dev)
    (out.float() * g.float()).sum().backward()
    plan = P.Plan(B, H, W, heads, d, levels=L, K=4, variant="B", dtype=torch.bfloat16, device=dev)
    plan.run(q.detach(), k.detach(), v.detach(), w.detach())
    dq, dk, dv, dw = plan.backward(q.detach(), k.detach(), v.detach(), g, w.detach())
    torch.cuda.synchronize()
    assert q.grad.dtype == torch.bfloat16 and w.grad.dtype == torch.float32
    assert grad_err(to_np(q.grad.float()), to_np(dq)) <= 1e-2
    assert grad_err(to_np(k.grad.float()), to_np(dk)) <= 1e-2
    assert grad_err(to_np(v.grad.float()), to_np(dv)) <= 1e-2
    assert torch.equal(w.grad, dw)
