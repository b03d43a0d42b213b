"""Pins of the oracle's backward pass (gradients of the layer with the kept-key sets held fixed).

The backward is pinned by things other than itself:
  * finite differences of the oracle's forward (which the forward pins tie to the paper), along
    single elements and along random directions over whole tensors; the kept keys are forced to the
    unperturbed run's, so the forward is a smooth function of q, k, v and w;
  * automatic differentiation (torch, float64) of independent formulations where the layer has a
    closed form: Eq. (1) for a single level, and QuadTree-B with every key kept, which is dense
    attention at every pooled level combined with w;
  * invariants: shifting every key by one vector leaves every softmax unchanged, so the key
    gradients of one head sum to zero; the value gradients sum to the weighted upstream gradient,
    because every attention row sums to one (for A, because the regions Omega partition the map).
Inputs are dyadic (multiples of 1/64) and the step 2^-12, so perturbed values and the pooled
pyramids are exact in fp32 and the central differences carry only their O(eps^2) error.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O


def dyadic(rng, shape, lo=-64, hi=65):
    return (rng.integers(lo, hi, size=shape) / 64.0).astype(np.float32)


EPS = 2.0 ** -12


def _loss_fn(levels, K, variant, scale, forced, dout):
    def f(q, k, v, w):
        r = O.forward(q, k, v, levels=levels, K=K, variant=variant, w=w, scale=scale, forced=forced)
        return float((r["out"] * dout).sum())
    return f


CASES = [
    # variant, B, H, W, heads, d, L, K, with_w, scale
    ("A", 1, 6, 7, 2, 4, 3, 2, False, None),
    ("B", 1, 6, 7, 2, 4, 3, 2, True, None),
    ("B", 2, 5, 5, 1, 4, 3, 3, False, 0.7),
    ("A", 1, 9, 8, 1, 4, 4, [0, 2, 3, 2], False, None),
    ("B", 1, 9, 8, 1, 4, 4, [0, 3, 1, 4], True, None),
    ("A", 1, 4, 5, 2, 4, 1, 3, False, None),          # one level: dense attention
    ("B", 1, 4, 5, 2, 4, 1, 3, True, None),
    ("A", 3, 1, 13, 1, 4, 3, 2, False, None),         # one-row maps (binary tree)
    ("B", 2, 1, 11, 2, 4, 4, 2, True, None),
    ("A", 1, 8, 8, 1, 4, 3, 16, False, None),         # every key kept
]


@pytest.mark.parametrize("variant,B,H,W,heads,d,L,K,with_w,scale", CASES)
def test_backward_matches_finite_differences(variant, B, H, W, heads, d, L, K, with_w, scale):
    rng = np.random.default_rng(B * 100 + H * 10 + W + L)
    q, k, v, g = (dyadic(rng, (B, H, W, heads, d)) for _ in range(4))
    w = (rng.integers(1, 64, size=(B, H * W, heads, L)) / 64.0).astype(np.float32) if with_w else None
    forced = O.forward(q, k, v, levels=L, K=K, variant=variant, w=w, scale=scale)["sel_idx"]
    grads = O.backward(q, k, v, g, levels=L, K=K, variant=variant, w=w, scale=scale, forced=forced)
    loss = _loss_fn(L, K, variant, scale, forced, g)
    tensors = {"q": q, "k": k, "v": v}
    if with_w:
        tensors["w"] = w
    for name, arr in tensors.items():
        grad = grads["d" + name]
        scale_g = max(np.abs(grad).max(), 1e-3)

        def at(delta):
            args = dict(q=q, k=k, v=v, w=w)
            args[name] = (arr + delta).astype(np.float32)
            return loss(args["q"], args["k"], args["v"], args["w"])

        # single elements
        for _ in range(6):
            idx = tuple(int(rng.integers(0, s)) for s in arr.shape)
            e = np.zeros_like(arr)
            e[idx] = EPS
            fd = (at(e) - at(-e)) / (2 * EPS)
            assert abs(fd - grad[idx]) <= 1e-7 * scale_g + 1e-9, (name, idx, fd, grad[idx])
        # random directions over the whole tensor
        for _ in range(2):
            u = rng.integers(-1, 2, size=arr.shape).astype(np.float32)
            fd = (at(EPS * u) - at(-EPS * u)) / (2 * EPS)
            exact = float((grad * u).sum())
            assert abs(fd - exact) <= 1e-6 * max(1.0, abs(exact)), (name, fd, exact)


def _torch_pool(x):
    """[B,H,W,C] -> mean of the valid 2x2 children (ceil), written with padding and counts."""
    B, H, W, C = x.shape
    Hp, Wp = H + H % 2, W + W % 2
    xs = torch.zeros((B, Hp, Wp, C), dtype=x.dtype)
    xs[:, :H, :W] = x
    cnt = torch.zeros((Hp, Wp), dtype=x.dtype)
    cnt[:H, :W] = 1
    s = xs.reshape(B, Hp // 2, 2, Wp // 2, 2, C).sum(dim=(2, 4))
    n = cnt.reshape(Hp // 2, 2, Wp // 2, 2).sum(dim=(1, 3))
    return s / n[None, :, :, None]


def _torch_dense(q, k, v, tau):
    """q, k, v [B, N, heads, d] -> Eq. (1) per head."""
    logits = torch.einsum("bihc,bjhc->bhij", q, k) * tau
    p = torch.softmax(logits, dim=-1)
    return torch.einsum("bhij,bjhc->bihc", p, v)


def _autograd(fn, q, k, v, w, g):
    ts = [torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (q, k, v)]
    tw = torch.tensor(w, dtype=torch.float64, requires_grad=True) if w is not None else None
    out = fn(*ts, tw)
    (out * torch.tensor(g, dtype=torch.float64)).sum().backward()
    return [t.grad.numpy() for t in ts], (tw.grad.numpy() if tw is not None else None)


@pytest.mark.parametrize("variant", ["A", "B"])
def test_backward_single_level_is_dense_attention_gradient(variant):
    """One level: both variants are Eq. (1) (times w_0 for B), differentiated by autograd."""
    rng = np.random.default_rng(5)
    B, H, W, NH, d = 2, 5, 6, 2, 8
    q, k, v, g = (rng.standard_normal((B, H, W, NH, d)).astype(np.float32) for _ in range(4))
    w = rng.random((B, H * W, NH, 1)).astype(np.float32) if variant == "B" else None
    tau = 1 / np.sqrt(d)

    def fn(tq, tk, tv, tw):
        o = _torch_dense(tq.reshape(B, H * W, NH, d), tk.reshape(B, H * W, NH, d), tv.reshape(B, H * W, NH, d), tau)
        if tw is not None:
            o = o * tw[..., 0:1]
        return o.reshape(B, H, W, NH, d)

    (eq, ek, ev), ew = _autograd(fn, q, k, v, w, g)
    r = O.backward(q, k, v, g, levels=1, K=4, variant=variant, w=w)
    for name, e in (("dq", eq), ("dk", ek), ("dv", ev)):
        np.testing.assert_allclose(r[name], e, atol=1e-12, rtol=0)
    if w is not None:
        np.testing.assert_allclose(r["dw"], ew, atol=1e-12, rtol=0)


@pytest.mark.parametrize("H,W,L", [(8, 8, 3), (7, 10, 3), (1, 16, 4)])
def test_backward_b_with_every_key_kept_is_pooled_dense_gradient(H, W, L):
    """QuadTree-B keeping every key: out = sum_l w_l * (dense attention of the pooled level l,
    broadcast to the finest tokens), Eqs. (5)-(6); gradients by autograd through the pooling."""
    rng = np.random.default_rng(6)
    B, NH, d = 1, 2, 4
    q, k, v, g = (dyadic(rng, (B, H, W, NH, d)) for _ in range(4))
    w = rng.random((B, H * W, NH, L)).astype(np.float32)
    tau = 0.5

    def fn(tq, tk, tv, tw):
        C = NH * d
        xq, xk, xv = (t.reshape(B, H, W, C) for t in (tq, tk, tv))
        out = torch.zeros((B, H, W, NH, d), dtype=torch.float64)
        ys = torch.arange(H)
        xs = torch.arange(W)
        for l in range(L):
            Hl, Wl = xq.shape[1], xq.shape[2]
            m = _torch_dense(xq.reshape(B, Hl * Wl, NH, d), xk.reshape(B, Hl * Wl, NH, d),
                             xv.reshape(B, Hl * Wl, NH, d), tau).reshape(B, Hl, Wl, NH, d)
            anc = m[:, (ys >> l)][:, :, (xs >> l)]
            out = out + tw[..., l].reshape(B, H, W, NH, 1) * anc
            xq, xk, xv = _torch_pool(xq), _torch_pool(xk), _torch_pool(xv)
        return out

    (eq, ek, ev), ew = _autograd(fn, q, k, v, w, g)
    r = O.backward(q, k, v, g, levels=L, K=64, variant="B", w=w, scale=tau)
    for name, e in (("dq", eq), ("dk", ek), ("dv", ev), ("dw", ew)):
        np.testing.assert_allclose(r[name], e, atol=1e-12, rtol=0)


@pytest.mark.parametrize("variant", ["A", "B"])
@pytest.mark.parametrize("H,W,L,K", [(9, 7, 3, 2), (16, 16, 4, 3), (1, 20, 4, 2)])
def test_backward_invariants(variant, H, W, L, K):
    """Per head: sum_j dk_j = 0 (a common shift of the keys leaves every softmax unchanged), and
    sum_j dv_j = sum_i sum_l w_il dout_i (B; w = 1/L when not given) or sum_i dout_i (A: the
    Omega regions of a query partition the map and their weights sum to one)."""
    rng = np.random.default_rng(7)
    B, NH, d = 2, 2, 4
    q, k, v, g = (rng.standard_normal((B, H, W, NH, d)).astype(np.float32) for _ in range(4))
    w = rng.random((B, H * W, NH, L)).astype(np.float32) if variant == "B" else None
    r = O.backward(q, k, v, g, levels=L, K=K, variant=variant, w=w)
    sk = r["dk"].sum(axis=(1, 2))
    assert np.abs(sk).max() <= 1e-12 * max(1.0, np.abs(r["dk"]).max() * H * W)
    sv = r["dv"].sum(axis=(1, 2))
    if variant == "B":
        wsum = w.astype(np.float64).sum(axis=-1).reshape(B, H, W, NH, 1)
        expect = (g.astype(np.float64) * wsum).sum(axis=(1, 2))
    else:
        expect = g.astype(np.float64).sum(axis=(1, 2))
    np.testing.assert_allclose(sv, expect, atol=1e-11, rtol=0)


def test_backward_forced_selection_is_the_oracle_choice():
    """Forcing the oracle's own kept keys gives the same gradients as leaving the choice to it."""
    rng = np.random.default_rng(8)
    q, k, v, g = (rng.standard_normal((1, 9, 9, 2, 4)).astype(np.float32) for _ in range(4))
    for variant in "AB":
        f = O.forward(q, k, v, levels=3, K=3, variant=variant)["sel_idx"]
        a = O.backward(q, k, v, g, levels=3, K=3, variant=variant)
        b = O.backward(q, k, v, g, levels=3, K=3, variant=variant, forced=f)
        for name in ("dq", "dk", "dv"):
            assert np.array_equal(a[name], b[name])


# ---------------------------------------------------------------- position encoding and given V levels

PE_CASES = [
    # variant, B, H, W, heads, d, L, K, with_w, pe, vgiven
    ("B", 1, 6, 7, 2, 4, 3, 2, True, True, False),
    ("A", 1, 7, 6, 1, 4, 3, 2, False, True, False),
    ("B", 1, 6, 7, 2, 4, 3, 2, True, False, True),
    ("A", 2, 5, 6, 1, 4, 3, 2, False, False, True),
    ("B", 1, 9, 8, 1, 4, 4, [0, 3, 1, 2], True, True, True),
    ("A", 1, 4, 5, 2, 4, 1, 3, False, True, False),         # one level
    ("B", 2, 1, 11, 1, 4, 3, 2, False, True, True),         # one-row maps
]


@pytest.mark.parametrize("variant,B,H,W,heads,d,L,K,with_w,pe,vgiven", PE_CASES)
def test_backward_with_position_encoding_and_given_v_matches_finite_differences(variant, B, H, W, heads, d, L, K,
                                                                                with_w, pe, vgiven):
    """The gradients of the multiscale position encoding's kernels and bias, of caller-supplied V levels,
    and of q, k, v, w with either present, against central differences of the forward (kept keys forced,
    dyadic inputs, step 2^-12)."""
    rng = np.random.default_rng(B * 1000 + H * 10 + W + L + 3 * pe + 7 * vgiven)
    q, k, v, g = (dyadic(rng, (B, H, W, heads, d)) for _ in range(4))
    C = heads * d
    w = (rng.integers(1, 64, size=(B, H * W, heads, L)) / 64.0).astype(np.float32) if with_w else None
    dims = O.level_dims(H, W, L)
    vl = [None] + [dyadic(rng, (B, dims[l][0], dims[l][1], heads, d)) for l in range(1, L)] if vgiven else None
    pw = dyadic(rng, (L, C, 3, 3), -32, 33) if pe else None
    pb = dyadic(rng, (L, C), -32, 33) if pe else None
    forced = O.forward(q, k, v, levels=L, K=K, variant=variant, w=w, v_levels=vl, pe_weight=pw,
                       pe_bias=pb)["sel_idx"]
    grads = O.backward(q, k, v, g, levels=L, K=K, variant=variant, w=w, forced=forced, v_levels=vl, pe_weight=pw,
                       pe_bias=pb)
    inputs = {"q": q, "k": k, "v": v, "w": w, "pw": pw, "pb": pb, "vl": vl}

    def loss(args):
        r = O.forward(args["q"], args["k"], args["v"], levels=L, K=K, variant=variant, w=args["w"], forced=forced,
                      v_levels=args["vl"], pe_weight=args["pw"], pe_bias=args["pb"])
        return float((r["out"] * g).sum())

    tensors = [("q", None, q, grads["dq"]), ("k", None, k, grads["dk"]), ("v", None, v, grads["dv"])]
    if with_w:
        tensors.append(("w", None, w, grads["dw"]))
    if pe:
        tensors += [("pw", None, pw, grads["dpe_weight"]), ("pb", None, pb, grads["dpe_bias"])]
    else:
        assert grads["dpe_weight"] is None
    if vgiven:
        tensors += [("vl", l, vl[l], grads["dv_levels"][l]) for l in range(1, L)]
    else:
        assert grads["dv_levels"] is None

    for name, lev, arr, grad in tensors:
        assert grad is not None and grad.shape == arr.shape, name
        scale_g = max(np.abs(grad).max(), 1e-3)

        def at(delta):
            args = dict(inputs)
            if lev is None:
                args[name] = (arr + delta).astype(np.float32)
            else:
                args["vl"] = list(vl)
                args["vl"][lev] = (arr + delta).astype(np.float32)
            return loss(args)

        for _ in range(4):
            idx = tuple(int(rng.integers(0, s)) for s in arr.shape)
            e = np.zeros_like(arr)
            e[idx] = EPS
            fd = (at(e) - at(-e)) / (2 * EPS)
            assert abs(fd - grad[idx]) <= 1e-7 * scale_g + 1e-9, (name, lev, idx, fd, grad[idx])
        u = rng.integers(-1, 2, size=arr.shape).astype(np.float32)
        fd = (at(EPS * u) - at(-EPS * u)) / (2 * EPS)
        exact = float((grad * u).sum())
        assert abs(fd - exact) <= 1e-6 * max(1.0, abs(exact)), (name, lev, fd, exact)


def _torch_depthwise(x, wk, bias):
    """[B,H,W,C] x [C,3,3] (+ [C]) -> the 3x3 depth-wise cross-correlation with zero padding, by torch."""
    C = x.shape[-1]
    y = torch.nn.functional.conv2d(x.permute(0, 3, 1, 2), wk.reshape(C, 1, 3, 3), bias=bias, padding=1, groups=C)
    return y.permute(0, 2, 3, 1)


@pytest.mark.parametrize("vgiven", [False, True])
@pytest.mark.parametrize("H,W,L", [(8, 8, 3), (7, 10, 3)])
def test_backward_b_every_key_kept_with_encoding_is_autograd_of_the_closed_form(vgiven, H, W, L):
    """QuadTree-B keeping every key, with the position encoding and pooled or given V levels: out =
    sum_l w_l * (dense attention of level l + depth-wise conv of V^l), broadcast to the finest tokens;
    every gradient (q, k, v, w, the kernels, the bias, the given V levels) by torch autograd in float64
    of that formula, with torch's own conv2d for the encoding."""
    rng = np.random.default_rng(16 + vgiven)
    B, NH, d = 1, 2, 4
    C = NH * d
    q, k, v, g = (dyadic(rng, (B, H, W, NH, d)) for _ in range(4))
    w = rng.random((B, H * W, NH, L)).astype(np.float32)
    dims = O.level_dims(H, W, L)
    vl = [None] + [dyadic(rng, (B, dims[l][0], dims[l][1], NH, d)) for l in range(1, L)] if vgiven else None
    pw = dyadic(rng, (L, C, 3, 3), -32, 33)
    pb = dyadic(rng, (L, C), -32, 33)
    tau = 0.5
    leaves = [torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (q, k, v, w, pw, pb)]
    tvl = [None] + [torch.tensor(vl[l], dtype=torch.float64, requires_grad=True) for l in range(1, L)] if vgiven else None
    tq, tk, tv, tw, tpw, tpb = leaves
    xq, xk, xv = (t.reshape(B, H, W, C) for t in (tq, tk, tv))
    out = torch.zeros((B, H, W, NH, d), dtype=torch.float64)
    ys, xs = torch.arange(H), torch.arange(W)
    for l in range(L):
        if l >= 1 and vgiven:
            xv = tvl[l].reshape(B, dims[l][0], dims[l][1], C)
        Hl, Wl = xq.shape[1], xq.shape[2]
        m = _torch_dense(xq.reshape(B, Hl * Wl, NH, d), xk.reshape(B, Hl * Wl, NH, d),
                         xv.reshape(B, Hl * Wl, NH, d), tau).reshape(B, Hl, Wl, NH, d)
        m = m + _torch_depthwise(xv, tpw[l], tpb[l]).reshape(B, Hl, Wl, NH, d)
        anc = m[:, (ys >> l)][:, :, (xs >> l)]
        out = out + tw[..., l].reshape(B, H, W, NH, 1) * anc
        xq, xk = _torch_pool(xq), _torch_pool(xk)
        if not vgiven:
            xv = _torch_pool(xv)
    (out * torch.tensor(g, dtype=torch.float64)).sum().backward()
    r = O.backward(q, k, v, g, levels=L, K=64, variant="B", w=w, scale=tau, v_levels=vl, pe_weight=pw, pe_bias=pb)
    for name, t in (("dq", tq), ("dk", tk), ("dv", tv), ("dw", tw), ("dpe_weight", tpw), ("dpe_bias", tpb)):
        np.testing.assert_allclose(r[name], t.grad.numpy(), atol=1e-11, rtol=0, err_msg=name)
    if vgiven:
        for l in range(1, L):
            np.testing.assert_allclose(r["dv_levels"][l], tvl[l].grad.numpy(), atol=1e-11, rtol=0)
