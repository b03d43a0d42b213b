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
