"""Independent numpy references used to pin the CPU oracle.

Nothing here is shared with the oracle or with the GPU library. Each function restates one fact the
paper (Tang et al., ICLR 2022) or plain mathematics fixes, in a different formulation from the
oracle's level-by-level loops:

* ``ceil_pool``        - 2x2 average pooling by padding and block sums (Sec. 3.2, pyramids);
* ``block_mean``       - direct 2^l x 2^l block mean of a power-of-two map;
* ``dense_attention``  - Eq. (1), softmax(Q K^T * tau) V per head;
* ``brute_quadtree``   - per finest query, the quadtree regions Gamma built as explicit sets of
                         tokens, coarsest first (Sec. 3.2, Fig. 1), with QuadTree-A messages over
                         Omega = Gamma - Gamma' (Eqs. 2-4) and QuadTree-B messages over Gamma
                         (Eqs. 5-6);
* ``hierarchical_weights`` - QuadTree-A when every key is kept at every level: the weight of a
                         finest key is the coarse softmax times the product of the 2x2 sibling
                         softmaxes along the key's ancestry (Eq. 4 unrolled).

These run in float64 on tiny maps only.
"""
from __future__ import annotations

import numpy as np


def ceil_pool(x: np.ndarray) -> np.ndarray:
    """[B,H,W,C] -> [B,ceil(H/2),ceil(W/2),C]: mean over the children that exist."""
    B, H, W, C = x.shape
    Hp, Wp = H + (H % 2), W + (W % 2)
    xs = np.zeros((B, Hp, Wp, C), np.float64)
    cnt = np.zeros((Hp, Wp), np.float64)
    xs[:, :H, :W] = x
    cnt[:H, :W] = 1.0
    s = xs.reshape(B, Hp // 2, 2, Wp // 2, 2, C).sum(axis=(2, 4))
    n = cnt.reshape(Hp // 2, 2, Wp // 2, 2).sum(axis=(1, 3))
    return s / n[None, :, :, None]


def pyramid(x: np.ndarray, L: int) -> list[np.ndarray]:
    out = [np.asarray(x, np.float64)]
    for _ in range(1, L):
        out.append(ceil_pool(out[-1]))
    return out


def block_mean(x: np.ndarray, level: int) -> np.ndarray:
    B, H, W, C = x.shape
    f = 2 ** level
    return np.asarray(x, np.float64).reshape(B, H // f, f, W // f, f, C).mean(axis=(2, 4))


def dense_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, tau: float) -> np.ndarray:
    """q, k, v [B, N, heads, d] -> [B, N, heads, d], Eq. (1) per head."""
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    logits = np.einsum("bihc,bjhc->bhij", q, k) * tau
    logits -= logits.max(axis=-1, keepdims=True)
    p = np.exp(logits)
    p /= p.sum(axis=-1, keepdims=True)
    return np.einsum("bhij,bjhc->bihc", p, v)


def _softmax(x: np.ndarray) -> np.ndarray:
    e = np.exp(x - x.max())
    return e / e.sum()


def _top(keys: dict, K: int) -> list:
    """The K entries of {(y, x, flat): key} with the largest key, ties to the lower flat index."""
    order = sorted(keys.items(), key=lambda kv: (-kv[1], kv[0][2]))
    return [t for t, _ in order[:K]]


def depthwise3x3(x: np.ndarray, kern: np.ndarray, bias=None) -> np.ndarray:
    """[B,H,W,C] -> [B,H,W,C]: 3x3 depth-wise cross-correlation with zero padding, kern [C,3,3]."""
    B, H, W, C = x.shape
    xp = np.zeros((B, H + 2, W + 2, C))
    xp[:, 1:-1, 1:-1] = x
    out = np.zeros((B, H, W, C))
    for ky in range(3):
        for kx in range(3):
            out += xp[:, ky:ky + H, kx:kx + W] * np.asarray(kern, np.float64)[:, ky, kx]
    if bias is not None:
        out += np.asarray(bias, np.float64)
    return out


def brute_quadtree(q, k, v, L: int, K, variant: str, tau: float, w=None, v_levels=None, pe_weight=None,
                   pe_bias=None) -> np.ndarray:
    """Output [B, H, W, heads, d] of QuadTree attention, query by query, with explicit regions.

    q, k, v: [B, H, W, heads, d]; w (variant B): [B, H*W, heads, L] or None (=> 1/L).
    K: one count, or a list whose entry l is the number of keys kept at level l (l >= 1).
    v_levels: None (V pooled like Q and K) or a list whose entry l (l >= 1) is V at level l,
    [B, H_l, W_l, heads, d].
    pe_weight [L, C, 3, 3] / pe_bias [L, C]: multiscale position encoding, a depth-wise 3x3 conv of
    V^l added to level l's message at the query's position.
    """
    Kl = [K] * L if np.ndim(K) == 0 else list(K)
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    B, H, W, NH, d = q.shape
    flat = lambda t: t.reshape(t.shape[0], t.shape[1], t.shape[2], NH * d)
    PQ, PK, PV = pyramid(flat(q), L), pyramid(flat(k), L), pyramid(flat(v), L)
    if v_levels is not None:
        for l in range(1, L):
            PV[l] = flat(np.asarray(v_levels[l], np.float64))
    PE = None
    if pe_weight is not None:
        PE = [depthwise3x3(PV[l], pe_weight[l], None if pe_bias is None else pe_bias[l]) for l in range(L)]
    out = np.zeros((B, H, W, NH, d))
    for b in range(B):
        for h in range(NH):
            sl = slice(h * d, (h + 1) * d)
            for y in range(H):
                for x in range(W):
                    c = L - 1
                    Hc, Wc = PK[c].shape[1:3]
                    region = [(yy, xx) for yy in range(Hc) for xx in range(Wc)]   # Gamma at the coarsest
                    parent_score = None                                           # A: s of kept parents
                    total = np.zeros(d)
                    for lvl in range(c, -1, -1):
                        Hl, Wl = PK[lvl].shape[1:3]
                        qv = PQ[lvl][b, y >> lvl, x >> lvl, sl]
                        logit = {(ty, tx, ty * Wl + tx): tau * float(qv @ PK[lvl][b, ty, tx, sl]) for ty, tx in region}
                        if variant == "B" or lvl == c:
                            names = list(logit)
                            p = _softmax(np.array([logit[t] for t in names]))
                            score = dict(zip(names, p))
                        else:
                            score = {}
                            for (py, px, pflat), sp in parent_score.items():
                                kids = [t for t in logit if (t[0] >> 1, t[1] >> 1) == (py, px)]
                                t_ = _softmax(np.array([logit[t] for t in kids]))
                                for t, tv in zip(kids, t_):
                                    score[t] = sp * tv
                        kept = _top(score, Kl[lvl]) if lvl > 0 else []
                        pe = 0.0 if PE is None else PE[lvl][b, y >> lvl, x >> lvl, sl]
                        if variant == "B":
                            m = sum(score[t] * PV[lvl][b, t[0], t[1], sl] for t in score)
                            wl = (1.0 / L) if w is None else float(w[b, y * W + x, h, lvl])
                            total = total + wl * (m + pe)
                        else:
                            rest = [t for t in score if t not in kept]
                            if rest:
                                total = total + sum(score[t] * PV[lvl][b, t[0], t[1], sl] for t in rest)
                            total = total + pe
                        if lvl > 0:
                            Hn, Wn = PK[lvl - 1].shape[1:3]
                            region = [(2 * t[0] + dy, 2 * t[1] + dx) for t in kept for dy in (0, 1) for dx in (0, 1)
                                      if 2 * t[0] + dy < Hn and 2 * t[1] + dx < Wn]
                            parent_score = {t: score[t] for t in kept}
                    out[b, y, x, h] = total
    return out


def hierarchical_weights(q, k, L: int, tau: float) -> np.ndarray:
    """QuadTree-A weights when every key is kept at every level: W[b, h, i, j] over finest tokens.

    W = softmax_coarse(q^c_{a(i)}, k^c_{a(j)}) * prod_{l < c} t^l, where t^l is the softmax of
    q^l_{a_l(i)} against the 2x2 siblings of a_l(j) (Eq. 4 unrolled down a power-of-two map).
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    B, H, W, NH, d = q.shape
    c = L - 1
    Wt = np.zeros((B, NH, H * W, H * W))
    for b in range(B):
        for h in range(NH):
            pq = [block_mean(q[b:b + 1, :, :, h, :], l)[0] for l in range(L)]
            pk = [block_mean(k[b:b + 1, :, :, h, :], l)[0] for l in range(L)]
            for i in range(H * W):
                yi, xi = divmod(i, W)
                qc = pq[c][yi >> c, xi >> c]
                lc = tau * np.einsum("yxc,c->yx", pk[c], qc)
                pc = np.exp(lc - lc.max())
                pc /= pc.sum()
                for j in range(H * W):
                    yj, xj = divmod(j, W)
                    wgt = pc[yj >> c, xj >> c]
                    for l in range(c - 1, -1, -1):
                        ql = pq[l][yi >> l, xi >> l]
                        ay, ax = yj >> l, xj >> l
                        sy, sx = (ay >> 1) * 2, (ax >> 1) * 2
                        sib = pk[l][sy:sy + 2, sx:sx + 2]
                        ls = tau * np.einsum("yxc,c->yx", sib, ql)
                        t = np.exp(ls - ls.max())
                        t /= t.sum()
                        wgt *= t[ay - sy, ax - sx]
                    Wt[b, h, i, j] = wgt
    return Wt


def nearest_bf16(x: float) -> float:
    """The bfloat16 value nearest to the finite float ``x``, ties to the even significand, written
    from the format's definition (8 significand bits, exponents -126..127, subnormals spaced 2^-133,
    IEEE overflow to infinity) with exact rational arithmetic: no bit manipulation."""
    from fractions import Fraction
    import math

    if x == 0.0:
        return x                                    # keeps the sign of zero
    sign = -1.0 if x < 0 else 1.0
    a = Fraction(abs(x))
    e = math.frexp(abs(x))[1] - 1                   # 2^e <= |x| < 2^(e+1)
    ulp = Fraction(2) ** (max(e, -126) - 7)         # spacing of bf16 values around |x|
    lo = (a / ulp).__floor__()                      # |x| lies in [lo*ulp, (lo+1)*ulp]
    below, above = a - lo * ulp, (lo + 1) * ulp - a
    n = lo if below < above or (below == above and lo % 2 == 0) else lo + 1
    r = n * ulp
    if r >= Fraction(2) ** 128:                     # beyond the largest finite value (2 - 2^-7) * 2^127
        return sign * math.inf
    return sign * float(r)
