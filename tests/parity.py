"""Comparison protocol between the GPU library and the CPU oracle.

* Pyramids: bit-exact (both sides pool in the same fixed fp32 order and round the same way).
* Selections: the GPU's kept set must be the exact top-K of the oracle's scores, except where the
  K-th and (K+1)-th scores lie within a relative 1e-5 of each other: then any set whose every member
  scores at least (1 - 1e-5) times every non-member is accepted (a near-tie). Scores are compared in
  the probability domain for QuadTree-B and as the recursive score s for QuadTree-A.
* Teacher forcing: the oracle is re-run with the GPU's selections at every level, so messages and
  outputs are compared on the same candidate sets even after a near-tie substitution.
* Messages and outputs: err = max over rows (b, token, head) of |g - r|_inf / max(|r|_inf,
  1e-3 * RMS(r)); the bar is 1e-4 for fp32 storage and 2e-2 for bf16 storage.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import oracle as O

TOL = {"f32": 1e-4, "bf16": 2e-2}
NEAR_TIE = 1e-5


def to_np(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.detach().cpu().numpy()


def rel_err(g: np.ndarray, r: np.ndarray) -> float:
    """Max over rows (last axis = head dim) of the row-wise relative infinity-norm error."""
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    assert g.shape == r.shape, (g.shape, r.shape)
    if r.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(r * r)))
    num = np.abs(g - r).max(axis=-1)
    den = np.maximum(np.abs(r).max(axis=-1), 1e-3 * rms)
    den = np.where(den > 0, den, 1.0)
    return float((num / den).max())


def check_selection(sel: np.ndarray, cand_idx: np.ndarray, cand_key: np.ndarray, K: int, rel: float = NEAR_TIE,
                    rows_mask: np.ndarray | None = None) -> dict:
    """Validate GPU selections ``sel`` [..., K] against oracle candidates [..., ncand].

    Returns counts of rows that are exact, accepted near-ties, and invalid (with an example)."""
    sel = sel.reshape(-1, K).astype(np.int64)
    ci = cand_idx.reshape(sel.shape[0], -1).astype(np.int64)
    ck = cand_key.reshape(sel.shape[0], -1)
    if rows_mask is not None:
        m = rows_mask.reshape(-1)
        sel, ci, ck = sel[m], ci[m], ck[m]
    valid = ci >= 0
    nvalid = valid.sum(1)
    keep = np.minimum(K, nvalid)
    slot = np.arange(K)[None, :]
    pad_ok = np.all(np.where(slot >= keep[:, None], sel == -1, True), axis=1)
    # which candidate each selected entry names
    match = (sel[:, :, None] == ci[:, None, :]) & valid[:, None, :] & (slot[:, :, None] < keep[:, None, None])
    named_once = match.sum(2)
    entries_ok = np.all(np.where(slot < keep[:, None], named_once == 1, True), axis=1)
    in_g = match.any(1)                                    # [rows, ncand]
    distinct_ok = in_g.sum(1) == keep
    big = np.inf
    min_g = np.where(in_g, ck, big).min(1)
    max_not = np.where(valid & ~in_g, ck, -big).max(1)
    near_ok = min_g >= max_not * (1 - rel)
    # exact top-K by (key desc, index asc)
    order = np.lexsort((np.where(valid, ci, np.iinfo(np.int64).max), -np.where(valid, ck, -big)), axis=1)
    rank = np.empty_like(order)
    np.put_along_axis(rank, order, np.arange(ci.shape[1])[None, :].repeat(ci.shape[0], 0), axis=1)
    exact_set = valid & (rank < keep[:, None])
    exact = np.all(exact_set == in_g, axis=1)
    ok = pad_ok & entries_ok & distinct_ok & (exact | near_ok)
    res = {"rows": int(sel.shape[0]), "exact": int((ok & exact).sum()), "near_tie": int((ok & ~exact).sum()),
           "bad": int((~ok).sum())}
    if res["bad"]:
        i = int(np.flatnonzero(~ok)[0])
        res["example"] = {"row": i, "sel": sel[i].tolist(), "cand": ci[i].tolist(),
                          "key": ck[i].tolist(), "pad_ok": bool(pad_ok[i]), "entries_ok": bool(entries_ok[i]),
                          "distinct_ok": bool(distinct_ok[i]), "min_g": float(min_g[i]), "max_not": float(max_not[i])}
    return res


def query_rows_mask(dims, level: int, B: int, heads: int) -> np.ndarray:
    """All queries of a level are real (no padding), so every row counts."""
    H, W = dims[level]
    return np.ones((B, heads, H * W), bool)


def assert_rows_ordered(idx: np.ndarray, key: np.ndarray) -> None:
    """Every selection row lists its kept keys by (score descending, index ascending), then the empty
    slots (index -1, score 0): the order the stage calls return."""
    idx = idx.reshape(-1, idx.shape[-1])
    key = key.reshape(-1, key.shape[-1]).astype(np.float64)
    live = idx >= 0
    n = live.sum(axis=1)
    # live entries first
    assert (live == (np.arange(idx.shape[1])[None, :] < n[:, None])).all(), "empty slots before kept keys"
    assert (key[~live] == 0).all()
    a_i, a_k = idx[:, :-1], key[:, :-1]
    b_i, b_k = idx[:, 1:], key[:, 1:]
    both = live[:, :-1] & live[:, 1:]
    ok = (a_k > b_k) | ((a_k == b_k) & (a_i < b_i))
    assert ok[both].all(), "kept keys not ordered by (score desc, index asc)"
