"""ctypes wrapper of the plain CPU oracle (``oracle.c``).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's CPU-baseline leg are
the only users. The GPU library never imports this module, and this module imports nothing from it.

Every array handed in is float32 NHWC ``[B, H, W, heads, d]``; every message and output comes back
as float64. Level 0 is the finest level.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
MAX_LEVELS = 16

VARIANTS = {"A": 0, "B": 1}
DTYPES = {"f32": 0, "bf16": 1}


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` with gcc (-O2, no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB_PATH):
        cmd = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
               "-Wall", "-Wextra", "-o", _LIB_PATH + ".tmp", _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


class _Args(ctypes.Structure):
    _fields_ = [
        ("q", ctypes.c_void_p), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("w", ctypes.c_void_p),
        ("B", ctypes.c_int), ("heads", ctypes.c_int), ("H", ctypes.c_int), ("W", ctypes.c_int),
        ("d", ctypes.c_int), ("L", ctypes.c_int), ("K", ctypes.c_int), ("variant", ctypes.c_int),
        ("dtype", ctypes.c_int), ("K_levels", ctypes.c_void_p), ("v_levels", ctypes.c_void_p),
        ("pe_weight", ctypes.c_void_p), ("pe_bias", ctypes.c_void_p),
        ("scale", ctypes.c_double),
        ("forced", ctypes.c_void_p),
        ("out", ctypes.c_void_p),
        ("pyr_q", ctypes.c_void_p), ("pyr_k", ctypes.c_void_p), ("pyr_v", ctypes.c_void_p),
        ("msg", ctypes.c_void_p),
        ("sel_idx", ctypes.c_void_p), ("sel_key", ctypes.c_void_p),
        ("cand_idx", ctypes.c_void_p), ("cand_key", ctypes.c_void_p),
    ]


class _BwdArgs(ctypes.Structure):
    _fields_ = [
        ("fwd", _Args),
        ("dout", ctypes.c_void_p),
        ("dq", ctypes.c_void_p), ("dk", ctypes.c_void_p), ("dv", ctypes.c_void_p), ("dw", ctypes.c_void_p),
        ("dpe_weight", ctypes.c_void_p), ("dpe_bias", ctypes.c_void_p), ("dv_levels", ctypes.c_void_p),
    ]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        lib.qo_forward.argtypes = [ctypes.POINTER(_Args)]
        lib.qo_forward.restype = ctypes.c_int
        lib.qo_backward.argtypes = [ctypes.POINTER(_BwdArgs)]
        lib.qo_backward.restype = ctypes.c_int
        lib.qo_pool_level.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                      ctypes.c_int, ctypes.c_void_p]
        lib.qo_pool_level.restype = ctypes.c_int
        lib.qo_level_dims.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
        lib.qo_level_dims.restype = ctypes.c_int
        _lib = lib
    return _lib


def level_dims(H: int, W: int, L: int) -> list[tuple[int, int]]:
    lib = _load()
    hl = (ctypes.c_int * MAX_LEVELS)()
    wl = (ctypes.c_int * MAX_LEVELS)()
    if lib.qo_level_dims(H, W, L, ctypes.addressof(hl), ctypes.addressof(wl)) != 0:
        raise ValueError("bad geometry")
    return [(hl[i], wl[i]) for i in range(L)]


def pool_level(x: np.ndarray, dtype: str = "f32") -> np.ndarray:
    """One 2x2 ceil-pooling step of an NHWC float32 map ``[B, H, W, C]``."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    B, H, W, C = x.shape
    out = np.empty((B, (H + 1) // 2, (W + 1) // 2, C), np.float32)
    if _load().qo_pool_level(x.ctypes.data, B, H, W, C, DTYPES[dtype], out.ctypes.data) != 0:
        raise ValueError("pool_level failed")
    return out


def _ptr_table(arrays):
    tbl = (ctypes.c_void_p * MAX_LEVELS)()
    for i, a in enumerate(arrays):
        tbl[i] = a.ctypes.data if a is not None else None
    return tbl


def forward(q, k, v, *, levels: int, K, variant: str, dtype: str = "f32", w=None, scale=None,
            forced=None, want_candidates: bool = False, want_pyramids: bool = False, v_levels=None,
            pe_weight=None, pe_bias=None) -> dict:
    """Run the oracle. ``q, k, v``: float32 ``[B, H, W, heads, d]`` (values representable in dtype).

    ``K``: one count for every level, or a sequence indexed by level whose entry l (1 <= l < levels)
    is the number of keys kept at level l (entry 0 is ignored).
    ``v_levels``: optional list indexed by level; entry l (1 <= l < levels) is V at level l,
    ``[B, H_l, W_l, heads, d]``, used instead of pooling V.
    ``pe_weight``: optional float32 ``[levels, heads*d, 3, 3]`` depth-wise kernels of the multiscale
    position encoding; ``pe_bias``: optional float32 ``[levels, heads*d]``.
    ``forced``: optional list indexed by level; entry l (1 <= l < levels) is an int32
    ``[B, heads, N_l, K_l]`` selection that replaces the oracle's own choice at that level.
    Returns a dict with ``out`` ``[B,H,W,heads,d]`` and per-level lists ``msg`` ``[B,N_l,heads,d]``,
    ``sel_idx``/``sel_key`` ``[B,heads,N_l,K]`` (None at level 0) and, on request,
    ``cand_idx``/``cand_key`` ``[B,heads,N_l,ncand]`` and the pyramids ``pyr_q/k/v`` ``[B,H_l,W_l,C]``.
    """
    q = np.ascontiguousarray(q, dtype=np.float32)
    k = np.ascontiguousarray(k, dtype=np.float32)
    v = np.ascontiguousarray(v, dtype=np.float32)
    B, H, W, NH, d = q.shape
    assert k.shape == q.shape and v.shape == q.shape
    C = NH * d
    L = levels
    dims = level_dims(H, W, L)
    N = [h * w_ for h, w_ in dims]
    wts = None
    if w is not None:
        wts = np.ascontiguousarray(w, dtype=np.float32)
        assert wts.shape == (B, H * W, NH, L), wts.shape
    if np.ndim(K) == 0:
        Kl = [int(K)] * L
    else:
        Kl = [int(x) for x in K]
        assert len(Kl) == L, "one K per level (entry 0 ignored)"
        Kl[0] = Kl[1] if L > 1 else max(Kl[0], 1)
    K_tbl = (ctypes.c_int * MAX_LEVELS)(*Kl)
    v_tbl = None
    v_keep = []
    if v_levels is not None:
        v_tbl = (ctypes.c_void_p * MAX_LEVELS)()
        for l in range(1, L):
            vl = np.ascontiguousarray(v_levels[l], dtype=np.float32)
            assert vl.size == B * N[l] * C, (vl.shape, (B, dims[l][0], dims[l][1], NH, d))
            v_keep.append(vl)
            v_tbl[l] = vl.ctypes.data
    out = np.zeros((B, H, W, NH, d), np.float64)
    msg = [np.zeros((B, N[l], NH, d), np.float64) for l in range(L)]
    sel_idx = [None] + [np.zeros((B, NH, N[l], Kl[l]), np.int32) for l in range(1, L)]
    sel_key = [None] + [np.zeros((B, NH, N[l], Kl[l]), np.float64) for l in range(1, L)]
    ncand = [4 * Kl[l + 1] for l in range(L - 1)] + [N[L - 1]]
    cand_idx = cand_key = None
    if want_candidates:
        cand_idx = [np.zeros((B, NH, N[l], ncand[l]), np.int32) for l in range(L)]
        cand_key = [np.zeros((B, NH, N[l], ncand[l]), np.float64) for l in range(L)]
    pyr = None
    if want_pyramids:
        pyr = {t: [None] + [np.zeros((B, dims[l][0], dims[l][1], C), np.float32) for l in range(1, L)]
               for t in "qkv"}
    forced_arrays = None
    if forced is not None:
        forced_arrays = [None] * L
        for l in range(1, L):
            if forced[l] is not None:
                f = np.ascontiguousarray(forced[l], dtype=np.int32)
                assert f.shape == (B, NH, N[l], Kl[l]), (f.shape, (B, NH, N[l], Kl[l]))
                forced_arrays[l] = f

    tables = {}
    tables["msg"] = _ptr_table(msg)
    tables["sel_idx"] = _ptr_table(sel_idx)
    tables["sel_key"] = _ptr_table(sel_key)
    if want_candidates:
        tables["cand_idx"] = _ptr_table(cand_idx)
        tables["cand_key"] = _ptr_table(cand_key)
    if want_pyramids:
        for t in "qkv":
            tables["pyr_" + t] = _ptr_table(pyr[t])
    if forced_arrays is not None:
        tables["forced"] = _ptr_table(forced_arrays)

    args = _Args()
    args.q, args.k, args.v = q.ctypes.data, k.ctypes.data, v.ctypes.data
    args.w = wts.ctypes.data if wts is not None else None
    args.B, args.heads, args.H, args.W, args.d = B, NH, H, W, d
    args.L, args.K, args.variant, args.dtype = L, Kl[1] if L > 1 else Kl[0], VARIANTS[variant], DTYPES[dtype]
    args.K_levels = ctypes.addressof(K_tbl)
    pe_keep = []
    if pe_weight is not None:
        pw = np.ascontiguousarray(pe_weight, dtype=np.float32)
        assert pw.shape == (L, C, 3, 3), pw.shape
        pe_keep.append(pw)
        args.pe_weight = pw.ctypes.data
        if pe_bias is not None:
            pb = np.ascontiguousarray(pe_bias, dtype=np.float32)
            assert pb.shape == (L, C), pb.shape
            pe_keep.append(pb)
            args.pe_bias = pb.ctypes.data
    args.v_levels = ctypes.addressof(v_tbl) if v_tbl is not None else None
    args.scale = float(scale) if scale is not None else 0.0
    args.out = out.ctypes.data
    for name, tbl in tables.items():
        setattr(args, name, ctypes.addressof(tbl))
    rc = _load().qo_forward(ctypes.byref(args))
    if rc != 0:
        raise RuntimeError(f"oracle forward failed with code {rc}")
    res = {"out": out, "msg": msg, "sel_idx": sel_idx, "sel_key": sel_key, "dims": dims}
    if want_candidates:
        res["cand_idx"], res["cand_key"] = cand_idx, cand_key
    if want_pyramids:
        res["pyr_q"], res["pyr_k"], res["pyr_v"] = pyr["q"], pyr["k"], pyr["v"]
    return res


def backward(q, k, v, dout, *, levels: int, K, variant: str, dtype: str = "f32", w=None, scale=None,
             forced=None, v_levels=None, pe_weight=None, pe_bias=None) -> dict:
    """Gradients of ``sum(dout * out)`` with the kept-key sets held fixed (the oracle's own, or
    ``forced`` as in ``forward``). ``dout``: float32 ``[B, H, W, heads, d]``. ``v_levels``,
    ``pe_weight``, ``pe_bias``: as in ``forward``. Returns float64 ``dq``, ``dk``, ``dv``
    ``[B, H, W, heads, d]``; for QuadTree-B with ``w`` given, ``dw`` ``[B, H*W, heads, levels]``
    (else None); with a position encoding ``dpe_weight`` ``[levels, heads*d, 3, 3]`` and ``dpe_bias``
    ``[levels, heads*d]`` (else None); with given V levels ``dv_levels``, a list whose entry l >= 1 is
    ``[B, H_l, W_l, heads, d]`` (else None)."""
    q = np.ascontiguousarray(q, dtype=np.float32)
    k = np.ascontiguousarray(k, dtype=np.float32)
    v = np.ascontiguousarray(v, dtype=np.float32)
    g = np.ascontiguousarray(dout, dtype=np.float32)
    B, H, W, NH, d = q.shape
    assert k.shape == q.shape and v.shape == q.shape and g.shape == q.shape
    L = levels
    dims = level_dims(H, W, L)
    N = [h * w_ for h, w_ in dims]
    if np.ndim(K) == 0:
        Kl = [int(K)] * L
    else:
        Kl = [int(x) for x in K]
        assert len(Kl) == L, "one K per level (entry 0 ignored)"
        Kl[0] = Kl[1] if L > 1 else max(Kl[0], 1)
    K_tbl = (ctypes.c_int * MAX_LEVELS)(*Kl)
    wts = None
    if w is not None:
        wts = np.ascontiguousarray(w, dtype=np.float32)
        assert wts.shape == (B, H * W, NH, L), wts.shape
    forced_arrays = None
    if forced is not None:
        forced_arrays = [None] * L
        for l in range(1, L):
            if forced[l] is not None:
                f = np.ascontiguousarray(forced[l], dtype=np.int32)
                assert f.shape == (B, NH, N[l], Kl[l]), (f.shape, (B, NH, N[l], Kl[l]))
                forced_arrays[l] = f
        forced_tbl = _ptr_table(forced_arrays)
    dq, dk, dv = (np.zeros((B, H, W, NH, d), np.float64) for _ in range(3))
    dw = np.zeros((B, H * W, NH, L), np.float64) if (variant == "B" and wts is not None) else None
    C = NH * d
    keep = []
    v_tbl = dvl_tbl = None
    dvl = None
    if v_levels is not None:
        v_tbl = (ctypes.c_void_p * MAX_LEVELS)()
        dvl_tbl = (ctypes.c_void_p * MAX_LEVELS)()
        dvl = [None] + [np.zeros((B, dims[l][0], dims[l][1], NH, d), np.float64) for l in range(1, L)]
        for l in range(1, L):
            vl = np.ascontiguousarray(v_levels[l], dtype=np.float32)
            assert vl.size == B * N[l] * C, (vl.shape, (B, dims[l][0], dims[l][1], NH, d))
            keep.append(vl)
            v_tbl[l] = vl.ctypes.data
            dvl_tbl[l] = dvl[l].ctypes.data
    dpw = dpb = None
    if pe_weight is not None:
        pw = np.ascontiguousarray(pe_weight, dtype=np.float32)
        assert pw.shape == (L, C, 3, 3), pw.shape
        keep.append(pw)
        dpw = np.zeros((L, C, 3, 3), np.float64)
        dpb = np.zeros((L, C), np.float64)
        pb = None
        if pe_bias is not None:
            pb = np.ascontiguousarray(pe_bias, dtype=np.float32)
            assert pb.shape == (L, C), pb.shape
            keep.append(pb)
    args = _BwdArgs()
    f = args.fwd
    f.q, f.k, f.v = q.ctypes.data, k.ctypes.data, v.ctypes.data
    f.w = wts.ctypes.data if wts is not None else None
    f.B, f.heads, f.H, f.W, f.d = B, NH, H, W, d
    f.L, f.K, f.variant, f.dtype = L, Kl[1] if L > 1 else Kl[0], VARIANTS[variant], DTYPES[dtype]
    f.K_levels = ctypes.addressof(K_tbl)
    f.scale = float(scale) if scale is not None else 0.0
    if forced_arrays is not None:
        f.forced = ctypes.addressof(forced_tbl)
    args.dout = g.ctypes.data
    args.dq, args.dk, args.dv = dq.ctypes.data, dk.ctypes.data, dv.ctypes.data
    args.dw = dw.ctypes.data if dw is not None else None
    if v_tbl is not None:
        f.v_levels = ctypes.addressof(v_tbl)
        args.dv_levels = ctypes.addressof(dvl_tbl)
    if pe_weight is not None:
        f.pe_weight = pw.ctypes.data
        f.pe_bias = pb.ctypes.data if pb is not None else None
        args.dpe_weight = dpw.ctypes.data
        args.dpe_bias = dpb.ctypes.data
    rc = _load().qo_backward(ctypes.byref(args))
    if rc != 0:
        raise RuntimeError(f"oracle backward failed with code {rc}")
    return {"dq": dq, "dk": dk, "dv": dv, "dw": dw, "dpe_weight": dpw, "dpe_bias": dpb if pe_bias is not None else None,
            "dv_levels": dvl}
