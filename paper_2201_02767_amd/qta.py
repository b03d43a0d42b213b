"""Python binding of the QuadTree attention C ABI (``include/qta.h``).

Argument marshalling only: every function here checks tensor shapes, allocates outputs with torch
on the inputs' device, and calls the library on torch's current HIP stream. All arithmetic happens
in the HIP kernels of ``libqta.so``. There is no fallback: if the library is missing the calls raise.

Tensors are NHWC: q, k, v are ``[B, H, W, heads, d]`` (fp32 or bf16, contiguous, on a GPU).
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libqta.so")
MAX_LEVELS = 16

_DTYPES = {torch.float32: 0, torch.bfloat16: 1}
_VARIANTS = {"A": 0, "B": 1}


class QtaError(RuntimeError):
    def __init__(self, func: str, status: int, msg: str):
        super().__init__(f"{func}: {msg} (status {status})")
        self.status = status


class WorkspaceLayout(ctypes.Structure):
    _fields_ = [
        ("levels", ctypes.c_int),
        ("H", ctypes.c_int * MAX_LEVELS),
        ("W", ctypes.c_int * MAX_LEVELS),
        ("blocked", ctypes.c_int * MAX_LEVELS),
        ("K", ctypes.c_int * MAX_LEVELS),
        ("q", ctypes.c_size_t * MAX_LEVELS),
        ("k", ctypes.c_size_t * MAX_LEVELS),
        ("v", ctypes.c_size_t * MAX_LEVELS),
        ("msg", ctypes.c_size_t * MAX_LEVELS),
        ("sel_idx", ctypes.c_size_t * MAX_LEVELS),
        ("sel_key", ctypes.c_size_t * MAX_LEVELS),
        ("pe0", ctypes.c_size_t),
        ("total", ctypes.c_size_t),
    ]


class Options(ctypes.Structure):
    _fields_ = [
        ("K_levels", ctypes.c_void_p),
        ("v_levels", ctypes.c_void_p),
        ("pe_weight", ctypes.c_void_p),
        ("pe_bias", ctypes.c_void_p),
        ("epipolar", ctypes.c_int),
        ("aux_stream", ctypes.c_void_p),
        ("aux_stream2", ctypes.c_void_p),
        ("dpe_weight", ctypes.c_void_p),
        ("dpe_bias", ctypes.c_void_p),
        ("dv_levels", ctypes.c_void_p),
    ]


_lib = None
_P = ctypes.c_void_p
_I = ctypes.c_int
_F = ctypes.c_float
_SIGS = {
    "qta_status_str": ([_I], ctypes.c_char_p),
    "qta_level_dims": ([_I, _I, _I, _P, _P], _I),
    "qta_get_workspace_layout": ([_I, _I, _I, _I, _I, _I, _I, _I, ctypes.POINTER(WorkspaceLayout)], _I),
    "qta_workspace_bytes": ([_I, _I, _I, _I, _I, _I, _I, _I], ctypes.c_size_t),
    "qta_get_workspace_layout_ex": ([_I, _I, _I, _I, _I, _I, _I, _I, _P, ctypes.POINTER(WorkspaceLayout)], _I),
    "qta_workspace_bytes_ex": ([_I, _I, _I, _I, _I, _I, _I, _I, _P], ctypes.c_size_t),
    "qta_forward": ([_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _F, _P, _P, ctypes.c_size_t, _P], _I),
    "qta_forward_ex": ([_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _F, _P, _P, _P, ctypes.c_size_t, _P], _I),
    "qta_forward_ex_noalloc": ([_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _F, _P, _P, _P], _I),
    "qta_backward_workspace_bytes_ex": ([_I, _I, _I, _I, _I, _I, _I, _I, _I, _P], ctypes.c_size_t),
    "qta_backward_ex": ([_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _F, _P, _P, ctypes.c_size_t,
                         _P, _P, _P, _P, _P, ctypes.c_size_t, _P], _I),
    "qta_backward_finest_ex": ([_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _F, _P, _P, ctypes.c_size_t,
                                _P, _P, _P, _P, _P, ctypes.c_size_t, _P], _I),
    "qta_build_pyramid": ([_P, _P, _I, _I, _I, _I, _I, _I, _P], _I),
    "qta_coarse_attn": ([_P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _F, _P, _P, _P, _P], _I),
    "qta_topk": ([_P, _P, _I, _I, _I, _P, _P, _P], _I),
    "qta_fine_attn": ([_P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _F, _P, _P, _P, _P, _P, _P], _I),
    "qta_finest_attn": ([_P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _F, _P, _P, _I, _P, _P, _P, _P], _I),
}


_AUX = {}


def _aux_stream(device, which: int = 0) -> "torch.cuda.Stream":
    """Auxiliary stream `which` (0 or 1) of a device, one each for the whole process and shared by
    every plan: each new stream takes the next hardware queue, and shared streams keep the
    backward's three streams on distinct queues however many plans exist."""
    dev = torch.device(device)
    idx = dev.index if dev.index is not None else torch.cuda.current_device()
    if idx not in _AUX:
        _AUX[idx] = (torch.cuda.Stream(device=idx), torch.cuda.Stream(device=idx))
    return _AUX[idx][which]


def lib() -> ctypes.CDLL:
    """Load ``libqta.so`` (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run paper_2201_02767_amd.build.build() first")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            fn = getattr(handle, name)
            fn.argtypes = args
            fn.restype = res
        _lib = handle
    return _lib


def _check(func: str, status: int) -> None:
    if status != 0:
        raise QtaError(func, status, lib().qta_status_str(status).decode())


def _stream(device: torch.device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _require(t: torch.Tensor, name: str, dtype=None, ndim=None) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on a GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got shape {tuple(t.shape)}")


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype not in _DTYPES:
        raise ValueError(f"unsupported dtype {t.dtype}; fp32 and bf16 are supported")
    return _DTYPES[t.dtype]


def _scale(scale) -> float:
    return 0.0 if scale is None else float(scale)


# ------------------------------------------------------------------------------------------------
# geometry
# ------------------------------------------------------------------------------------------------

def level_dims(H: int, W: int, levels: int) -> list[tuple[int, int]]:
    hl = (ctypes.c_int * MAX_LEVELS)()
    wl = (ctypes.c_int * MAX_LEVELS)()
    _check("qta_level_dims", lib().qta_level_dims(H, W, levels, ctypes.addressof(hl), ctypes.addressof(wl)))
    return [(hl[i], wl[i]) for i in range(levels)]


def k_levels(K, levels: int) -> list[int]:
    """One K for every level, or a sequence whose entry l (1 <= l < levels) is level l's K (entry 0
    unused), as the list the library reads."""
    if isinstance(K, int):
        return [K] * levels
    Kl = [int(x) for x in K]
    if len(Kl) != levels:
        raise ValueError(f"K needs one entry per level ({levels}), got {len(Kl)}")
    Kl[0] = 0
    return Kl


def _k_table(Kl):
    return (ctypes.c_int * MAX_LEVELS)(*Kl)


_FAKE_PTR = 256      # a non-NULL, aligned, never-dereferenced device address (layout queries only)


def _layout_options(K, levels, v_supplied, pe, epipolar=False):
    """Options for a layout query (only which options are present matters there)."""
    tbl = _k_table(k_levels(K, levels))
    opt = Options()
    opt.K_levels = ctypes.addressof(tbl)
    opt.epipolar = int(bool(epipolar))
    vt = None
    if v_supplied:
        vt = (ctypes.c_void_p * MAX_LEVELS)(*([_FAKE_PTR] * MAX_LEVELS))
        opt.v_levels = ctypes.addressof(vt)
    if pe:
        opt.pe_weight = _FAKE_PTR
    return opt, (tbl, vt)


def workspace_layout(B, heads, H, W, d, levels, K, dtype: torch.dtype, v_supplied: bool = False,
                     pe: bool = False, epipolar: bool = False) -> WorkspaceLayout:
    lay = WorkspaceLayout()
    opt, keep = _layout_options(K, levels, v_supplied, pe, epipolar)
    _check("qta_get_workspace_layout_ex",
           lib().qta_get_workspace_layout_ex(B, heads, H, W, d, levels, 1, _DTYPES[dtype], ctypes.byref(opt),
                                             ctypes.byref(lay)))
    return lay


def workspace_bytes(B, heads, H, W, d, levels, K, dtype: torch.dtype, v_supplied: bool = False,
                    pe: bool = False, epipolar: bool = False) -> int:
    opt, keep = _layout_options(K, levels, v_supplied, pe, epipolar)
    return int(lib().qta_workspace_bytes_ex(B, heads, H, W, d, levels, 1, _DTYPES[dtype], ctypes.byref(opt)))


# ------------------------------------------------------------------------------------------------
# the whole forward
# ------------------------------------------------------------------------------------------------

class Plan:
    """Pre-allocated output and workspace for repeated forwards of one problem shape.

    ``K``: one count for every level, or one entry per level (entry l is level l's K, entry 0
    unused). ``v_supplied``: V's coarser levels come from the caller (``v_levels`` of run/prepare).
    ``pe``: a multiscale position encoding is applied (``pe_weight``/``pe_bias`` of run/prepare).
    ``epipolar``: attention along rows only (every row an independent 1 x W map; levels, workspace
    views and ``v_levels`` then follow the B*H maps of 1 x W).
    """

    def __init__(self, B, H, W, heads, d, *, levels, K, variant, dtype, device, scale=None, v_supplied=False,
                 pe=False, epipolar=False):
        self.B, self.H, self.W, self.heads, self.d = B, H, W, heads, d
        self.levels, self.variant, self.dtype = levels, variant, dtype
        self.K_levels = k_levels(K, levels)
        self.K = K if isinstance(K, int) else self.K_levels
        self.scale = scale
        self.v_supplied = bool(v_supplied)
        self.pe = bool(pe)
        self.epipolar = bool(epipolar)
        # the maps the library works on: B*H rows of 1 x W for epipolar attention
        self.mB, self.mH = (B * H, 1) if self.epipolar else (B, H)
        self.device = torch.device(device)
        self.layout = workspace_layout(B, heads, H, W, d, levels, K, dtype, self.v_supplied, self.pe, self.epipolar)
        self._k_tbl = _k_table(self.K_levels)
        nbytes = max(int(self.layout.total), 256)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self.out = torch.empty((B, H, W, heads, d), dtype=dtype, device=self.device)

    def _args(self, q, k, v, w, v_levels, pe_weight, pe_bias):
        for name, t in (("q", q), ("k", k), ("v", v)):
            _require(t, name, self.dtype, 5)
            if tuple(t.shape) != (self.B, self.H, self.W, self.heads, self.d):
                raise ValueError(f"{name} has shape {tuple(t.shape)}")
        if w is not None:
            _require(w, "w", torch.float32, 4)
            if tuple(w.shape) != (self.B, self.H * self.W, self.heads, self.levels):
                raise ValueError(f"w has shape {tuple(w.shape)}")
        if (v_levels is not None) != self.v_supplied:
            raise ValueError("v_levels must be given exactly when the plan was made with v_supplied=True")
        vtbl = None
        if v_levels is not None:
            vtbl = (ctypes.c_void_p * MAX_LEVELS)()
            for l in range(1, self.levels):
                t = v_levels[l]
                _require(t, f"v_levels[{l}]", self.dtype, 5)
                if tuple(t.shape) != (self.mB, self.layout.H[l], self.layout.W[l], self.heads, self.d):
                    raise ValueError(f"v_levels[{l}] has shape {tuple(t.shape)}")
                vtbl[l] = t.data_ptr()
        if (pe_weight is not None) != self.pe:
            raise ValueError("pe_weight must be given exactly when the plan was made with pe=True")
        C = self.heads * self.d
        if pe_weight is not None:
            _require(pe_weight, "pe_weight", torch.float32)
            if tuple(pe_weight.shape) != (self.levels, C, 3, 3):
                raise ValueError(f"pe_weight has shape {tuple(pe_weight.shape)}")
            if pe_bias is not None:
                _require(pe_bias, "pe_bias", torch.float32)
                if tuple(pe_bias.shape) != (self.levels, C):
                    raise ValueError(f"pe_bias has shape {tuple(pe_bias.shape)}")
        elif pe_bias is not None:
            raise ValueError("pe_bias needs pe_weight")
        opt = Options()
        opt.K_levels = ctypes.addressof(self._k_tbl)
        opt.v_levels = ctypes.addressof(vtbl) if vtbl is not None else None
        opt.pe_weight = pe_weight.data_ptr() if pe_weight is not None else None
        opt.pe_bias = pe_bias.data_ptr() if pe_bias is not None else None
        opt.epipolar = int(self.epipolar)
        return opt, vtbl

    def _call_args(self, q, k, v, w, opt, stream):
        return (_ptr(q), _ptr(k), _ptr(v), _ptr(w), self.B, self.heads, self.H, self.W, self.d, self.levels,
                self.K_levels[1] if self.levels > 1 else max(self.K_levels[0], 1), _VARIANTS[self.variant],
                _DTYPES[self.dtype], _scale(self.scale), ctypes.byref(opt), _ptr(self.out), _ptr(self.workspace),
                self.workspace.numel(), stream)

    def run(self, q, k, v, w=None, stream=None, v_levels=None, pe_weight=None, pe_bias=None):
        opt, vtbl = self._args(q, k, v, w, v_levels, pe_weight, pe_bias)
        s = _stream(self.device) if stream is None else ctypes.c_void_p(stream)
        _check("qta_forward_ex", lib().qta_forward_ex(*self._call_args(q, k, v, w, opt, s)))
        return self.out

    def prepare(self, q, k, v, w=None, v_levels=None, pe_weight=None, pe_bias=None):
        """Validate once and return a zero-argument callable that re-issues this forward on the
        current stream (for timing loops and graph capture: no per-call Python checks)."""
        opt, vtbl = self._args(q, k, v, w, v_levels, pe_weight, pe_bias)
        fn = lib().qta_forward_ex
        args = self._call_args(q, k, v, w, opt, _stream(self.device))
        keep = (q, k, v, w, vtbl, v_levels, opt, pe_weight, pe_bias)

        def call():
            st = fn(*args)
            if st != 0:
                _check("qta_forward_ex", st)
            return keep
        return call

    def prepare_finest(self, q, k, v, w=None):
        """A zero-argument callable that re-runs only the finest-level kernel (attention at level 0
        with the fused combination) on the selections and messages this plan's last run left in
        its workspace."""
        if self.levels < 2:
            raise ValueError("a single-level problem has no finest-level stage")
        fn = lib().qta_finest_attn
        sidx, skey = self.selection(1)
        msgs = [self.message(j) for j in range(1, self.levels)]
        table = (ctypes.c_void_p * (self.levels - 1))(*[m.data_ptr() for m in msgs])
        args = (_ptr(q), _ptr(k), _ptr(v), self.mB, self.heads, self.mH, self.W, self.d, self.K_levels[1],
                _VARIANTS[self.variant], _DTYPES[self.dtype], _scale(self.scale), _ptr(sidx), _ptr(skey),
                self.levels, ctypes.addressof(table), _ptr(w), _ptr(self.out), _stream(self.device))
        keep = (q, k, v, w, table, msgs)

        def call():
            st = fn(*args)
            if st != 0:
                _check("qta_finest_attn", st)
            return keep
        return call

    def prepare_coarse(self):
        """A zero-argument callable that re-runs only the coarsest level (attention with its top-K,
        through ``qta_coarse_attn``) on the coarsest pyramid level this plan's last run left in its
        workspace, writing the same message and selections again."""
        if self.levels < 2:
            raise ValueError("a single-level problem has no separate coarse stage")
        c = self.levels - 1
        lay = self.layout
        shape = (self.mB, lay.H[c], lay.W[c], self.heads, self.d)
        qc, kc = self._view(lay.q[c], shape, self.dtype), self._view(lay.k[c], shape, self.dtype)
        if self.v_supplied:
            raise ValueError("the coarse stage alone is timed with pooled V levels")
        vc = self._view(lay.v[c], shape, self.dtype)
        sidx, skey = self.selection(c)
        msg = self.message(c)
        fn = lib().qta_coarse_attn
        args = (_ptr(qc), _ptr(kc), _ptr(vc), self.mB, self.heads, lay.H[c], lay.W[c], self.d, self.K_levels[c],
                _VARIANTS[self.variant], _DTYPES[self.dtype], _scale(self.scale), _ptr(msg), _ptr(sidx), _ptr(skey),
                _stream(self.device))
        keep = (qc, kc, vc, sidx, skey, msg)

        def call():
            st = fn(*args)
            if st != 0:
                _check("qta_coarse_attn", st)
            return keep
        return call

    # ---- backward ----
    def _bwd_buffers(self, want_dw):
        if getattr(self, "_grads", None) is None:
            opt, keep = _layout_options(self.K_levels, self.levels, self.v_supplied, self.pe, self.epipolar)
            nbytes = lib().qta_backward_workspace_bytes_ex(
                self.B, self.heads, self.H, self.W, self.d, self.levels,
                self.K_levels[1] if self.levels > 1 else max(self.K_levels[0], 1), _VARIANTS[self.variant],
                _DTYPES[self.dtype], ctypes.byref(opt))
            if nbytes == 0:
                raise ValueError("unsupported problem for the backward pass")
            shape = (self.B, self.H, self.W, self.heads, self.d)
            self.bwd_workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
            self._grads = [torch.empty(shape, dtype=torch.float32, device=self.device) for _ in range(3)]
            self._dw = None
            # the gradients of the position encoding and of given V levels (their own inputs)
            C = self.heads * self.d
            self.grad_extra = {}
            if self.pe:
                self.grad_extra["dpe_weight"] = torch.empty((self.levels, C, 3, 3), dtype=torch.float32,
                                                            device=self.device)
                self.grad_extra["dpe_bias"] = torch.empty((self.levels, C), dtype=torch.float32, device=self.device)
            if self.v_supplied:
                lay = self.layout
                self.grad_extra["dv_levels"] = [None] + [
                    torch.empty((self.mB, lay.H[l], lay.W[l], self.heads, self.d), dtype=torch.float32,
                                device=self.device) for l in range(1, self.levels)]
        if want_dw and self._dw is None:
            self._dw = torch.empty((self.B, self.H * self.W, self.heads, self.levels), dtype=torch.float32,
                                   device=self.device)
        return self._grads, (self._dw if want_dw else None)

    def _bwd_args(self, q, k, v, w, dout, stream, overlap=True, v_levels=None, pe_weight=None, pe_bias=None):
        opt, vtbl = self._args(q, k, v, w, v_levels, pe_weight, pe_bias)
        _require(dout, "dout", self.dtype, 5)
        if tuple(dout.shape) != (self.B, self.H, self.W, self.heads, self.d):
            raise ValueError(f"dout has shape {tuple(dout.shape)}")
        want_dw = self.variant == "B" and w is not None
        (dq, dk, dv), dw = self._bwd_buffers(want_dw)
        dvl_tbl = None
        if self.pe:
            opt.dpe_weight = self.grad_extra["dpe_weight"].data_ptr()
            opt.dpe_bias = self.grad_extra["dpe_bias"].data_ptr()
        if self.v_supplied:
            dvl_tbl = (ctypes.c_void_p * MAX_LEVELS)()
            for l in range(1, self.levels):
                dvl_tbl[l] = self.grad_extra["dv_levels"][l].data_ptr()
            opt.dv_levels = ctypes.addressof(dvl_tbl)
        if overlap:
            # the process's second and third streams on this device for the sorts and key passes
            # (the library orders them against the caller's stream)
            opt.aux_stream = _aux_stream(self.device, 0).cuda_stream
            opt.aux_stream2 = _aux_stream(self.device, 1).cuda_stream
        args = (_ptr(q), _ptr(k), _ptr(v), _ptr(w), _ptr(dout), self.B, self.heads, self.H, self.W, self.d,
                self.levels, self.K_levels[1] if self.levels > 1 else max(self.K_levels[0], 1),
                _VARIANTS[self.variant], _DTYPES[self.dtype], _scale(self.scale), ctypes.byref(opt),
                _ptr(self.workspace), self.workspace.numel(), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dw),
                _ptr(self.bwd_workspace), self.bwd_workspace.numel(), stream)
        return args, (opt, vtbl, dvl_tbl), (dq, dk, dv, dw)

    def backward(self, q, k, v, dout, w=None, stream=None, overlap=True, v_levels=None, pe_weight=None, pe_bias=None):
        """Gradients (dq, dk, dv, dw) in fp32 of the last ``run`` on the same inputs, for the upstream
        gradient ``dout`` (the kept keys of that run held fixed). ``dw`` is None unless QuadTree-B
        with ``w``. With given V levels or a position encoding (pass the forward's ``v_levels``,
        ``pe_weight``, ``pe_bias``), their gradients are in ``self.grad_extra``: ``dpe_weight``,
        ``dpe_bias`` and ``dv_levels`` (entry l >= 1). The returned tensors are the plan's own
        buffers, overwritten by the next call. ``overlap``: run the finest level's sort and key pass
        on a second stream and the coarser levels' on a third (both one per device for the process),
        beside the query passes and the coarse level (False: everything on the one stream)."""
        s = _stream(self.device) if stream is None else ctypes.c_void_p(stream)
        args, opt, grads = self._bwd_args(q, k, v, w, dout, s, overlap, v_levels, pe_weight, pe_bias)
        _check("qta_backward_ex", lib().qta_backward_ex(*args))
        return grads

    def prepare_backward(self, q, k, v, dout, w=None, finest_only=False, v_levels=None, pe_weight=None, pe_bias=None):
        """Validate once and return a zero-argument callable that re-issues this backward on the
        current stream (``finest_only``: just its level-0 kernel, for timing it; the gradients are
        then no longer the layer's)."""
        args, opt, grads = self._bwd_args(q, k, v, w, dout, _stream(self.device), True, v_levels, pe_weight, pe_bias)
        fn = lib().qta_backward_finest_ex if finest_only else lib().qta_backward_ex
        keep = (q, k, v, w, dout, opt, grads)

        def call():
            st = fn(*args)
            if st != 0:
                _check("qta_backward_ex", st)
            return keep
        return call

    # views into the workspace after run()
    def _view(self, off, shape, dtype):
        n = 1
        for s_ in shape:
            n *= s_
        nbytes = n * torch.empty((), dtype=dtype).element_size()
        return self.workspace[off:off + nbytes].view(dtype).view(shape)

    def pyramid(self, which: str, level: int):
        """Pyramid level `level` (>= 1) of q, k or v as [B, H_l, W_l, heads, d] (B*H maps of one row
        for epipolar attention); blocked storage is unpacked into a new tensor."""
        lay = self.layout
        off = getattr(lay, which)[level]
        H, W = lay.H[level], lay.W[level]
        if not lay.blocked[level]:
            return self._view(off, (self.mB, H, W, self.heads, self.d), self.dtype)
        return self._unblock(off, H, W)

    def _unblock(self, off, H, W):
        Hp, Wp = (H + 1) // 2, (W + 1) // 2
        t = self._view(off, (self.mB, self.heads, Hp, Wp, 2, 2, self.d), self.dtype)
        t = t.permute(0, 2, 4, 3, 5, 1, 6).reshape(self.mB, 2 * Hp, 2 * Wp, self.heads, self.d)
        return t[:, :H, :W].contiguous()

    def message(self, level: int):
        lay = self.layout
        return self._view(lay.msg[level], (self.mB, lay.H[level] * lay.W[level], self.heads, self.d), torch.float32)

    def selection(self, level: int):
        lay = self.layout
        shape = (self.mB, self.heads, lay.H[level] * lay.W[level], lay.K[level])
        return (self._view(lay.sel_idx[level], shape, torch.int32),
                self._view(lay.sel_key[level], shape, torch.float32))


def forward(q, k, v, *, levels: int, K, variant: str, w=None, scale=None, v_levels=None, pe_weight=None,
            pe_bias=None, epipolar: bool = False) -> torch.Tensor:
    """QuadTree attention forward; returns ``out`` [B, H, W, heads, d] in q's dtype. ``K``: one count
    or one per level (entry 0 unused); ``v_levels``: None, or a list whose entry l (l >= 1) is V at
    level l, [B, H_l, W_l, heads, d]; ``pe_weight`` fp32 [levels, heads*d, 3, 3] and ``pe_bias`` fp32
    [levels, heads*d]: the multiscale position encoding; ``epipolar``: attention along rows only."""
    _require(q, "q", None, 5)
    B, H, W, heads, d = q.shape
    plan = Plan(B, H, W, heads, d, levels=levels, K=K, variant=variant, dtype=q.dtype, device=q.device,
                scale=scale, v_supplied=v_levels is not None, pe=pe_weight is not None, epipolar=epipolar)
    return plan.run(q, k, v, w, v_levels=v_levels, pe_weight=pe_weight, pe_bias=pe_bias)


NOALLOC_WORKSPACE_BYTES = 64 << 20      # QTA_NOALLOC_WORKSPACE_BYTES of include/qta.h


def forward_noalloc(q, k, v, out, *, levels: int, K, variant: str, w=None, scale=None, epipolar: bool = False):
    """``qta_forward_ex_noalloc``: the forward into the caller's ``out`` (same shape and dtype as q),
    with the library's own per-device workspace array, so nothing is allocated (the binding allocates
    nothing either). ``K``: one count or one per level (entry 0 unused). Calls on one device that can
    overlap in time race on that array."""
    for name, t in (("q", q), ("k", k), ("v", v), ("out", out)):
        _require(t, name, q.dtype, 5)
        if tuple(t.shape) != tuple(q.shape):
            raise ValueError(f"{name} has shape {tuple(t.shape)}")
    B, H, W, heads, d = q.shape
    if w is not None:
        _require(w, "w", torch.float32, 4)
    Kl = k_levels(K, levels)
    tbl = _k_table(Kl)
    opt = Options()
    opt.K_levels = ctypes.addressof(tbl)
    opt.epipolar = int(bool(epipolar))
    _check("qta_forward_ex_noalloc", lib().qta_forward_ex_noalloc(
        _ptr(q), _ptr(k), _ptr(v), _ptr(w), B, heads, H, W, d, levels, Kl[1] if levels > 1 else max(Kl[0], 1),
        _VARIANTS[variant], _dtype_code(q), _scale(scale), ctypes.byref(opt), _ptr(out), _stream(q.device)))
    return out


class _QuadTreeAttention(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, w, plan):
        out = plan.run(q, k, v, w).clone()
        ctx.plan = plan
        if w is not None:
            ctx.save_for_backward(q, k, v, w)
        else:
            ctx.save_for_backward(q, k, v)
        return out

    @staticmethod
    def backward(ctx, dout):
        saved = ctx.saved_tensors
        q, k, v = saved[:3]
        w = saved[3] if len(saved) > 3 else None
        dq, dk, dv, dw = ctx.plan.backward(q, k, v, dout.to(q.dtype).contiguous(), w)
        cast = lambda t: None if t is None else t.to(q.dtype)
        return cast(dq), cast(dk), cast(dv), (dw.clone() if dw is not None else None), None


def attention(q, k, v, *, levels: int, K, variant: str, w=None, scale=None, epipolar: bool = False,
              plan: "Plan | None" = None) -> torch.Tensor:
    """Differentiable QuadTree attention (autograd): the forward of ``forward`` and, on backward,
    the gradients of q, k, v (in q's dtype) and w (fp32) from ``qta_backward_ex``, with the kept keys
    of the forward held fixed. Pass a ``plan`` to reuse its buffers; a plan's workspace holds one
    forward at a time, so a plan must not be shared by two layers awaiting their backward."""
    _require(q, "q", None, 5)
    B, H, W, heads, d = q.shape
    if plan is None:
        plan = Plan(B, H, W, heads, d, levels=levels, K=K, variant=variant, dtype=q.dtype, device=q.device,
                    scale=scale, epipolar=epipolar)
    return _QuadTreeAttention.apply(q, k, v, w, plan)


# ------------------------------------------------------------------------------------------------
# stage calls
# ------------------------------------------------------------------------------------------------

def build_pyramid(x: torch.Tensor, levels: int) -> list[torch.Tensor]:
    """Levels 1..levels-1 of an NHWC map ``[B, H, W, C]``; returns a list indexed by level (entry 0 is x)."""
    _require(x, "x", None, 4)
    B, H, W, C = x.shape
    dims = level_dims(H, W, levels)
    total = sum(B * h * w_ * C for h, w_ in dims[1:])
    buf = torch.empty(max(total, 1), dtype=x.dtype, device=x.device)
    _check("qta_build_pyramid", lib().qta_build_pyramid(
        _ptr(x), _ptr(buf), B, H, W, C, levels, _dtype_code(x), _stream(x.device)))
    out, off = [x], 0
    for h, w_ in dims[1:]:
        n = B * h * w_ * C
        out.append(buf[off:off + n].view(B, h, w_, C))
        off += n
    return out


def coarse_attn(qc, kc, vc, *, K: int, variant: str, scale=None, select: bool = True):
    """Coarsest-level attention. Returns (msg [B,N,heads,d] fp32, sel_idx, sel_key) (None without selection)."""
    for name, t in (("qc", qc), ("kc", kc), ("vc", vc)):
        _require(t, name, qc.dtype, 5)
    B, Hc, Wc, heads, d = qc.shape
    N = Hc * Wc
    msg = torch.empty((B, N, heads, d), dtype=torch.float32, device=qc.device)
    sel_idx = sel_key = None
    if select:
        sel_idx = torch.empty((B, heads, N, K), dtype=torch.int32, device=qc.device)
        sel_key = torch.empty((B, heads, N, K), dtype=torch.float32, device=qc.device)
    _check("qta_coarse_attn", lib().qta_coarse_attn(
        _ptr(qc), _ptr(kc), _ptr(vc), B, heads, Hc, Wc, d, K, _VARIANTS[variant], _dtype_code(qc), _scale(scale),
        _ptr(msg), _ptr(sel_idx), _ptr(sel_key), _stream(qc.device)))
    return msg, sel_idx, sel_key


def topk(keys: torch.Tensor, K: int, cand_idx: torch.Tensor | None = None):
    """Row-wise top-K of fp32 ``keys`` [rows, n]; returns (idx int32 [rows, K], key fp32 [rows, K])."""
    _require(keys, "keys", torch.float32, 2)
    rows, n = keys.shape
    if cand_idx is not None:
        _require(cand_idx, "cand_idx", torch.int32, 2)
        if tuple(cand_idx.shape) != (rows, n):
            raise ValueError("cand_idx must match keys")
    idx = torch.empty((rows, K), dtype=torch.int32, device=keys.device)
    key = torch.empty((rows, K), dtype=torch.float32, device=keys.device)
    _check("qta_topk", lib().qta_topk(_ptr(keys), _ptr(cand_idx), rows, n, K, _ptr(idx), _ptr(key),
                                      _stream(keys.device)))
    return idx, key


def fine_attn(ql, kl, vl, parent_idx, parent_key, *, K: int, variant: str, scale=None):
    """Intermediate-level attention. Returns (msg fp32 [B,N,heads,d], sel_idx, sel_key [B,heads,N,K])."""
    for name, t in (("ql", ql), ("kl", kl), ("vl", vl)):
        _require(t, name, ql.dtype, 5)
    _require(parent_idx, "parent_idx", torch.int32, 4)
    if parent_key is not None:
        _require(parent_key, "parent_key", torch.float32, 4)
    B, Hl, Wl, heads, d = ql.shape
    N = Hl * Wl
    msg = torch.empty((B, N, heads, d), dtype=torch.float32, device=ql.device)
    sel_idx = torch.empty((B, heads, N, K), dtype=torch.int32, device=ql.device)
    sel_key = torch.empty((B, heads, N, K), dtype=torch.float32, device=ql.device)
    _check("qta_fine_attn", lib().qta_fine_attn(
        _ptr(ql), _ptr(kl), _ptr(vl), B, heads, Hl, Wl, d, K, _VARIANTS[variant], _dtype_code(ql), _scale(scale),
        _ptr(parent_idx), _ptr(parent_key), _ptr(msg), _ptr(sel_idx), _ptr(sel_key), _stream(ql.device)))
    return msg, sel_idx, sel_key


def finest_attn(q0, k0, v0, parent_idx, parent_key, coarser_msgs, *, K: int, variant: str, w=None, scale=None):
    """Level-0 attention fused with the combination; ``coarser_msgs[j-1]`` is level j's fp32 message."""
    for name, t in (("q0", q0), ("k0", k0), ("v0", v0)):
        _require(t, name, q0.dtype, 5)
    _require(parent_idx, "parent_idx", torch.int32, 4)
    B, H, W, heads, d = q0.shape
    levels = len(coarser_msgs) + 1
    for j, m in enumerate(coarser_msgs):
        _require(m, f"coarser_msgs[{j}]", torch.float32, 4)
    if w is not None:
        _require(w, "w", torch.float32, 4)
    table = (ctypes.c_void_p * max(levels - 1, 1))(*[m.data_ptr() for m in coarser_msgs])
    out = torch.empty_like(q0)
    _check("qta_finest_attn", lib().qta_finest_attn(
        _ptr(q0), _ptr(k0), _ptr(v0), B, heads, H, W, d, K, _VARIANTS[variant], _dtype_code(q0), _scale(scale),
        _ptr(parent_idx), _ptr(parent_key), levels, ctypes.addressof(table), _ptr(w), _ptr(out),
        _stream(q0.device)))
    return out
