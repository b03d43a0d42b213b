"""C-ABI checks that need no GPU: the library loads, exports what the header declares, and rejects
bad arguments on the host before any launch. Only validation paths are exercised here (every call
below fails validation, so nothing reaches the device)."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import paper_2201_02767_amd as P
from oracle import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qta.h")

OK, INVALID, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3
FAKE = 0x100000          # an aligned, never-dereferenced address: validation fails before use
F32, BF16 = 0, 1
VA, VB = 0, 1


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(qta_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    lib = P.lib()
    names = declared_functions()
    assert "qta_forward" in names and len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    lib = P.lib()
    for code, text in [(0, b"ok"), (1, b"invalid argument"), (2, b"unsupported shape or type"),
                       (3, b"workspace too small"), (4, b"HIP launch failed"), (99, b"unknown status")]:
        assert lib.qta_status_str(code) == text


@pytest.mark.parametrize("H,W,L", [(16, 16, 3), (60, 80, 3), (120, 160, 4), (56, 56, 3), (200, 336, 5), (15, 13, 4),
                                   (1, 9, 4)])
def test_level_dims_match_oracle(H, W, L):
    assert P.level_dims(H, W, L) == O.level_dims(H, W, L)


def test_level_dims_rejects_levels_above_a_single_token():
    with pytest.raises(P.QtaError):
        P.level_dims(2, 2, 3)          # 2x2 -> 1x1 -> (1x1 again)
    with pytest.raises(P.QtaError):
        P.level_dims(4, 4, 17)
    with pytest.raises(P.QtaError):
        P.level_dims(0, 4, 1)


def _tok_bytes(blocked, B, H, W, C, tb):
    if blocked:
        return B * ((H + 1) // 2) * ((W + 1) // 2) * 4 * C * tb
    return B * H * W * C * tb


@pytest.mark.parametrize("K,expect_blocked", [(16, True), (20, True)])
def test_workspace_layout_is_aligned_and_disjoint(K, expect_blocked):
    lay = P.workspace_layout(2, 2, 200, 336, 32, 5, K, torch.bfloat16)
    regions = []
    assert lay.blocked[0] == 0 and lay.blocked[4] == 0     # input and coarsest level stay NHWC
    for l in range(1, 5):
        N = lay.H[l] * lay.W[l]
        assert lay.blocked[l] == (1 if expect_blocked and 1 <= l <= 3 else 0)
        tok = _tok_bytes(lay.blocked[l], 2, lay.H[l], lay.W[l], 64, 2)
        regions += [(lay.q[l], tok), (lay.k[l], tok), (lay.v[l], tok), (lay.msg[l], 2 * N * 64 * 4),
                    (lay.sel_idx[l], 2 * 2 * N * K * 4), (lay.sel_key[l], 2 * 2 * N * K * 4)]
    regions.sort()
    for (o1, n1), (o2, _) in zip(regions, regions[1:]):
        assert o1 % 256 == 0 and o1 + n1 <= o2
    assert regions[-1][0] + regions[-1][1] <= lay.total
    assert P.workspace_bytes(2, 2, 200, 336, 32, 5, K, torch.bfloat16) == lay.total


def test_workspace_layout_nhwc_with_given_v_levels():
    """With V's coarser levels given by the caller, every pyramid level stays NHWC."""
    lay = P.workspace_layout(2, 2, 200, 336, 32, 5, 16, torch.bfloat16, v_supplied=True)
    assert all(lay.blocked[l] == 0 for l in range(5))


def test_workspace_bytes_zero_on_bad_shapes():
    lib = P.lib()
    assert lib.qta_workspace_bytes(1, 1, 16, 16, 48, 3, 4, F32) == 0     # d unsupported
    assert lib.qta_workspace_bytes(1, 1, 16, 16, 32, 3, 65, F32) == 0    # K too large
    assert lib.qta_workspace_bytes(1, 1, 64, 64, 32, 1, 4, F32) == 0     # 4096 coarse tokens
    assert lib.qta_workspace_bytes(0, 1, 16, 16, 32, 3, 4, F32) == 0
    assert lib.qta_workspace_bytes(1, 1, 16, 16, 32, 1, 4, F32) >= 256   # valid single level: minimal, nonzero


def _fwd(lib, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, w=None, B=1, heads=1, H=16, W=16, d=32, L=3, K=4, var=VA, dt=F32, scale=0.0,
             out=FAKE, ws=FAKE, wsb=0, stream=None)
    a.update(kw)
    return lib.qta_forward(a["q"], a["k"], a["v"], a["w"], a["B"], a["heads"], a["H"], a["W"], a["d"], a["L"], a["K"],
                           a["var"], a["dt"], a["scale"], a["out"], a["ws"], a["wsb"], a["stream"])


def test_forward_validation():
    lib = P.lib()
    assert _fwd(lib) == WORKSPACE                           # valid shape, zero workspace
    assert _fwd(lib, q=None) == INVALID
    assert _fwd(lib, out=None) == INVALID
    assert _fwd(lib, q=FAKE + 4) == INVALID                 # misaligned
    assert _fwd(lib, ws=FAKE + 16, wsb=1 << 30) == INVALID  # workspace not 256-aligned
    assert _fwd(lib, B=0) == INVALID
    assert _fwd(lib, K=0) == INVALID
    assert _fwd(lib, L=0) == INVALID
    assert _fwd(lib, L=17) == INVALID
    assert _fwd(lib, H=2, W=2, L=3) == INVALID              # level above a 1x1 map
    assert _fwd(lib, var=7) == INVALID
    assert _fwd(lib, dt=5) == INVALID
    assert _fwd(lib, d=16) == UNSUPPORTED
    assert _fwd(lib, K=65) == UNSUPPORTED
    assert _fwd(lib, H=64, W=64, L=1) == UNSUPPORTED        # coarsest level above the cap
    assert _fwd(lib, H=64, W=64, L=2) == WORKSPACE          # 32x32 = 1024 coarse tokens is allowed
    assert _fwd(lib, H=4096, W=4096, L=8) == UNSUPPORTED    # 2^24 tokens in one map
    assert _fwd(lib, H=2048, W=4096, heads=32, L=8) == UNSUPPORTED   # 2^31 bytes in one map
    assert _fwd(lib, H=2048, W=4096, L=8) == WORKSPACE


def test_stage_validation():
    lib = P.lib()
    # qta_build_pyramid: C*bytes must be a multiple of 16
    assert lib.qta_build_pyramid(FAKE, FAKE, 1, 8, 8, 6, 3, F32, None) == UNSUPPORTED
    assert lib.qta_build_pyramid(None, FAKE, 1, 8, 8, 8, 3, F32, None) == INVALID
    assert lib.qta_build_pyramid(FAKE, FAKE, 1, 2, 2, 8, 3, F32, None) == INVALID
    # qta_coarse_attn
    assert lib.qta_coarse_attn(FAKE, FAKE, FAKE, 1, 1, 4, 4, 32, 4, VB, F32, 0.0, None, None, None, None) == INVALID
    assert lib.qta_coarse_attn(FAKE, FAKE, FAKE, 1, 1, 4, 4, 32, 4, VB, F32, 0.0, FAKE, FAKE, None, None) == INVALID
    assert lib.qta_coarse_attn(FAKE, FAKE, FAKE, 1, 1, 33, 32, 32, 4, VB, F32, 0.0, FAKE, None, None, None) == UNSUPPORTED
    assert lib.qta_coarse_attn(FAKE, FAKE, FAKE, 1, 1, 4, 4, 64 + 1, 4, VB, F32, 0.0, FAKE, None, None, None) == UNSUPPORTED
    # qta_topk
    assert lib.qta_topk(FAKE, None, 0, 8, 2, FAKE, None, None) == INVALID
    assert lib.qta_topk(FAKE, None, 4, 5000, 2, FAKE, None, None) == UNSUPPORTED
    assert lib.qta_topk(FAKE, None, 4, 64, 65, FAKE, None, None) == UNSUPPORTED
    assert lib.qta_topk(None, None, 4, 64, 4, FAKE, None, None) == INVALID
    # qta_fine_attn: A needs parent scores; all outputs required
    assert lib.qta_fine_attn(FAKE, FAKE, FAKE, 1, 1, 8, 8, 32, 4, VA, F32, 0.0, FAKE, None, FAKE, FAKE, FAKE,
                             None) == INVALID
    assert lib.qta_fine_attn(FAKE, FAKE, FAKE, 1, 1, 8, 8, 32, 4, VB, F32, 0.0, FAKE, None, FAKE, None, FAKE,
                             None) == INVALID
    assert lib.qta_fine_attn(FAKE, FAKE, FAKE, 1, 1, 1, 1, 32, 4, VB, F32, 0.0, FAKE, None, FAKE, FAKE, FAKE,
                             None) == INVALID
    # qta_finest_attn: needs at least two levels and every coarser message
    table = (ctypes.c_void_p * 2)(FAKE, None)
    assert lib.qta_finest_attn(FAKE, FAKE, FAKE, 1, 1, 8, 8, 32, 4, VB, F32, 0.0, FAKE, None, 1, ctypes.addressof(table),
                               None, FAKE, None) == INVALID
    assert lib.qta_finest_attn(FAKE, FAKE, FAKE, 1, 1, 8, 8, 32, 4, VB, F32, 0.0, FAKE, None, 3, ctypes.addressof(table),
                               None, FAKE, None) == INVALID
    assert lib.qta_finest_attn(FAKE, FAKE, FAKE, 1, 1, 8, 8, 32, 4, VB, F32, 0.0, FAKE, None, 2, None,
                               None, FAKE, None) == INVALID


def test_binding_refuses_cpu_tensors():
    x = torch.zeros(1, 4, 4, 1, 32)
    with pytest.raises(ValueError):
        P.forward(x, x, x, levels=2, K=1, variant="B")


def _fastdiv_params(d):
    # the divisor parameters the library derives on the host (round-up multiply-high division)
    s = 0
    while (1 << s) < d:
        s += 1
    m = (1 << (32 + s)) // d - (1 << 32) + 1
    return m, s


@pytest.mark.parametrize("d", list(range(1, 70)) + [99, 127, 128, 129, 168, 1000, 4095, 4096, 4097, 65535, 1 << 20,
                                                      (1 << 23) + 1])
def test_fast_division_parameters_are_exact(d):
    """Quotients by multiply-high + shift equal floor division for every index the kernels divide:
    0 <= n < 2^24 (map sizes are below 2^24 tokens), checked at the edges and on a random sample."""
    m, s = _fastdiv_params(d)
    assert 0 <= m < (1 << 32)
    rng = np.random.default_rng(d)
    n = np.concatenate([np.arange(0, 4 * d + 8), rng.integers(0, 1 << 24, 4096), [(1 << 24) - 1, (1 << 31) - 1],
                        np.arange(max(0, (1 << 24) - 3 * d), 1 << 24, max(1, d // 7))]).astype(np.uint64)
    hi = (n * np.uint64(m)) >> np.uint64(32)
    q = (hi + n) >> np.uint64(s)
    assert np.all(hi + n < (1 << 32))
    assert np.array_equal(q, n // np.uint64(d))


def _klv(*vals):
    t = (ctypes.c_int * 16)()
    for i, x in enumerate(vals):
        t[i] = x
    return t


def test_layout_with_k_schedule_and_supplied_v():
    """Selections are sized by each level's K; every intermediate level is blocked whatever its
    parents' K (80 candidates included); with V supplied no V level is stored and nothing is
    blocked."""
    lib = P.lib()
    B, heads, H, W, d, L = 2, 2, 60, 80, 32, 4
    for Ks, blocked in (([0, 4, 16, 8], [0, 1, 1, 0]), ([0, 8, 20, 8], [0, 1, 1, 0])):
        lay = P.workspace_layout(B, heads, H, W, d, L, Ks, torch.float32)
        assert [lay.blocked[l] for l in range(L)] == blocked
        assert [lay.K[l] for l in range(1, L)] == Ks[1:]
        for l in range(1, L):
            N = lay.H[l] * lay.W[l]
            assert lay.sel_key[l] - lay.sel_idx[l] >= B * heads * N * Ks[l] * 4
        assert P.workspace_bytes(B, heads, H, W, d, L, Ks, torch.float32) == lay.total
    lay_v = P.workspace_layout(B, heads, H, W, d, L, [0, 4, 16, 8], torch.float32, v_supplied=True)
    assert all(lay_v.v[l] == 0 and lay_v.blocked[l] == 0 for l in range(L))
    assert lay_v.total < P.workspace_layout(B, heads, H, W, d, L, [0, 4, 16, 8], torch.float32).total


def test_forward_ex_validation():
    lib = P.lib()

    def fwd(Kl=None, vtbl=None, pw=None, pb=None, L=3, wsb=0):
        opt = P.qta.Options()
        opt.K_levels = Kl
        opt.v_levels = vtbl
        opt.pe_weight = pw
        opt.pe_bias = pb
        return lib.qta_forward_ex(FAKE, FAKE, FAKE, None, 1, 1, 16, 16, 32, L, 4, VA, F32, 0.0, ctypes.byref(opt),
                                  FAKE, FAKE, wsb, None)
    assert lib.qta_forward_ex(FAKE, FAKE, FAKE, None, 1, 1, 16, 16, 32, 3, 4, VA, F32, 0.0, None, FAKE, FAKE, 0,
                              None) == WORKSPACE                           # NULL options: plain qta_forward
    assert fwd(ctypes.addressof(_klv(0, 4, 8))) == WORKSPACE               # valid shape, zero workspace
    assert fwd(ctypes.addressof(_klv(0, 4, 0))) == INVALID
    assert fwd(ctypes.addressof(_klv(0, 65, 4))) == UNSUPPORTED
    assert fwd(ctypes.addressof(_klv(9, 4, 8))) == WORKSPACE               # entry 0 is not read
    vt = (ctypes.c_void_p * 16)()
    vt[1] = FAKE
    assert fwd(None, ctypes.addressof(vt)) == INVALID                      # level 2 missing
    vt[2] = FAKE + 8
    assert fwd(None, ctypes.addressof(vt)) == INVALID                      # misaligned
    vt[2] = FAKE
    assert fwd(None, ctypes.addressof(vt)) == WORKSPACE
    assert fwd(pb=FAKE) == INVALID                                         # a bias needs weights
    assert fwd(pw=FAKE + 4) == INVALID                                     # weights not 16-byte aligned
    assert fwd(pw=FAKE, pb=FAKE) == WORKSPACE
    assert fwd(pw=FAKE, L=1) == WORKSPACE                                  # one level with an encoding needs it
    opt = P.qta.Options()
    opt.K_levels = ctypes.addressof(_klv(0, 4, 65))
    assert lib.qta_workspace_bytes_ex(1, 1, 16, 16, 32, 3, 4, F32, ctypes.byref(opt)) == 0


def test_position_encoding_workspace():
    """Level 0's encoding is computed inside the kernel that produces level 0's message (no workspace
    buffer) on maps of more than one row when 4*K_1 <= 64, and for a single level when the map takes
    the tiled coarse kernel (more than 64 tokens); otherwise the workspace adds it, fp32, after
    everything else."""
    for H, L in ((40, 3), (20, 1)):
        base = P.workspace_layout(2, 2, H, 30, 32, L, 8, torch.bfloat16)
        fused = P.workspace_layout(2, 2, H, 30, 32, L, 8, torch.bfloat16, pe=True)
        assert fused.pe0 == 0 and fused.total == base.total
    for K, H, L in ((20, 40, 3), (8, 1, 3), (8, 2, 1)):       # wide slots, one row, one level of 60 tokens
        base = P.workspace_layout(2, 2, H, 30, 32, L, K, torch.bfloat16)
        lay = P.workspace_layout(2, 2, H, 30, 32, L, K, torch.bfloat16, pe=True)
        assert lay.pe0 >= base.total - 256 and lay.pe0 % 256 == 0
        assert lay.total >= lay.pe0 + 2 * H * 30 * 64 * 4
    single = P.workspace_layout(1, 1, 8, 8, 32, 1, 4, torch.float32, pe=True)       # 64 tokens: not fused
    assert single.total >= 8 * 8 * 32 * 4


def test_epipolar_layout_is_that_of_one_row_maps():
    """Attention along rows works on B*H maps of one row: the same workspace as that problem."""
    for dt in (torch.float32, torch.bfloat16):
        for pe in (False, True):
            a = P.workspace_layout(2, 8, 120, 160, 32, 4, 8, dt, pe=pe, epipolar=True)
            b = P.workspace_layout(240, 8, 1, 160, 32, 4, 8, dt, pe=pe)
            assert a.total == b.total and a.pe0 == b.pe0
            for f in ("H", "W", "blocked", "K", "q", "k", "v", "msg", "sel_idx", "sel_key"):
                assert list(getattr(a, f)) == list(getattr(b, f)), f
    lay = P.workspace_layout(3, 1, 7, 37, 32, 3, [0, 2, 4], torch.float32, epipolar=True)
    assert list(lay.H)[:3] == [1, 1, 1] and list(lay.W)[:3] == [37, 19, 10]


def test_epipolar_row_count_limit():
    """B*H rows must fit the map count; a count past 2^31 - 1 is rejected, not wrapped."""
    with pytest.raises(P.QtaError):
        P.workspace_layout(1 << 16, 1, 1 << 16, 8, 32, 2, 4, torch.float32, epipolar=True)


def test_backward_validation():
    """qta_backward_ex rejects before any launch: what it does not cover, missing pointers, small
    workspaces."""
    lib = P.lib()

    def bwd(L=3, K=4, Kl=None, vtbl=None, pw=None, dout=FAKE, wsb=1 << 40, gwsb=1 << 40, variant=VA):
        opt = P.qta.Options()
        opt.K_levels = Kl
        opt.v_levels = vtbl
        opt.pe_weight = pw
        return lib.qta_backward_ex(FAKE, FAKE, FAKE, None, dout, 1, 1, 16, 16, 32, L, K, variant, F32, 0.0,
                                   ctypes.byref(opt), FAKE, wsb, FAKE, FAKE, FAKE, None, FAKE, gwsb, None)
    assert bwd(dout=None) == INVALID
    assert bwd(dout=FAKE + 4) == INVALID                                    # not 16-byte aligned
    assert bwd(K=17) == UNSUPPORTED                                         # 68 candidates per group
    assert bwd(Kl=ctypes.addressof(_klv(0, 4, 20))) == UNSUPPORTED
    vt = (ctypes.c_void_p * 16)()
    vt[1] = vt[2] = FAKE
    # given V levels need somewhere to put their gradients, the encoding too
    assert bwd(vtbl=ctypes.addressof(vt)) == INVALID                        # no dv_levels
    assert bwd(pw=FAKE) == INVALID                                          # no dpe_weight
    opt = P.qta.Options()
    opt.v_levels = ctypes.addressof(vt)
    dvl = (ctypes.c_void_p * 16)()
    dvl[1] = FAKE
    opt.dv_levels = ctypes.addressof(dvl)                                   # level 2's missing
    assert lib.qta_backward_ex(FAKE, FAKE, FAKE, None, FAKE, 1, 1, 16, 16, 32, 3, 4, VA, F32, 0.0, ctypes.byref(opt),
                               FAKE, 1 << 40, FAKE, FAKE, FAKE, None, FAKE, 1 << 40, None) == INVALID
    opt = P.qta.Options()
    opt.pe_weight = FAKE
    opt.pe_bias = FAKE
    opt.dpe_weight = FAKE                                                   # dpe_bias missing for a bias
    assert lib.qta_backward_ex(FAKE, FAKE, FAKE, None, FAKE, 1, 1, 16, 16, 32, 3, 4, VA, F32, 0.0, ctypes.byref(opt),
                               FAKE, 1 << 40, FAKE, FAKE, FAKE, None, FAKE, 1 << 40, None) == INVALID
    opt.pe_bias = None
    assert lib.qta_backward_ex(FAKE, FAKE, FAKE, None, FAKE, 1, 40, 16, 16, 32, 3, 4, VA, F32, 0.0,
                               ctypes.byref(opt), FAKE, 1 << 40, FAKE, FAKE, FAKE, None, FAKE, 1 << 40,
                               None) == UNSUPPORTED                         # the encoding with C > 256
    need_pe = lib.qta_backward_workspace_bytes_ex(1, 1, 16, 16, 32, 3, 4, VA, F32, ctypes.byref(opt))
    assert need_pe > lib.qta_backward_workspace_bytes_ex(1, 1, 16, 16, 32, 3, 4, VA, F32, None)
    assert bwd(wsb=0) == WORKSPACE                                          # the forward's workspace
    assert bwd(gwsb=0) == WORKSPACE
    assert bwd(L=1, gwsb=0) == WORKSPACE                                    # one level still needs statistics
    need_a = lib.qta_backward_workspace_bytes_ex(1, 1, 16, 16, 32, 3, 4, VA, F32, None)
    need_b = lib.qta_backward_workspace_bytes_ex(1, 1, 16, 16, 32, 3, 4, VB, F32, None)
    assert need_a > need_b > 0                                              # A adds the score gradients
    assert bwd(gwsb=need_a - 1) == WORKSPACE
    assert lib.qta_backward_workspace_bytes_ex(1, 1, 16, 16, 32, 3, 4, 7, F32, None) == 0


def test_binding_structs_match_the_header(tmp_path):
    """The ctypes mirrors of the header's structs have the C layout: size and every field's offset,
    as a C compiler lays them out from include/qta.h."""
    import subprocess

    structs = {"qta_options": P.qta.Options, "qta_workspace_layout": P.qta.WorkspaceLayout}
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "qta.h"', "int main(void) {"]
    for cname, cls in structs.items():
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for fname, _ in cls._fields_:
            lines.append(f'printf("{cname} {fname} %zu\\n", offsetof({cname}, {fname}));')
    lines += ["return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l.strip()}
    for cname, cls in structs.items():
        assert got[(cname, "size")] == ctypes.sizeof(cls), cname
        for fname, _ in cls._fields_:
            assert got[(cname, fname)] == getattr(cls, fname).offset, f"{cname}.{fname}"


def test_noalloc_forward_rejects_problems_beyond_its_array():
    """qta_forward_ex_noalloc: a problem whose workspace exceeds QTA_NOALLOC_WORKSPACE_BYTES is
    rejected with QTA_ERR_WORKSPACE on the host (before the device array is looked up or any launch);
    invalid arguments as in qta_forward_ex."""
    lib = P.lib()
    text = open(HEADER).read()
    assert "#define QTA_NOALLOC_WORKSPACE_BYTES ((size_t)64 << 20)" in text
    assert P.NOALLOC_WORKSPACE_BYTES == 64 << 20
    # epipolar stereo-sized problem: 141 MiB of workspace
    opt = P.Options()
    opt.epipolar = 1
    need = lib.qta_workspace_bytes_ex(2, 8, 120, 160, 32, 4, 8, BF16, ctypes.byref(opt))
    assert need > 64 << 20
    st = lib.qta_forward_ex_noalloc(FAKE, FAKE, FAKE, None, 2, 8, 120, 160, 32, 4, 8, VB, BF16, 0.0,
                                    ctypes.byref(opt), FAKE, None)
    assert st == WORKSPACE
    # without a null pointer check failing first, a too-large plain problem is a workspace error too
    assert lib.qta_workspace_bytes(64, 8, 120, 160, 32, 4, 8, F32) > 64 << 20
    assert lib.qta_forward_ex_noalloc(FAKE, FAKE, FAKE, None, 64, 8, 120, 160, 32, 4, 8, VB, F32, 0.0, None,
                                      FAKE, None) == WORKSPACE
    # invalid arguments are still invalid
    assert lib.qta_forward_ex_noalloc(None, FAKE, FAKE, None, 1, 1, 16, 16, 32, 3, 4, VA, F32, 0.0, None,
                                      FAKE, None) == INVALID
    assert lib.qta_forward_ex_noalloc(FAKE, FAKE, FAKE, None, 1, 1, 16, 16, 48, 3, 4, VA, F32, 0.0, None,
                                      FAKE, None) == UNSUPPORTED
