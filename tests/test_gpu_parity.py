"""GPU parity: every stage of the HIP library against the CPU oracle on the same seeded inputs.

Cases span several workgroup tiles with ragged tails, odd maps, both variants, both storage types,
d = 32 and 64, K from 1 to 64, and the five workloads at their full sizes.
"""
import sys

import numpy as np
import pytest
import torch

import paper_2201_02767_amd as P
from paper_2201_02767_amd.inputs import WORKLOADS, make_level_weights, make_pe, make_qkv, make_v_levels, round_bf16
from oracle import oracle as O
from tests import brute
from tests.parity import TOL, assert_rows_ordered, check_selection, rel_err, to_np

pytestmark = pytest.mark.gpu

TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    P.lib()
    return torch.device("cuda:0")


def announce(msg: str) -> None:
    print(f"[gpu case] {msg}", file=sys.stderr, flush=True)


def rand_qkv(seed, B, H, W, heads, d, dtype, scale=1.0):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(3):
        x = (rng.standard_normal((B, H, W, heads, d)) * scale).astype(np.float32)
        if dtype == "bf16":
            x = round_bf16(x)
        out.append(x)
    return out


def dev_t(x, dtype, dev):
    return torch.from_numpy(np.ascontiguousarray(x)).to(dev).to(TDT[dtype])


# ------------------------------------------------------------------------------------------------
# end-to-end protocol
# ------------------------------------------------------------------------------------------------

def run_and_compare(dev, q, k, v, *, levels, K, variant, dtype, w=None, scale=None, label="", v_levels=None,
                    pe_weight=None, pe_bias=None, epipolar=False):
    """GPU forward vs teacher-forced oracle; returns a dict of the measured agreement. ``K``: one
    count or one per level; ``v_levels``: None or the caller's V levels (numpy, entry l >= 1);
    ``epipolar``: attention along rows, checked against the oracle on the B*H one-row maps."""
    B, H, W, heads, d = q.shape
    announce(f"forward {label} B={B} H={H} W={W} heads={heads} d={d} L={levels} K={K} {variant} {dtype}"
             f"{' V levels given' if v_levels is not None else ''}{' epipolar' if epipolar else ''}")
    plan = P.Plan(B, H, W, heads, d, levels=levels, K=K, variant=variant, dtype=TDT[dtype], device=dev, scale=scale,
                  v_supplied=v_levels is not None, pe=pe_weight is not None, epipolar=epipolar)
    Kl = P.k_levels(K, levels)
    wt = None if w is None else torch.from_numpy(w).to(dev)
    vl = None if v_levels is None else [None] + [dev_t(v_levels[l], dtype, dev) for l in range(1, levels)]
    pw = None if pe_weight is None else torch.from_numpy(np.ascontiguousarray(pe_weight)).to(dev)
    pb = None if pe_bias is None else torch.from_numpy(np.ascontiguousarray(pe_bias)).to(dev)
    out = plan.run(dev_t(q, dtype, dev), dev_t(k, dtype, dev), dev_t(v, dtype, dev), wt, v_levels=vl, pe_weight=pw,
                   pe_bias=pb)
    torch.cuda.synchronize()
    g_out = to_np(out)
    g_sel = [None] + [to_np(plan.selection(l)[0]) for l in range(1, levels)]
    if epipolar:        # the oracle sees what the library computes: B*H maps of one row
        q, k, v = (x.reshape(B * H, 1, W, heads, d) for x in (q, k, v))
        w = None if w is None else w.reshape(B * H, W, heads, levels)
        g_out = g_out.reshape(B * H, 1, W, heads, d)
    ref = O.forward(q, k, v, levels=levels, K=K, variant=variant, dtype=dtype, w=w, scale=scale,
                    forced=g_sel, want_candidates=True, want_pyramids=True, v_levels=v_levels, pe_weight=pe_weight,
                    pe_bias=pe_bias)
    res = {"sel": {}, "msg": {}}
    for l in range(1, levels):
        for name in ("qk" if v_levels is not None else "qkv"):
            gp = to_np(plan.pyramid(name, l)).reshape(ref["pyr_" + name][l].shape)
            assert np.array_equal(gp, ref["pyr_" + name][l]), f"pyramid {name} level {l} differs"
        assert g_sel[l].shape[-1] == Kl[l]
        chk = check_selection(g_sel[l], ref["cand_idx"][l], ref["cand_key"][l], Kl[l])
        assert chk["bad"] == 0, f"level {l} selection: {chk}"
        res["sel"][l] = chk
        e = rel_err(to_np(plan.message(l)), ref["msg"][l])
        res["msg"][l] = e
        assert e <= TOL[dtype], f"level {l} message error {e}"
        gk = to_np(plan.selection(l)[1])
        sel_ok = g_sel[l] >= 0
        # the kept keys' scores agree with the oracle's (A carries them down as s_parent)
        np.testing.assert_allclose(gk[sel_ok], ref["sel_key"][l][sel_ok], rtol=2e-3 if dtype == "bf16" else 2e-5,
                                   atol=1e-6)
    e = rel_err(g_out, ref["out"])
    res["out"] = e
    assert e <= TOL[dtype], f"output error {e}"
    # the oracle's own (unforced) choice agrees wherever there is no near-tie
    return res, g_out, ref


# ------------------------------------------------------------------------------------------------
# stage: pyramid (bit-exact)
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,B,H,W,C,L", [
    ("f32", 1, 16, 16, 32, 3), ("bf16", 2, 25, 42, 64, 5), ("f32", 1, 15, 13, 256, 4), ("bf16", 1, 1, 9, 64, 4),
    ("f32", 3, 37, 53, 96, 6), ("bf16", 2, 200, 336, 64, 5), ("f32", 1, 60, 80, 256, 3),
    # 16 top tokens per workgroup; tokens too wide for the staged pass (80 chunks, fp32 and bf16)
    ("bf16", 1, 33, 17, 32, 4), ("f32", 1, 19, 23, 320, 4), ("bf16", 2, 9, 11, 640, 3),
    # three-level pass: 3 of 4 chunk slots per thread used; one-row maps with two level-2 rounds;
    # 8 top tokens per workgroup
    ("f32", 2, 21, 27, 160, 4), ("bf16", 3, 1, 45, 1600, 4), ("f32", 2, 9, 7, 8, 4),
    # four-level pass: 2 top tokens per workgroup; 4 chunk slots per thread; one-row maps; a ragged
    # map; after a two-level pass (7 levels)
    ("f32", 2, 9, 7, 8, 5), ("f32", 1, 37, 29, 64, 5), ("bf16", 2, 1, 77, 64, 5), ("bf16", 1, 17, 35, 32, 5),
    ("f32", 1, 70, 90, 32, 7),
])
def test_pyramid_bit_exact(dev, dtype, B, H, W, C, L):
    rng = np.random.default_rng(H * W + C)
    x = rng.standard_normal((B, H, W, C)).astype(np.float32)
    if dtype == "bf16":
        x = round_bf16(x)
    announce(f"pyramid {dtype} {B}x{H}x{W}x{C} L={L}")
    levels = P.build_pyramid(dev_t(x, dtype, dev), L)
    torch.cuda.synchronize()
    ref = x
    for l in range(1, L):
        ref = O.pool_level(ref, dtype)
        assert np.array_equal(to_np(levels[l]), ref), f"level {l}"


@pytest.mark.parametrize("W", [2, 9, 130])
def test_pyramid_bf16_rounding_ties(dev, W):
    """Pooled bf16 tokens whose fp32 mean lands exactly halfway between two bf16 values: on a one-row
    map each token averages a pair, here a bf16 value and the next one up (or the same value). The
    kernels' nearest-even rounding must equal the oracle's, whose rounding is pinned to the format's
    definition on the CPU; both tie directions occur (even kept significands round down, odd up)."""
    rng = np.random.default_rng(77 + W)
    C = 64
    a = round_bf16((rng.standard_normal((1, 1, W, C)) * np.exp2(rng.integers(-60, 60, size=(1, 1, W, C))))
                   .astype(np.float32))
    x = a.copy()
    up = rng.random((1, 1, W // 2, C)) < 0.8
    x[:, :, 1::2] = (a[:, :, 0:W - 1:2].view(np.uint32) + np.where(up, 0x10000, 0).astype(np.uint32)).view(np.float32)
    announce(f"pyramid bf16 rounding ties 1x1x{W}x{C}")
    levels = P.build_pyramid(dev_t(x, "bf16", dev), 2)
    torch.cuda.synchronize()
    ref = O.pool_level(x, "bf16")
    assert np.array_equal(to_np(levels[1]).view(np.uint32), ref.view(np.uint32))
    m = ((x[:, :, 0:W - 1:2] + x[:, :, 1::2]) * np.float32(0.5)).astype(np.float32).view(np.uint32)
    ties = (m & 0xFFFF) == 0x8000
    assert ties.mean() > 0.5 and (ties & ((m >> 16) & 1 == 1)).any() and (ties & ((m >> 16) & 1 == 0)).any()


# ------------------------------------------------------------------------------------------------
# stage: top-K
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("rows,n,K", [(5, 7, 3), (64, 64, 8), (33, 100, 16), (17, 300, 64), (9, 1024, 16),
                                      (4, 3000, 32), (3, 16, 64)])
def test_topk_matches_full_sort(dev, rows, n, K):
    rng = np.random.default_rng(rows * n + K)
    keys = rng.integers(-20, 20, size=(rows, n)).astype(np.float32) / 4      # many exact ties
    names = rng.permutation(rows * n).reshape(rows, n).astype(np.int32) % (3 * n)
    names[rng.random((rows, n)) < 0.2] = -1                                    # non-candidates
    announce(f"topk rows={rows} n={n} K={K}")
    for cand in (None, names):
        idx, key = P.topk(torch.from_numpy(keys).to(dev), K,
                          None if cand is None else torch.from_numpy(cand).to(dev))
        torch.cuda.synchronize()
        idx, key = to_np(idx), to_np(key)
        for r in range(rows):
            nm = np.arange(n) if cand is None else cand[r]
            ok = nm >= 0
            kk, ii = keys[r][ok], nm[ok]
            order = np.lexsort((ii, -kk))
            m = min(K, len(ii))
            assert idx[r, :m].tolist() == ii[order[:m]].tolist()
            assert np.all(idx[r, m:] == -1)
            assert np.array_equal(key[r, :m], kk[order[:m]])
            assert np.all(key[r, m:] == 0)


# ------------------------------------------------------------------------------------------------
# stages in isolation, teacher-forced from the oracle
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("variant,dtype,d,K", [("B", "f32", 32, 8), ("A", "f32", 64, 4), ("B", "bf16", 64, 16),
                                               ("A", "bf16", 32, 5)])
def test_stages_teacher_forced(dev, variant, dtype, d, K):
    B, H, W, heads, L = 2, 45, 38, 2, 4
    q, k, v = rand_qkv(11 + K, B, H, W, heads, d, dtype)
    w = np.random.default_rng(3).random((B, H * W, heads, L)).astype(np.float32) if variant == "B" else None
    ref = O.forward(q, k, v, levels=L, K=K, variant=variant, dtype=dtype, w=w, want_candidates=True,
                    want_pyramids=True)
    dims = ref["dims"]

    def pyr(name, l):
        if l == 0:
            return {"q": q, "k": k, "v": v}[name]
        Hl, Wl = dims[l]
        return ref["pyr_" + name][l].reshape(B, Hl, Wl, heads, d)

    # coarsest level
    c = L - 1
    announce(f"coarse stage {variant} {dtype} d={d} K={K}")
    msg, sidx, skey = P.coarse_attn(*(dev_t(pyr(n, c), dtype, dev) for n in "qkv"), K=K, variant=variant)
    torch.cuda.synchronize()
    chk = check_selection(to_np(sidx), ref["cand_idx"][c], ref["cand_key"][c], K)
    assert chk["bad"] == 0, chk
    assert_rows_ordered(to_np(sidx), to_np(skey))
    forced = O.forward(q, k, v, levels=L, K=K, variant=variant, dtype=dtype, w=w,
                       forced=[None] * c + [to_np(sidx)])
    assert rel_err(to_np(msg), forced["msg"][c]) <= TOL[dtype]
    # intermediate levels, each fed the oracle's parent selections
    for l in range(c - 1, 0, -1):
        announce(f"fine stage level {l} {variant} {dtype} d={d} K={K}")
        pidx = torch.from_numpy(ref["sel_idx"][l + 1]).to(dev)
        pkey = torch.from_numpy(ref["sel_key"][l + 1].astype(np.float32)).to(dev)
        msg, sidx, skey = P.fine_attn(*(dev_t(pyr(n, l), dtype, dev) for n in "qkv"), pidx, pkey, K=K, variant=variant)
        torch.cuda.synchronize()
        chk = check_selection(to_np(sidx), ref["cand_idx"][l], ref["cand_key"][l], K)
        assert chk["bad"] == 0, chk
        assert_rows_ordered(to_np(sidx), to_np(skey))
        frc = [None] * L
        frc[l] = to_np(sidx)
        for j in range(l + 1, L):
            frc[j] = ref["sel_idx"][j]
        forced = O.forward(q, k, v, levels=L, K=K, variant=variant, dtype=dtype, w=w, forced=frc)
        assert rel_err(to_np(msg), forced["msg"][l]) <= TOL[dtype]
    # finest level with the combination
    announce(f"finest stage {variant} {dtype} d={d} K={K}")
    pidx = torch.from_numpy(ref["sel_idx"][1]).to(dev)
    pkey = torch.from_numpy(ref["sel_key"][1].astype(np.float32)).to(dev)
    msgs = [torch.from_numpy(ref["msg"][j].astype(np.float32)).to(dev) for j in range(1, L)]
    out = P.finest_attn(dev_t(q, dtype, dev), dev_t(k, dtype, dev), dev_t(v, dtype, dev), pidx, pkey, msgs, K=K,
                        variant=variant, w=None if w is None else torch.from_numpy(w).to(dev))
    torch.cuda.synchronize()
    assert rel_err(to_np(out), ref["out"]) <= TOL[dtype]


@pytest.mark.parametrize("variant", ["A", "B"])
def test_stage_selection_order_with_ties_and_empty_slots(dev, variant):
    """The stage calls' row order on exact ties and padded rows: constant queries and keys make every
    logit equal, so each row keeps the lowest indices, listed in ascending order; with more slots than
    keys (K = 6 on a 2 x 2 coarsest map) the two empty slots come last as (-1, 0). The intermediate
    stage gets parents whose candidate sets all tie in the same way."""
    B, heads, d = 2, 2, 32
    one = np.ones((B, 2, 2, heads, d), np.float32)
    rng = np.random.default_rng(5)
    vc = rng.standard_normal(one.shape).astype(np.float32)
    announce(f"stage selection order {variant}")
    msg, sidx, skey = P.coarse_attn(dev_t(one, "f32", dev), dev_t(one, "f32", dev), dev_t(vc, "f32", dev), K=6,
                                    variant=variant)
    torch.cuda.synchronize()
    idx, key = to_np(sidx), to_np(skey)
    assert_rows_ordered(idx, key)
    assert (idx[..., :4] == np.arange(4)).all() and (idx[..., 4:] == -1).all()
    np.testing.assert_allclose(key[..., :4], 0.25, rtol=1e-6)
    # level 1 of a 4 x 6 map: parents (2 x 3 map) each kept keys 5, 0, 3 of the parent level
    Hl, Wl, K = 4, 6, 3
    ql = np.ones((B, Hl, Wl, heads, d), np.float32)
    pidx = np.broadcast_to(np.array([5, 0, 3], np.int32), (B, heads, 6, K)).copy()
    pkey = np.full((B, heads, 6, K), 1.0 / 3, np.float32)
    msg, sidx, skey = P.fine_attn(dev_t(ql, "f32", dev), dev_t(ql, "f32", dev), dev_t(ql, "f32", dev),
                                  torch.from_numpy(pidx).to(dev), torch.from_numpy(pkey).to(dev), K=K, variant=variant)
    torch.cuda.synchronize()
    idx, key = to_np(sidx), to_np(skey)
    assert_rows_ordered(idx, key)
    # candidates: children of parent keys 0, 3 and 5 (level-1 flat indices); equal scores keep the
    # three lowest: 0, 1 and 6 (children (0,0), (0,1), (1,0) of parent key 0)
    assert (idx == np.array([0, 1, 6], np.int32)).all()


# ------------------------------------------------------------------------------------------------
# end-to-end: shapes that span tiles, ragged tails and the degenerate cases
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("variant", ["A", "B"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("B,H,W,heads,d,L,K", [
    (1, 16, 16, 1, 32, 3, 4),       # tiny workload shape
    (2, 37, 53, 2, 32, 4, 8),       # odd map, several tiles, ragged tail
    (1, 30, 41, 3, 64, 3, 16),      # d = 64, three heads
    (1, 23, 19, 1, 32, 5, 1),       # K = 1, deep pyramid on an odd map
    (1, 1, 40, 2, 32, 4, 3),        # single row
    (1, 12, 12, 1, 32, 3, 20),      # K above the candidate count (two slot chunks)
    (1, 30, 26, 2, 64, 3, 24),      # 96 candidates per sibling group, d = 64 (two slots per lane)
    (2, 37, 53, 1, 32, 4, 32),      # 128 candidates, ragged map, four levels (detection's K)
    (1, 20, 24, 2, 64, 3, 64),      # K = 64 (four slot chunks)
    (1, 29, 32, 2, 64, 3, 8),       # coarse level of exactly 64 tokens (8 x 8), d = 64
])
def test_forward_parity(dev, variant, dtype, B, H, W, heads, d, L, K):
    q, k, v = rand_qkv(B * H * W + L * K, B, H, W, heads, d, dtype)
    w = np.random.default_rng(5).random((B, H * W, heads, L)).astype(np.float32) if variant == "B" else None
    run_and_compare(dev, q, k, v, levels=L, K=K, variant=variant, dtype=dtype, w=w)


@pytest.mark.parametrize("variant", ["A", "B"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_single_level_is_dense_attention(dev, variant, dtype):
    B, H, W, heads, d = 2, 9, 11, 2, 32
    q, k, v = rand_qkv(21, B, H, W, heads, d, dtype)
    announce(f"single level {variant} {dtype}")
    out = P.forward(dev_t(q, dtype, dev), dev_t(k, dtype, dev), dev_t(v, dtype, dev), levels=1, K=4, variant=variant)
    torch.cuda.synchronize()
    ref = brute.dense_attention(q.reshape(B, H * W, heads, d), k.reshape(B, H * W, heads, d),
                                v.reshape(B, H * W, heads, d), 1 / np.sqrt(d))
    assert rel_err(to_np(out).reshape(ref.shape), ref) <= TOL[dtype]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_largest_coarse_level(dev, dtype):
    """1024 coarse tokens, the cap: 64x64 map, two levels."""
    q, k, v = rand_qkv(22, 1, 64, 64, 1, 32, dtype, scale=0.5)
    run_and_compare(dev, q, k, v, levels=2, K=8, variant="B", dtype=dtype, label="coarse cap")


def test_piecewise_constant_a_equals_dense(dev):
    """QuadTree-A on maps whose Q and K are constant per coarsest cell equals dense attention."""
    rng = np.random.default_rng(23)
    L, H, W, d = 3, 32, 32, 32
    f = 2 ** (L - 1)
    cq = rng.standard_normal((1, H // f, W // f, 1, d)).astype(np.float32) * 0.5
    ck = rng.standard_normal((1, H // f, W // f, 1, d)).astype(np.float32) * 0.5
    q = np.repeat(np.repeat(cq, f, 1), f, 2)
    k = np.repeat(np.repeat(ck, f, 1), f, 2)
    v = rng.standard_normal((1, H, W, 1, d)).astype(np.float32)
    for K in (1, 3):
        announce(f"piecewise constant K={K}")
        out = P.forward(dev_t(q, "f32", dev), dev_t(k, "f32", dev), dev_t(v, "f32", dev), levels=L, K=K, variant="A")
        torch.cuda.synchronize()
        ref = brute.dense_attention(q.reshape(1, -1, 1, d), k.reshape(1, -1, 1, d), v.reshape(1, -1, 1, d),
                                    1 / np.sqrt(d))
        assert rel_err(to_np(out).reshape(ref.shape), ref) <= 1e-4


@pytest.mark.parametrize("variant", ["A", "B"])
def test_constant_values_give_constant_output(dev, variant):
    rng = np.random.default_rng(24)
    B, H, W, heads, d, L = 1, 29, 31, 2, 32, 4
    q, k, _ = rand_qkv(25, B, H, W, heads, d, "f32")
    c = rng.standard_normal((heads, d)).astype(np.float32)
    v = np.broadcast_to(c, (B, H, W, heads, d)).copy()
    announce(f"constant v {variant}")
    out = P.forward(dev_t(q, "f32", dev), dev_t(k, "f32", dev), dev_t(v, "f32", dev), levels=L, K=3, variant=variant)
    torch.cuda.synchronize()
    assert rel_err(to_np(out), np.broadcast_to(c, out.shape)) <= 1e-5


def test_deterministic(dev):
    q, k, v = rand_qkv(26, 2, 40, 44, 2, 32, "bf16")
    announce("determinism")
    outs = []
    for _ in range(2):
        plan = P.Plan(2, 40, 44, 2, 32, levels=4, K=8, variant="B", dtype=torch.bfloat16, device=dev)
        o = plan.run(dev_t(q, "bf16", dev), dev_t(k, "bf16", dev), dev_t(v, "bf16", dev))
        torch.cuda.synchronize()
        outs.append((to_np(o).tobytes(), to_np(plan.selection(1)[0]).tobytes(), to_np(plan.message(2)).tobytes()))
    assert outs[0] == outs[1]


def test_explicit_scale(dev):
    q, k, v = rand_qkv(27, 1, 20, 20, 1, 32, "f32")
    run_and_compare(dev, q, k, v, levels=3, K=4, variant="B", dtype="f32", scale=0.05, label="scale")


# ------------------------------------------------------------------------------------------------
# the workloads at full size
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["tiny", "matching", "stereo", "backbone", "highres", "detection", "matching_ksched",
                                  "backbone_vgiven", "backbone_pe", "stereo_epipolar"])
def test_workload_full_size(dev, name):
    wl = WORKLOADS[name]
    q, k, v = make_qkv(wl)
    w = make_level_weights(wl) if wl.variant == "B" else None
    vl = make_v_levels(wl) if wl.v_given else None
    pw, pb = make_pe(wl) if wl.pe else (None, None)
    res, _, _ = run_and_compare(dev, q, k, v, levels=wl.levels, K=wl.K, variant=wl.variant, dtype=wl.dtype, w=w,
                                label=name, v_levels=vl, pe_weight=pw, pe_bias=pb, epipolar=wl.epipolar)
    announce(f"{name}: out err {res['out']:.2e}; msg err {res['msg']}; selections {res['sel']}")


def test_tiny_all_coarse_keys(dev):
    """The 16x16 workload with K = 16 = every coarse token."""
    wl = WORKLOADS["tiny"].with_(K=16)
    q, k, v = make_qkv(wl)
    run_and_compare(dev, q, k, v, levels=wl.levels, K=wl.K, variant="A", dtype="f32", label="tiny K=16")


@pytest.mark.parametrize("variant", ["A", "B"])
def test_tiny_every_key_kept_matches_closed_forms(dev, variant):
    """K = 64 keeps every key at every level of the 16x16 map: B is dense attention per level
    (combined with w), A is the hierarchical closed form; both are checked through the oracle, which
    the CPU pins tie to those closed forms."""
    wl = WORKLOADS["tiny"].with_(K=64, variant=variant)
    q, k, v = make_qkv(wl)
    w = make_level_weights(wl) if variant == "B" else None
    run_and_compare(dev, q, k, v, levels=wl.levels, K=64, variant=variant, dtype="f32", w=w, label="tiny K=64")


# ------------------------------------------------------------------------------------------------
# per-level K (Sec. 4.1.1 schedule) and caller-supplied V levels (Sec. 3.2)
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("variant,dtype,B,H,W,heads,d,Ks", [
    ("B", "f32", 1, 60, 80, 8, 32, [0, 8, 16]),        # the feature-matching schedule at full size
    ("A", "f32", 2, 37, 29, 2, 32, [0, 4, 8, 16]),     # doubling over 4 levels, ragged map
    ("B", "bf16", 1, 45, 38, 3, 64, [0, 16, 8, 4]),    # shrinking K going up
    ("A", "bf16", 1, 33, 47, 1, 32, [0, 2, 20, 5]),    # 4K_l above 64 at one level: wide kernel there
    ("B", "f32", 2, 16, 16, 1, 32, [0, 16, 64]),       # every coarse key kept, 64 candidates below
])
def test_forward_k_schedule(dev, variant, dtype, B, H, W, heads, d, Ks):
    L = len(Ks)
    q, k, v = rand_qkv(500 + sum(Ks) + H, B, H, W, heads, d, dtype)
    w = np.random.default_rng(9).random((B, H * W, heads, L)).astype(np.float32) if variant == "B" else None
    run_and_compare(dev, q, k, v, levels=L, K=Ks, variant=variant, dtype=dtype, w=w, label=f"K schedule {Ks}")


@pytest.mark.parametrize("variant,dtype,B,H,W,heads,d,L,K", [
    ("B", "bf16", 4, 56, 56, 1, 64, 3, 8),             # backbone-like self-attention, V levels given
    ("A", "f32", 2, 37, 29, 2, 32, 4, 4),
    ("B", "f32", 1, 25, 31, 2, 32, 3, [0, 4, 8]),
])
def test_forward_supplied_v_levels(dev, variant, dtype, B, H, W, heads, d, L, K):
    q, k, v = rand_qkv(600 + H * W + L, B, H, W, heads, d, dtype)
    dims = O.level_dims(H, W, L)
    rng = np.random.default_rng(77)
    vl = [None]
    for l in range(1, L):
        x = rng.standard_normal((B, dims[l][0], dims[l][1], heads, d)).astype(np.float32)
        vl.append(round_bf16(x) if dtype == "bf16" else x)
    w = np.random.default_rng(9).random((B, H * W, heads, L)).astype(np.float32) if variant == "B" else None
    run_and_compare(dev, q, k, v, levels=L, K=K, variant=variant, dtype=dtype, w=w, v_levels=vl,
                    label="V levels given")


def test_supplied_pooled_v_levels_reproduce_default(dev):
    """Handing the library its own pooled V levels gives the default forward's output bit for bit."""
    B, H, W, heads, d, L, K = 1, 30, 22, 2, 32, 3, 8
    q, k, v = rand_qkv(700, B, H, W, heads, d, "f32")
    announce("V levels given = pooled V")
    plan = P.Plan(B, H, W, heads, d, levels=L, K=K, variant="B", dtype=torch.float32, device=dev)
    tq, tk, tv = (dev_t(x, "f32", dev) for x in (q, k, v))
    ref = plan.run(tq, tk, tv).clone()
    vl = [None] + [plan.pyramid("v", l).contiguous() for l in range(1, L)]
    plan2 = P.Plan(B, H, W, heads, d, levels=L, K=K, variant="B", dtype=torch.float32, device=dev, v_supplied=True)
    out = plan2.run(tq, tk, tv, v_levels=vl)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)


# ------------------------------------------------------------------------------------------------
# multiscale position encoding (Sec. 3.2)
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("variant,dtype,B,H,W,heads,d,L,K,given_v", [
    ("B", "f32", 1, 60, 80, 8, 32, 3, 8, False),       # matching shape, blocked intermediate level
    ("A", "bf16", 2, 37, 29, 2, 64, 4, 4, False),      # ragged map, d = 64
    ("B", "bf16", 1, 33, 47, 1, 32, 3, 20, False),     # 80 candidates: the wide kernel at both levels
    ("A", "f32", 1, 25, 31, 2, 32, 3, [0, 4, 8], True),    # with a K schedule and given V levels
    ("B", "f32", 2, 12, 9, 2, 32, 1, 4, False),        # single level: the coarse kernel forms the output
])
def test_forward_position_encoding(dev, variant, dtype, B, H, W, heads, d, L, K, given_v):
    q, k, v = rand_qkv(800 + H * W + L, B, H, W, heads, d, dtype)
    rng = np.random.default_rng(88)
    C = heads * d
    pw = (rng.standard_normal((L, C, 3, 3)) * 0.3).astype(np.float32)
    pb = (rng.standard_normal((L, C)) * 0.1).astype(np.float32)
    vl = None
    if given_v:
        dims = O.level_dims(H, W, L)
        vl = [None] + [rng.standard_normal((B, dims[l][0], dims[l][1], heads, d)).astype(np.float32)
                       for l in range(1, L)]
        if dtype == "bf16":
            vl = [None] + [round_bf16(x) for x in vl[1:]]
    w = np.random.default_rng(9).random((B, H * W, heads, L)).astype(np.float32) if variant == "B" else None
    if L == 1:
        announce(f"position encoding, single level {variant} {dtype}")
        plan = P.Plan(B, H, W, heads, d, levels=1, K=K, variant=variant, dtype=TDT[dtype], device=dev, pe=True)
        out = plan.run(dev_t(q, dtype, dev), dev_t(k, dtype, dev), dev_t(v, dtype, dev),
                       None if w is None else torch.from_numpy(w).to(dev),
                       pe_weight=torch.from_numpy(pw).to(dev), pe_bias=torch.from_numpy(pb).to(dev))
        torch.cuda.synchronize()
        ref = O.forward(q, k, v, levels=1, K=K, variant=variant, dtype=dtype, w=w, pe_weight=pw, pe_bias=pb)
        assert rel_err(to_np(out), ref["out"]) <= TOL[dtype]
        return
    run_and_compare(dev, q, k, v, levels=L, K=K, variant=variant, dtype=dtype, w=w, v_levels=vl, pe_weight=pw,
                    pe_bias=pb, label="position encoding")


# ------------------------------------------------------------------------------------------------
# attention along epipolar lines (Sec. 4.1.2): every row its own one-row map, a binary tree
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("variant,dtype,B,H,W,heads,d,L,K,given_v,pe", [
    ("B", "bf16", 2, 7, 160, 8, 32, 4, 8, False, False),    # stereo-like rows
    ("A", "f32", 1, 5, 37, 2, 32, 3, 4, False, False),      # ragged rows
    ("A", "bf16", 2, 3, 93, 1, 64, 5, [0, 2, 4, 8, 16], False, False),   # K schedule; 4 levels of pairs
    ("B", "f32", 1, 4, 50, 2, 32, 3, 20, False, False),     # 40 candidates per query
    ("A", "bf16", 2, 3, 333, 1, 64, 3, 40, False, False),   # 80 per query, 160 slots per item (four per lane)
    ("B", "bf16", 1, 6, 41, 2, 32, 3, 4, True, True),       # given V levels and the position encoding
    # 1200 coarse rows of 10 tokens, d = 64: several query rows per wave in the small-map coarse kernel
    ("A", "f32", 1, 600, 40, 2, 64, 3, 8, False, False),
    ("B", "bf16", 1, 600, 40, 2, 64, 3, 8, False, False),
    # coarse rows of 5 tokens with K = 8: padded selections, several rows per wave
    ("A", "bf16", 1, 600, 40, 2, 32, 4, 8, False, False),
])
def test_forward_epipolar(dev, variant, dtype, B, H, W, heads, d, L, K, given_v, pe):
    q, k, v = rand_qkv(900 + H * W + L, B, H, W, heads, d, dtype)
    rng = np.random.default_rng(91)
    w = rng.random((B, H * W, heads, L)).astype(np.float32) if variant == "B" else None
    vl = None
    if given_v:
        dims = O.level_dims(1, W, L)
        vl = [None] + [rng.standard_normal((B * H, 1, dims[l][1], heads, d)).astype(np.float32)
                       for l in range(1, L)]
        if dtype == "bf16":
            vl = [None] + [round_bf16(x) for x in vl[1:]]
    pw = (rng.standard_normal((L, heads * d, 3, 3)) * 0.3).astype(np.float32) if pe else None
    pb = (rng.standard_normal((L, heads * d)) * 0.1).astype(np.float32) if pe else None
    run_and_compare(dev, q, k, v, levels=L, K=K, variant=variant, dtype=dtype, w=w, v_levels=vl, pe_weight=pw,
                    pe_bias=pb, epipolar=True, label="epipolar")


def test_epipolar_rows_are_independent_at_full_size(dev):
    """On the full stereo workload, sampled rows run alone (as a 1 x 160 map) give the same output as
    in the epipolar run over all 240 rows, bit for bit: the rows do not interact."""
    wl = WORKLOADS["stereo_epipolar"]
    announce("epipolar rows independent, stereo 2 x 120 x 160")
    q, k, v = make_qkv(wl)
    w = make_level_weights(wl)
    plan = P.Plan(wl.B, wl.H, wl.W, wl.heads, wl.d, levels=wl.levels, K=wl.K, variant="B", dtype=torch.bfloat16,
                  device=dev, epipolar=True)
    out = to_np(plan.run(dev_t(q, "bf16", dev), dev_t(k, "bf16", dev), dev_t(v, "bf16", dev),
                         torch.from_numpy(w).to(dev)))
    one = P.Plan(1, 1, wl.W, wl.heads, wl.d, levels=wl.levels, K=wl.K, variant="B", dtype=torch.bfloat16, device=dev)
    w_rows = w.reshape(wl.B, wl.H, wl.W, wl.heads, wl.levels)
    for b, y in [(0, 0), (0, 57), (1, 119), (1, 3)]:
        row = [dev_t(np.ascontiguousarray(x[b:b + 1, y:y + 1]), "bf16", dev) for x in (q, k, v)]
        o = to_np(one.run(*row, torch.from_numpy(np.ascontiguousarray(w_rows[b, y])).reshape(1, wl.W, wl.heads,
                                                                                               wl.levels).to(dev)))
        torch.cuda.synchronize()
        assert np.array_equal(o[0, 0], out[b, y]), f"row {b},{y} differs from its run alone"
