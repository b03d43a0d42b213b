"""GPU check of qta_forward_ex_noalloc (the forward whose workspace is the library's own per-device
array) against qta_forward_ex with a caller workspace: two calls in a row, the second on a smaller
problem, each compared element by element with the workspace forward on the same inputs. Both run
the same kernels in the same order, so the outputs must be bit-identical; the parity bar of the
forward (1e-4 fp32, 2e-2 bf16 per row) is asserted as well."""
import sys

import numpy as np
import pytest
import torch

import paper_2201_02767_amd as P
from paper_2201_02767_amd.inputs import WORKLOADS, make_level_weights, make_qkv
from tests.parity import TOL, rel_err, to_np

pytestmark = pytest.mark.gpu

TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


def announce(msg: str) -> None:
    print(f"[gpu case] {msg}", file=sys.stderr, flush=True)


def _inputs(wl, dev):
    tdt = TDT[wl.dtype]
    q, k, v = (torch.from_numpy(x).to(dev).to(tdt).contiguous() for x in make_qkv(wl))
    w = torch.from_numpy(make_level_weights(wl)).to(dev) if wl.variant == "B" else None
    return q, k, v, w


def _compare(wl, dev, out_na=None):
    q, k, v, w = _inputs(wl, dev)
    announce(f"no-alloc forward {wl.name} B={wl.B} H={wl.H} W={wl.W} heads={wl.heads} d={wl.d} L={wl.levels} "
             f"K={wl.K} {wl.variant} {wl.dtype}")
    plan = P.Plan(wl.B, wl.H, wl.W, wl.heads, wl.d, levels=wl.levels, K=wl.K, variant=wl.variant,
                  dtype=TDT[wl.dtype], device=dev)
    ref = plan.run(q, k, v, w).clone()
    out = torch.full_like(q, float("nan")) if out_na is None else out_na
    P.forward_noalloc(q, k, v, out, levels=wl.levels, K=wl.K, variant=wl.variant, w=w)
    torch.cuda.synchronize()
    g, r = to_np(out), to_np(ref)
    assert np.isfinite(g).all()
    assert rel_err(g, r) <= TOL[wl.dtype]
    assert np.array_equal(g.view(np.uint32) if g.dtype == np.float32 else g, r.view(np.uint32) if r.dtype == np.float32 else r)


def test_noalloc_forward_matches_the_workspace_forward_twice_in_a_row():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    dev = torch.device("cuda:0")
    # the largest workload first (38 MiB of the 64 MiB array), then a smaller one, whose call finds the
    # first call's contents in the array
    _compare(WORKLOADS["highres"], dev)
    _compare(WORKLOADS["matching"], dev)
    # and a tiny QuadTree-A problem after both, with three levels
    _compare(WORKLOADS["tiny"], dev)


def test_noalloc_forward_rejects_a_problem_beyond_its_array():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    dev = torch.device("cuda:0")
    wl = WORKLOADS["stereo"]
    q = torch.zeros((wl.B, wl.H, wl.W, wl.heads, wl.d), dtype=torch.bfloat16, device=dev)
    out = torch.empty_like(q)
    with pytest.raises(P.QtaError) as e:
        P.forward_noalloc(q, q, q, out, levels=wl.levels, K=wl.K, variant=wl.variant, epipolar=True)
    assert e.value.status == 3
