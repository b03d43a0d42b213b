"""Benchmark: query tokens/s of one QuadTree attention layer on one MI355X.

A step is one whole forward (pyramids, coarse attention with top-K, every finer level, the fused
combination) over one batch of synthetic input that is already resident in HBM. The default
workload is the largest one, dense-prediction high-resolution self-attention (2 x 200x336 tokens,
2 heads x 32, bf16, 5 levels, K=16, QuadTree-B). Prints one JSON line with the throughput, the
finest-level kernel's HBM roofline fraction (timed with HIP events on the stream it runs on, in
algorithmic bytes and, from committed rocprofv3 counters, in measured bytes), the whole layer's
fraction of its HBM roofline, the coarse level's MFMA figures, and the CPU oracle timed on the host.

With --backward a step is one whole backward pass instead (the gradients of q, k, v and w for an
upstream gradient, the kept keys of one preceding forward held fixed), and the roofline kernel is
the finest level's backward.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--backward]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "query tokens/sec per QuadTree attention layer + % of HBM/MFMA roofline, 1 GPU"
METRIC_BWD = ("query tokens/sec per QuadTree attention layer, backward pass (gradients of q, k, v, w) + % of HBM "
              "roofline, 1 GPU")
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}      # dense MFMA peaks of MI355X per input type
COARSE_MFMA_TARGET = 0.40
PROFILES = os.path.join(ROOT, "profiles")
_CSRC = os.path.join(ROOT, "paper_2201_02767_amd", "csrc")
# every source compiled into the roofline kernel: its counters are stale once one of them changes
FINE_SRC = [os.path.join(_CSRC, f) for f in ("fine.hip", "fine_item.h", "qta_device.h", "qta_internal.h")]
BWD_SRC = [os.path.join(_CSRC, f) for f in ("backward.hip", "qta_device.h", "qta_internal.h")]
COARSE_SRC = [os.path.join(_CSRC, f) for f in ("coarse.hip", "qta_device.h", "qta_internal.h")]


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def finest_kernel_bytes(wl) -> dict:
    """Algorithmic HBM bytes of one launch of the finest-level kernel (attention at level 0 with the
    fused combination), counting every tensor once plus one gather of each sibling group's
    candidate key and value rows:
      per (batch, head):  N0*d*b (queries) + N1*K*sigma (parent selections; sigma = 4 B for B, 8 B
      for A, which also reads the scores) + N1*c*K*2*d*b (gathered key/value rows, c = 4 children
      per kept key, 2 on one-row maps) + N1*(L-1)*d*4 (the ancestors' fp32 messages, once per
      sibling group) + [B] N0*L*4 (level weights) + N0*d*b (output)."""
    from paper_2201_02767_amd.inputs import Workload  # noqa: F401  (type only)
    import paper_2201_02767_amd as P

    mB, mH = (wl.B * wl.H, 1) if wl.epipolar else (wl.B, wl.H)      # the maps the library works on
    dims = P.level_dims(mH, wl.W, wl.levels)
    n0 = dims[0][0] * dims[0][1]
    n1 = dims[1][0] * dims[1][1]
    b = 2 if wl.dtype == "bf16" else 4
    sigma = 4 if wl.variant == "B" else 8
    K1 = P.k_levels(wl.K, wl.levels)[1]       # keys each level-1 parent kept
    parts = {
        "queries": n0 * wl.d * b,
        "parent_selections": n1 * K1 * sigma,
        "gather": n1 * (2 if mH == 1 else 4) * K1 * 2 * wl.d * b,
        "ancestor_messages": n1 * (wl.levels - 1) * wl.d * 4,
        "level_weights": n0 * wl.levels * 4 if wl.variant == "B" else 0,
        "output": n0 * wl.d * b,
    }
    units = mB * wl.heads
    return {k: v * units for k, v in parts.items()}


def finest_backward_kernel_bytes(wl) -> dict:
    """Algorithmic HBM bytes of the finest level's backward step (its query pass, the counting sort
    of the kept pairs, its key pass), every tensor once, per (batch, head), with c = 4 children per
    kept key (2 on one-row maps) and M = N1*K kept (parent, key) pairs:
      query pass:  N0*d*b (q) + N0*d*b (dout) + [B with w] 4*N0*L (w) + M*sigma (parent selections)
                   + M*c*2*d*b (gathered key/value rows) + 4*N0*d (dq) + 8*N0 (statistics; A: 8*N0*K)
                   + [B with w] 4*N0*L (dw) + 4*N1*d*(L-1) (message gradients of the coarser levels,
                   one row per sibling group and level) + [A] 4*M (score gradients) + 4*M (counts)
      sort:        4*M (the pairs, grouped by key)
      key pass:    4*M (the pairs) + M*c*(2*d*b + 8) (the parents' children: q and dout rows,
                   statistics) + N1*c*2*d*b (the keys' k and v rows) + 2*4*N0*d (dk, dv)."""
    import paper_2201_02767_amd as P

    mB, mH = (wl.B * wl.H, 1) if wl.epipolar else (wl.B, wl.H)
    dims = P.level_dims(mH, wl.W, wl.levels)
    n0 = dims[0][0] * dims[0][1]
    n1 = dims[1][0] * dims[1][1]
    b = 2 if wl.dtype == "bf16" else 4
    sigma = 4 if wl.variant == "B" else 8
    K1 = P.k_levels(wl.K, wl.levels)[1]
    c = 2 if mH == 1 else 4
    d, L = wl.d, wl.levels
    B_w = wl.variant == "B"
    M = n1 * K1
    parts = {
        "queries": n0 * d * b,
        "upstream_gradient": n0 * d * b,
        "level_weights": 4 * n0 * L if B_w else 0,
        "parent_selections": M * sigma,
        "gather": M * c * 2 * d * b,
        "dq": 4 * n0 * d,
        "statistics": 8 * n0 * (1 if B_w else K1),
        "dw": 4 * n0 * L if B_w else 0,
        "message_gradients": 4 * n1 * d * (L - 1),
        "score_gradients": 0 if B_w else 4 * M,
        "counts_and_pairs": 4 * M * 3,
        "key_pass_queries": M * c * (2 * d * b + 8),
        "key_pass_keys": n1 * c * 2 * d * b,
        "dk_dv": 2 * 4 * n0 * d,
    }
    units = mB * wl.heads
    return {k: v * units for k, v in parts.items()}


def kernel_source_hash(srcs=FINE_SRC) -> str:
    h = hashlib.sha256()
    for src in srcs:
        with open(src, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, kernel: str = "fine_attn_finest", src=FINE_SRC):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it was taken on the
    current kernel source; None otherwise."""
    path = os.path.join(PROFILES, f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_sha256_16") != kernel_source_hash(src):
        return None
    return rec.get("bytes_per_launch")


def measured_mfma(workload: str):
    """The coarse kernel's MFMA counters from the committed rocprofv3 summary
    (profiles/coarse_mfma_<workload>.json), if taken on the current coarse source; None otherwise."""
    path = os.path.join(PROFILES, f"coarse_mfma_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_sha256_16") != kernel_source_hash(COARSE_SRC):
        return None
    return rec


def _level_geometry(wl):
    """Token counts per level of the maps the library works on (B*H one-row maps for epipolar
    attention), the number of such (map, head) units, storage bytes, children per kept key, K per level."""
    import paper_2201_02767_amd as P

    mB, mH = (wl.B * wl.H, 1) if wl.epipolar else (wl.B, wl.H)
    N = [h * w for h, w in P.level_dims(mH, wl.W, wl.levels)]
    b = 2 if wl.dtype == "bf16" else 4
    return N, mB * wl.heads, b, (2 if mH == 1 else 4), P.k_levels(wl.K, wl.levels)


def layer_bytes(wl) -> dict:
    """Algorithmic HBM bytes of one whole layer (every tensor streamed once, plus one gather of each
    sibling group's candidate key and value rows), per (batch, head) with b storage bytes, sigma = 4 B
    (B) or 8 B (A: index and score) per kept entry, c children per kept key, c = L-1 the coarsest level:
      pyramid  read q, k, v at level 0 and write every coarser level: (2 or 3)*(N0 + sum_{l>=1} N_l)*d*b
               (V's levels are the caller's when given);
      coarse   3*Nc*d*b + 4*Nc*d (message) + Nc*Kc*sigma (selections);
      level l  N_l*d*b (queries) + N_{l+1}*K_{l+1}*sigma (parents' selections)
               + N_{l+1}*c*K_{l+1}*2*d*b (gathered key and value rows)
               + [l >= 1] N_l*(4*d + K_l*sigma) (message, selections)
               + [l = 0] N0*d*b (output) + N1*(L-1)*4*d (ancestors' messages) + [B] 4*N0*L (w);
      position encoding (when used) sum_l N_l*d*b (V read once more at every level)."""
    N, units, b, ch, Kl = _level_geometry(wl)
    d, L = wl.d, wl.levels
    sigma = 4 if wl.variant == "B" else 8
    ntens = 2 if wl.v_given else 3
    parts = {"pyramid": ntens * sum(N) * d * b if L > 1 else 0}
    c = L - 1
    if L == 1:
        parts["coarse"] = 4 * N[0] * d * b
    else:
        parts["coarse"] = 3 * N[c] * d * b + 4 * N[c] * d + N[c] * Kl[c] * sigma
    for l in range(L - 2, -1, -1):
        x = N[l] * d * b + N[l + 1] * Kl[l + 1] * sigma + N[l + 1] * ch * Kl[l + 1] * 2 * d * b
        if l >= 1:
            x += N[l] * (4 * d + Kl[l] * sigma)
        else:
            x += N[0] * d * b + N[1] * (L - 1) * 4 * d + (4 * N[0] * L if wl.variant == "B" else 0)
        parts[f"level{l}"] = x
    if wl.pe:
        parts["position_encoding"] = sum(N) * d * b
    return {k: v * units for k, v in parts.items()}


def coarse_flops(wl) -> int:
    """QK^T and PV of the coarsest level at 2 flops per multiply-add: 4*d*Nc^2 per (batch, head)."""
    N, units, _, _, _ = _level_geometry(wl)
    return 4 * wl.d * N[-1] ** 2 * units


def host_cpu() -> dict:
    """Core count and model of the host the oracle runs on."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = None
    return {"host_cores": os.cpu_count(), "host_cores_usable": usable, "host_cpu": model}


def cpu_baseline(wl, arrays, seconds: float, backward: bool = False) -> dict:
    """The oracle as it stands, single-threaded on the host, on whole layers of the workload (its
    backward, which also runs the forward it differentiates, with --backward). ``arrays``: the
    numpy inputs the GPU run used."""
    from oracle import oracle

    q, k, v, w, vl, pw, pb, g = arrays
    if wl.epipolar:     # every row its own 1 x W map
        q, k, v = (x.reshape(wl.B * wl.H, 1, wl.W, wl.heads, wl.d) for x in (q, k, v))
        w = None if w is None else w.reshape(wl.B * wl.H, wl.W, wl.heads, wl.levels)
    if backward:
        g = g.reshape(q.shape)
    runs, t0 = 0, time.perf_counter()
    while True:
        if backward:
            oracle.backward(q, k, v, g, levels=wl.levels, K=wl.K, variant=wl.variant, dtype=wl.dtype, w=w,
                            v_levels=vl, pe_weight=pw, pe_bias=pb)
        else:
            oracle.forward(q, k, v, levels=wl.levels, K=wl.K, variant=wl.variant, dtype=wl.dtype, w=w,
                           v_levels=vl, pe_weight=pw, pe_bias=pb)
        runs += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    rec = {"value": wl.tokens * runs / el, "unit": "query tokens/s", "cores": 1, "kind": "oracle",
           "sample": f"{runs} whole {wl.name} layer {'backward pass(es)' if backward else 'forward(s)'} "
                     f"({wl.B}x{wl.H}x{wl.W}, {wl.heads}x{wl.d}, L={wl.levels}, K={wl.K}) in {el:.1f} s, "
                     "one thread (the oracle is single-threaded C, fp64)"}
    rec.update(host_cpu())
    return rec


def _time_launches(fn, n, stream, e0, e1) -> float:
    """Average microseconds per call of ``fn`` over ``n`` calls, HIP events on ``stream``."""
    import torch

    for _ in range(10):
        fn()
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(n):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / n


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="highres")
    ap.add_argument("--kernel-launches", type=int, default=500, help="launches timed for the roofline kernel")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--backward", action="store_true", help="time the backward pass instead of the forward")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run plain device copies of this many MiB (to scale HBM byte counters) and exit")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}). "
              "Each (batch, head) is an independent quadtree, so a multi-GPU run would shard batch x heads with "
              "no communication; no multi-GPU figure is produced.", file=sys.stderr)
        return 2

    import torch

    if args.calibrate_copy_mib:
        n = args.calibrate_copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"bench: 5 device copies of {n} bytes (each reads {n} and writes {n} bytes)")
        return 0

    import paper_2201_02767_amd as P
    from paper_2201_02767_amd.inputs import WORKLOADS, make_dout, make_level_weights, make_pe, make_qkv, make_v_levels

    if args.workload not in WORKLOADS:
        print(f"unknown workload {args.workload}; choose from {sorted(WORKLOADS)}", file=sys.stderr)
        return 2
    wl = WORKLOADS[args.workload]
    log(f"bench: generating the {wl.name} inputs")
    qn, kn, vn = make_qkv(wl)
    wn = make_level_weights(wl) if wl.variant == "B" else None
    vln = make_v_levels(wl) if wl.v_given else None
    pwn, pbn = make_pe(wl) if wl.pe else (None, None)
    gn = make_dout(wl) if args.backward else None

    dev = torch.device("cuda:0")
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    q, k, v = (torch.from_numpy(x).to(dev).to(tdt).contiguous() for x in (qn, kn, vn))
    w = torch.from_numpy(wn).to(dev) if wn is not None else None
    vl = None
    if wl.v_given:
        vl = [None] + [torch.from_numpy(x).to(dev).to(tdt).contiguous() for x in vln[1:]]
    pw = pb = None
    if wl.pe:
        pw, pb = torch.from_numpy(pwn).to(dev), torch.from_numpy(pbn).to(dev)
    plan = P.Plan(wl.B, wl.H, wl.W, wl.heads, wl.d, levels=wl.levels, K=wl.K, variant=wl.variant, dtype=tdt,
                  device=dev, v_supplied=wl.v_given, pe=wl.pe, epipolar=wl.epipolar)
    step = plan.prepare(q, k, v, w, v_levels=vl, pe_weight=pw, pe_bias=pb)
    log(f"bench: {wl} on {torch.cuda.get_device_name(0)}")
    if args.backward:
        g = torch.from_numpy(gn).to(dev).to(tdt).contiguous()
        step()                                   # the forward whose kept keys the backward holds fixed
        step = plan.prepare_backward(q, k, v, g, w, v_levels=vl, pe_weight=pw, pe_bias=pb)
        log("bench: timing the backward pass")

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_per_step = e0.elapsed_time(e1) / args.steps
    value = wl.tokens / (ms_per_step / 1e3)
    log(f"bench: {args.steps} steps, {ms_per_step * 1e3:.2f} us/step (events), wall {wall * 1e6 / args.steps:.2f} "
        f"us/step, {value:.4g} query tokens/s")

    # the dominant kernel alone, on the same stream, on the selections the forward left behind
    roof = None
    if wl.levels >= 2 and args.backward:
        k_us = _time_launches(plan.prepare_backward(q, k, v, g, w, finest_only=True, v_levels=vl, pe_weight=pw,
                                                    pe_bias=pb), args.kernel_launches, stream, e0, e1)
        parts = finest_backward_kernel_bytes(wl)
        algo = sum(parts.values())
        achieved = algo / (k_us * 1e-6) / 1e9
        traffic = measured_traffic(wl.name, "bwd_level_finest", BWD_SRC)
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": "finest-level backward step (query pass, counting sort, key pass; 6 launches)",
                "kernel_us": round(k_us, 3),
                "algorithmic_bytes": algo}
        log(f"bench: finest-level backward step {k_us:.2f} us/launch, {algo / 1e6:.1f} MB algorithmic -> "
            f"{achieved:.0f} GB/s ({100 * achieved / HBM_PEAK_GBS:.1f}% of {HBM_PEAK_GBS:.0f})")
    elif wl.levels >= 2:
        k_us = _time_launches(plan.prepare_finest(q, k, v, w), args.kernel_launches, stream, e0, e1)
        parts = finest_kernel_bytes(wl)
        algo = sum(parts.values())
        achieved = algo / (k_us * 1e-6) / 1e9
        traffic = measured_traffic(wl.name)
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": "fine_attn_kernel (finest level, fused combine)", "kernel_us": round(k_us, 3),
                "algorithmic_bytes": algo}
        if traffic:
            # the same launch time against the bytes the counters saw cross the L2 (HBM or MALL)
            roof["traffic_frac"] = round(traffic / (k_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)
        log(f"bench: finest-level kernel {k_us:.2f} us/launch, {algo / 1e6:.1f} MB algorithmic -> "
            f"{achieved:.0f} GB/s ({100 * achieved / HBM_PEAK_GBS:.1f}% of {HBM_PEAK_GBS:.0f})"
            + (f"; counters {traffic / 1e6:.1f} MB -> {100 * roof['traffic_frac']:.1f}%" if traffic else ""))

        # the whole layer against its own HBM roofline (every tensor once, one gather per sibling group)
        lparts = layer_bytes(wl)
        lbytes = sum(lparts.values())
        lach = lbytes / (ms_per_step * 1e-3) / 1e9
        roof["layer"] = {"bound": "hbm", "algorithmic_bytes": lbytes, "us": round(ms_per_step * 1e3, 3),
                         "achieved": round(lach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": round(lach / HBM_PEAK_GBS, 4),
                         "roofline_us": round(lbytes / (HBM_PEAK_GBS * 1e9) * 1e6, 2)}
        log(f"bench: whole layer {lbytes / 1e6:.1f} MB algorithmic in {ms_per_step * 1e3:.2f} us -> {lach:.0f} GB/s "
            f"({100 * lach / HBM_PEAK_GBS:.1f}% of {HBM_PEAK_GBS:.0f})")

        # the coarsest level on MFMA: device-wide flop rate, and the MFMA-busy share of the CUs it occupies
        if not wl.v_given:
            c_us = _time_launches(plan.prepare_coarse(), args.kernel_launches, stream, e0, e1)
            fl = coarse_flops(wl)
            tf = fl / (c_us * 1e-6) / 1e12
            peak = MFMA_PEAK_TFLOPS[wl.dtype]
            coarse = {"kernel": "qta_coarse_attn stage call: coarse_attn_kernel (coarsest level with top-K), then "
                                "the ordering pass over its selection rows", "kernel_us": round(c_us, 3),
                      "flops": fl, "achieved": round(tf, 3), "peak": peak, "unit": "TFLOP/s",
                      "frac_device": round(tf / peak, 6), "target": COARSE_MFMA_TARGET,
                      "compared_with_target": "mfma_busy_frac_occupied"}
            mf = measured_mfma(wl.name)
            coarse["mfma_busy_frac_occupied"] = mf.get("mfma_busy_frac_occupied") if mf else None
            coarse["mfma_busy_frac_device"] = mf.get("mfma_busy_frac_device") if mf else None
            roof["coarse"] = coarse
            log(f"bench: coarse level {c_us:.2f} us/launch, {fl / 1e6:.1f} MFLOP -> {tf:.2f} TFLOP/s "
                f"({100 * tf / peak:.3f}% of {peak:.0f}); MFMA busy on occupied CUs "
                f"{coarse['mfma_busy_frac_occupied']}")

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, (qn, kn, vn, wn, vln, pwn, pbn, gn), args.cpu_seconds, args.backward)
        log(f"bench: oracle {cpu['value']:.4g} query tokens/s ({cpu['sample']}; host {cpu['host_cores']} cores, "
            f"{cpu['host_cpu']})")

    rec = {
        "metric": METRIC_BWD if args.backward else METRIC, "value": round(value, 1), "unit": "query tokens/s",
        "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32" if wl.dtype == "f32" else "bf16", "data": "synthetic",
        "config": {"workload": wl.name, "B": wl.B, "H": wl.H, "W": wl.W, "heads": wl.heads, "d": wl.d,
                   "levels": wl.levels, "K": wl.K if isinstance(wl.K, int) else list(wl.K)[1:],
                   "v_levels": "given" if wl.v_given else "pooled", "position_encoding": wl.pe,
                   "attention": "epipolar rows" if wl.epipolar else "2-D",
                   "pass": "backward" if args.backward else "forward",
                   "variant": wl.variant, "global_batch": wl.B,
                   "seq_len": wl.H * wl.W, "parallelism": "none (1 GPU)"},
        "roofline": roof, "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
