#!/usr/bin/env python3
"""Benchmark of the hot path on one MI355X: jagged dynamic-mask HSTU attention with the
gate + Group-LayerNorm that follows it (MTGR, arXiv 2505.18654, Sec. 4.2), fwd + bwd.

One step = plan (tile summaries + work list) -> attention fwd -> gate + Group-LN fwd ->
Group-LN bwd -> attention bwd (dQ kernel, then dK/dV kernel), on one synthetic batch of
the MTGR-large shape (64 users, 16 user tokens, lognormal history, 8 heads x 128) whose
inputs are resident in HBM before the timed region.  Prints ONE JSON line.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--workload mtgr_large]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16 = 2.5e15        # MI355X dense bf16 MFMA, FLOP/s
PEAK_FP32 = 157.3e12      # MI355X fp32 vector, FLOP/s
PEAK_HBM = 8.0e12         # MI355X HBM3E, B/s
METRIC = "jagged HSTU attn fwd+bwd tokens/s and TFLOP/s (% bf16 MFMA peak), 1 MI355X"
CSRC = os.path.join(ROOT, "paper_2505_18654_amd", "csrc")


def visible_pairs(layout) -> np.ndarray:
    """Mask-visible (i, j) pairs per user, counted segment by segment (Sec. 4.2 rules)."""
    out = np.zeros(layout.num_users, np.int64)
    for b in range(layout.num_users):
        sl = layout.user_slice(b)
        seg, ts = layout.seg[sl], layout.ts[sl].astype(np.int64)
        n = len(seg)
        n_s = int(np.sum(seg <= 1))
        rt = np.sort(ts[seg == 2])
        rt_q = ts[seg == 2]
        cand = ts[seg == 3]
        earlier_rt = np.searchsorted(rt, rt_q, side="left").sum() + np.searchsorted(rt, cand, side="left").sum()
        dyn = n - n_s
        out[b] = n_s * n_s + dyn * n_s + earlier_rt + dyn
    return out


def candidate_pairs(layout) -> np.ndarray:
    """Mask-visible pairs whose query is a candidate, per user: every static key, the RT keys
    strictly earlier than the candidate, and the candidate itself (Sec. 4.2 rules)."""
    out = np.zeros(layout.num_users, np.int64)
    for b in range(layout.num_users):
        sl = layout.user_slice(b)
        seg, ts = layout.seg[sl], layout.ts[sl].astype(np.int64)
        n_s = int(np.sum(seg <= 1))
        rt = np.sort(ts[seg == 2])
        cand = ts[seg == 3]
        out[b] = len(cand) * (n_s + 1) + int(np.searchsorted(rt, cand, side="left").sum())
    return out


# The sources each kernel is compiled from (its own file plus the shared device headers): a
# counter figure stays valid while none of them changes.
KERNEL_SOURCES = {
    "attn_fwd_bf16_kernel": ["attn_fwd.hip"],
    "attn_bwd_dkdv_bf16_kernel": ["attn_bwd_dkdv.hip", "attn_bwd_common.h"],
    "attn_bwd_dq_ds_bf16_kernel": ["attn_bwd_dqds.hip", "attn_bwd_common.h"],
    "gln_fwd_kernel": ["group_ln.hip"],
    "gln_bwd_kernel": ["group_ln.hip"],
    "gemm_bf16_kernel": ["gemm.hip"],
}
SHARED_SOURCES = ["mtgr_device.h", "mtgr_internal.h"]


def source_hash(kernel: str) -> str:
    h = hashlib.sha256()
    for name in sorted(KERNEL_SOURCES[kernel] + SHARED_SOURCES):
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str, field: str = "bytes_per_launch"):
    """HBM bytes per launch (or another counter-derived figure of the kernel, such as its
    effective shader clock) from the committed rocprofv3 counter runs, if they were taken on the
    current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    entry = data.get(f"{kernel}@{workload}")
    if not entry or entry.get("source_hash") != source_hash(kernel):
        return None
    return entry.get(field)


def cpu_baseline(layout, budget_s: float):
    """The oracle (plain fp64 C, OpenMP) on a bounded sample of the same batch: the users
    with the smallest visible-pair count first, until about `budget_s` seconds of work."""
    import oracle
    from synth import make_values
    pairs = visible_pairs(layout)
    H, dh = layout.spec.heads, layout.spec.head_dim
    order = list(np.argsort(pairs, kind="stable"))
    # calibrate the oracle's pair rate on one small user
    probe = [int(order[len(order) // 4])]
    t_probe = _oracle_step(layout, probe)
    rate = max(pairs[probe[0]] * H / max(t_probe, 1e-6), 1.0)      # (pair * head) / s
    chosen, work = [], 0.0
    for b in order[::-1]:                                             # mix: largest first
        cost = pairs[b] * H / rate
        if work + cost > budget_s and chosen:
            continue
        chosen.append(int(b))
        work += cost
        if work >= 0.6 * budget_s:
            break
    t = _oracle_step(layout, chosen)
    tokens = int(sum(layout.offsets[b + 1] - layout.offsets[b] for b in chosen))
    threads = int(os.environ.get("OMP_NUM_THREADS", 0)) or len(os.sched_getaffinity(0))
    return {"value": tokens / t, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "cpus_visible": len(os.sched_getaffinity(0)),
            "sample": f"{len(chosen)} of {layout.num_users} users ({tokens} tokens, "
                      f"{int(pairs[chosen].sum())} visible pairs x {H} heads), same path fwd+bwd, "
                      f"fp64, {t:.1f} s",
            "seconds": round(t, 2)}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


NOMINAL_MHZ = 2400.0      # the clock at which the published MI355X peaks are quoted


def shader_clock_mhz(seconds: float = 0.05) -> float:
    """Shader clock while every CU's matrix cores are busy (mtgr_debug_clock_probe: a back-to-
    back MFMA loop per workgroup, shader-clock cycles over constant-rate ticks), median over
    the workgroups.  Run right after the timed region, on a GPU at its working temperature."""
    import torch
    from paper_2505_18654_amd import hstu
    blocks = torch.cuda.get_device_properties(0).multi_processor_count
    out = torch.zeros(3 * blocks, dtype=torch.int64, device="cuda")
    iters = max(int(seconds * NOMINAL_MHZ * 1e6 / 128), 1)        # 4 MFMAs of 32 cycles each
    khz = hstu.mtgr_debug_clock_probe(iters, blocks, out)
    torch.cuda.synchronize()
    o = out.view(blocks, 3).cpu().numpy().astype(np.float64)
    return float(np.median(o[:, 0] / o[:, 1] * khz / 1e3))


def _oracle_step(layout, users) -> float:
    import oracle
    from synth import make_values
    sub = layout.subset(users)
    vals = make_values(sub)
    H, dh = layout.spec.heads, layout.spec.head_dim
    T = sub.total_tokens
    t0 = time.perf_counter()
    o = oracle.attn_fwd(sub.offsets, sub.seg, sub.ts, vals["q"], vals["k"], vals["v"], vals["rab"])
    x = o.reshape(T, H * dh)
    oracle.gln_fwd(x, vals["u"], sub.seg, vals["gamma"], vals["beta"])
    dx, _, _, _ = oracle.gln_bwd(x, vals["u"], sub.seg, vals["gamma"], vals["dy"])
    oracle.attn_bwd(sub.offsets, sub.seg, sub.ts, vals["q"], vals["k"], vals["v"], dx.reshape(T, H, dh),
                    vals["rab"])
    return time.perf_counter() - t0


def sampled_parity(layout, inp, res, users):
    """Forward attention output of a few users against the oracle, per user:
    literal = max |gpu - ref| / rms_user(ref) (the stated bar), and storage_adjusted = the
    same after subtracting each reference value's bf16 storage rounding (half an ulp)."""
    import oracle
    from synth import make_values
    sub = layout.subset(users)
    vals = make_values(sub, tensors=("q", "k", "v"))
    ref = oracle.attn_fwd(sub.offsets, sub.seg, sub.ts, vals["q"], vals["k"], vals["v"], inp["rab_np"])
    rows = np.concatenate([np.arange(layout.offsets[b], layout.offsets[b + 1]) for b in users])
    got = res["o"].float().cpu().numpy()[rows]
    lit, adj, row = 0.0, 0.0, 0
    for b in users:
        n = int(layout.offsets[b + 1] - layout.offsets[b])
        g, w = got[row:row + n], ref[row:row + n]
        row += n
        rms = float(np.sqrt(np.mean(w ** 2)))
        if not rms:
            continue
        diff = np.abs(g - w)
        half_ulp = np.where(w != 0, np.ldexp(1.0, np.frexp(np.abs(w))[1] - 9), 0.0)
        lit = max(lit, float(diff.max()) / rms)
        adj = max(adj, float(np.maximum(diff - half_ulp, 0.0).max()) / rms)
    return lit, adj


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="mtgr_large",
                    choices=["tiny", "small", "mtgr_small", "mtgr_large", "serving"])
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the HIP-graph replay of the step after the timed region")
    ap.add_argument("--layer", action="store_true",
                    help="time one whole encoder layer (Group-LN, projection GEMM, bias + SiLU, "
                         "attention, gate + Group-LN, output GEMM; forward and backward) instead "
                         "of the attention path, and print its own JSON line")
    ap.add_argument("--no-gemm-detail", action="store_true",
                    help="with --layer: skip timing each dense product on its own after the timed "
                         "region (for kernel traces of the layer steps alone)")
    ap.add_argument("--embedding", action="store_true",
                    help="time the dynamic embedding table instead (de-duplication, lookup with "
                         "insertion, gather and sparse SGD of the workload's sparse IDs) and print "
                         "its own JSON line")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB three times (scale of the "
                         "FETCH_SIZE / WRITE_SIZE counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: measures one GPU only; --gpus {args.gpus} is not supported "
              "(users are independent, so the path would shard by user across GPUs with no "
              "exchange in the forward pass and one small all-reduce of the parameter gradients)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    if args.calibrate_copy:
        n = args.calibrate_copy * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n * 4}), flush=True)
        return
    from paper_2505_18654_amd import ops
    from synth import make_layout
    from synth.torch_inputs import device_inputs

    layout = make_layout(args.workload)
    spec = layout.spec
    if args.layer:
        return bench_layer(args, layout)
    if args.embedding:
        return bench_embedding(args, layout)
    H, dh = spec.heads, spec.head_dim
    d = H * dh
    T = layout.total_tokens
    lens = np.diff(layout.offsets)
    check_users = sorted({int(np.argmin(lens)), int(np.argsort(lens)[len(lens) // 2])})
    fwd_only = spec.fwd_only
    tensors = ("q", "k", "v", "u") if fwd_only else ("q", "k", "v", "u", "dy")
    inp = device_inputs(layout, "cuda", exact_users=check_users, tensors=tensors)
    jag = ops.Jagged(inp["offsets"], inp["seg"], inp["ts"], inp["max_seqlen"])
    q, k, v, u = inp["q"], inp["k"], inp["v"], inp["u"]
    rab, gamma, beta, seg = inp["rab"], inp["gamma"], inp["beta"], inp["seg"]

    # preallocated outputs and workspace: nothing is allocated inside the timed region
    o = torch.empty_like(q)
    y = torch.empty((T, d), dtype=q.dtype, device="cuda")
    mean = torch.empty(T, dtype=torch.float32, device="cuda")
    rstd = torch.empty(T, dtype=torch.float32, device="cuda")
    dx = torch.empty((T, d), dtype=q.dtype, device="cuda")
    du = torch.empty((T, d), dtype=q.dtype, device="cuda")
    dg = torch.empty_like(gamma)
    db = torch.empty_like(gamma)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    drab = torch.empty_like(rab) if rab is not None else None
    ws = ops.workspace_for(ops.attn_problem(jag, q, k, v, o, rab), "cuda", backward=not fwd_only)
    gws = ops.gln_workspace(y, gamma.shape[0])

    # backward: on the matrix-core path the dK/dV kernel stores dS, then dQ is formed from it
    # (two calls, timed apart); on the vector path (fp32, or bf16 with head_dim 16) the two
    # kernels each recompute S and dP
    mfma_path = spec.dtype == "bf16" and dh in (32, 64, 128)
    part_dkdv, part_dq = ("dkdv_keep_ds", "dq_from_ds") if mfma_path else ("dkdv", "dq")
    stages = ["plan", "attn_fwd", "gln_fwd"] + ([] if fwd_only else ["gln_bwd", "attn_bwd_dkdv", "attn_bwd_dq"])

    def run(name):
        if name == "plan":
            ops.attn_plan(q, jag, workspace=ws, rab=rab)
        elif name == "attn_fwd":
            ops.attn_fwd(q, k, v, jag, rab, out=o, workspace=ws, planned=True)
        elif name == "gln_fwd":
            ops.gln_fwd(o.view(T, d), u, seg, gamma, beta, y=y, stats=(mean, rstd))
        elif name == "gln_bwd":
            ops.gln_bwd(inp["dy"], o.view(T, d), u, seg, gamma, mean, rstd, grads=(dx, du, dg, db),
                        workspace=gws)
        elif name == "attn_bwd_dkdv":
            ops.attn_bwd(q, k, v, dx.view(T, H, dh), jag, rab, grads=(dq, dk, dv, drab), workspace=ws,
                         planned=True, parts=part_dkdv)
        elif name == "attn_bwd_dq":
            ops.attn_bwd(q, k, v, dx.view(T, H, dh), jag, rab, grads=(dq, dk, dv, drab), workspace=ws,
                         planned=True, parts=part_dq)

    kflops_stages = ("attn_fwd", "attn_bwd_dkdv", "attn_bwd_dq")

    def timed_steps(n, bracket):
        # n steps; the stages in `bracket` are each bracketed by a pair of events on the launching
        # stream.  An event pair between two kernels leaves a gap of a few microseconds, so the
        # timed steps bracket only the dominant attention kernel and the other stages are timed in
        # a pass of their own after the timed region.
        ev = {s: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in range(n)] for s in bracket}
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(n):
            for s in stages:
                if s in ev:
                    ev[s][i][0].record()
                run(s)
                if s in ev:
                    ev[s][i][1].record()
        torch.cuda.synchronize()
        return time.perf_counter() - t0, {s: float(np.mean([a.elapsed_time(b) for a, b in ev[s]])) for s in ev}

    # warm-up steps (their stage events pick the dominant attention kernel: the slowest one)
    _, warm_ms = timed_steps(args.warmup, stages) if args.warmup else (0.0, {})
    if not warm_ms:
        _, warm_ms = timed_steps(1, stages)
    dom = max((s for s in kflops_stages if s in warm_ms), key=lambda s: warm_ms[s])
    elapsed, dom_ms = timed_steps(args.steps, (dom,))
    _, stage_ms = timed_steps(args.steps, stages)     # every stage, after the timed region
    stage_ms[dom] = dom_ms[dom]                       # the dominant kernel: from the timed steps

    pairs = int(visible_pairs(layout).sum())
    f_fwd = 4.0 * dh * H * pairs
    f_bwd = 0.0 if fwd_only else 8.0 * dh * H * pairs
    ms_step = elapsed * 1e3 / args.steps
    tflops = (f_fwd + f_bwd) / (ms_step * 1e-3) / 1e12

    # dominant kernel and its roofline (algorithmic flops per launch / event-timed duration)
    # algorithmic split of F_bwd = 8 dh per pair: the dK/dV kernel forms dP, dV and dK (6 dh),
    # the dQ kernel dQ (2 dh); recomputation of S is not counted
    kflops = {"attn_fwd": f_fwd, "attn_bwd_dkdv": f_bwd * 3 / 4, "attn_bwd_dq": f_bwd / 4}
    if mfma_path:
        kname = {"attn_fwd": "attn_fwd_bf16_kernel", "attn_bwd_dq": "attn_bwd_dq_ds_bf16_kernel",
                 "attn_bwd_dkdv": "attn_bwd_dkdv_bf16_kernel"}
        bound, peak = "mfma", PEAK_BF16
    else:   # fp32 vector FMAs (the published fp32 vector peak: 256 CUs x 128 FMA lanes x 2 x 2.4 GHz)
        kname = {"attn_fwd": "attn_fwd_vec_kernel", "attn_bwd_dq": "attn_bwd_dq_vec_kernel",
                 "attn_bwd_dkdv": "attn_bwd_dkdv_vec_kernel"}
        bound, peak = "alu", PEAK_FP32
    achieved = kflops[dom] / (stage_ms[dom] * 1e-3)
    mhz = shader_clock_mhz()
    peak_clk = peak * mhz / NOMINAL_MHZ
    roofline = {"bound": bound, "kernel": kname[dom], "achieved": achieved / 1e12, "peak": peak / 1e12,
                "unit": "TFLOP/s", "frac": achieved / peak,
                "traffic": measured_traffic(kname[dom], args.workload) if kname[dom] in KERNEL_SOURCES else None,
                "peak_at_measured_clock": peak_clk / 1e12, "frac_at_measured_clock": achieved / peak_clk}
    kmhz = measured_traffic(kname[dom], args.workload, "clock_mhz") if kname[dom] in KERNEL_SOURCES else None
    if kmhz:
        roofline["frac_at_kernel_clock"] = achieved / (peak * kmhz / NOMINAL_MHZ)
    clock = {"measured_mhz": round(mhz, 1), "nominal_mhz": NOMINAL_MHZ,
             "how": "median shader clock over all CUs during a back-to-back MFMA loop run right after "
                    "the timed region (mtgr_debug_clock_probe)",
             "dominant_kernel_mhz": kmhz,
             "dominant_kernel_how": "GRBM_GUI_ACTIVE / 8 over the kernel's dispatch duration in the committed "
                                    "counter run on the same sources (profiles/traffic.json), or null"}
    gln_bytes = T * (3 * d * 2 + 8) + (0 if fwd_only else T * (5 * d * 2 + 8))
    gln_ms = stage_ms["gln_fwd"] + stage_ms.get("gln_bwd", 0.0)

    # The same step captured once in a HIP graph and replayed (after the timed region; the
    # library allocates, synchronises and copies nothing on this path, so a caller can record
    # it): what a graph-capturing caller saves in launch overhead, largest on the small batches.
    graph = None if args.no_graph else graph_replay(lambda: [run(s) for s in stages], args.steps, T)

    res = {"o": o}
    err_lit, err_adj = sampled_parity(layout, inp, res, check_users)

    # Serving: the candidate rows alone (one pass per user scoring all of its candidates),
    # timed apart from the step above; reported as an extra field, not as `value`.
    cand_rows = None
    if fwd_only:
        o_c = torch.empty_like(q)
        for _ in range(max(args.warmup, 1)):
            ops.attn_fwd(q, k, v, jag, rab, out=o_c, workspace=ws, planned=True, cand_rows=True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            ops.attn_fwd(q, k, v, jag, rab, out=o_c, workspace=ws, planned=True, cand_rows=True)
        e1.record()
        torch.cuda.synchronize()
        ms_c = e0.elapsed_time(e1) / args.steps
        n_cand = int(np.sum(layout.seg == 3))
        cand_pairs = int(candidate_pairs(layout).sum())
        f_cand = 4.0 * dh * H * cand_pairs
        cand_rows = {"attn_fwd_cand_rows_ms": ms_c, "candidates": n_cand,
                     "candidates_per_s": n_cand / (ms_c * 1e-3),
                     "candidate_pairs": cand_pairs,
                     "full_attn_fwd_ms": stage_ms["attn_fwd"]}
        # The user side (U | S | R) held in a cache across requests: a request brings only its
        # candidates (plan of the request included in every timed call; the cache's plan is
        # built once, when the cache is filled).
        side = np.flatnonzero(layout.seg != 3)
        cand = np.flatnonzero(layout.seg == 3)
        per_user = lambda m: np.concatenate([[0], np.cumsum([np.sum(m[layout.user_slice(b)])
                                                              for b in range(layout.num_users)])])
        jag_s = ops.Jagged.from_host(per_user(layout.seg != 3), layout.seg[side], layout.ts[side])
        jag_c = ops.Jagged.from_host(per_user(layout.seg == 3), layout.seg[cand], layout.ts[cand])
        i_s, i_c = torch.from_numpy(side).cuda(), torch.from_numpy(cand).cuda()
        cache = ops.user_cache(k[i_s].contiguous(), v[i_s].contiguous(), jag_s)
        qc, kc, vc = q[i_c].contiguous(), k[i_c].contiguous(), v[i_c].contiguous()
        o_k = torch.empty_like(qc)
        ws_k = ops.workspace_for(ops.attn_problem(jag_c, qc, kc, vc, o_k, rab), "cuda")
        for _ in range(max(args.warmup, 1)):
            ops.attn_fwd_cached(qc, kc, vc, jag_c, cache, rab, out=o_k, workspace=ws_k)
        e0.record()
        for _ in range(args.steps):
            ops.attn_fwd_cached(qc, kc, vc, jag_c, cache, rab, out=o_k, workspace=ws_k)
        e1.record()
        torch.cuda.synchronize()
        ms_k = e0.elapsed_time(e1) / args.steps
        ref_c = o_c[i_c].float()
        diff = float((o_k.float() - ref_c).abs().max() / ref_c.pow(2).mean().sqrt())
        cand_rows["cached_user_side"] = {
            "attn_fwd_cached_ms": ms_k, "candidates_per_s": n_cand / (ms_k * 1e-3),
            "tflops_candidate_pairs": f_cand / (ms_k * 1e-3) / 1e12,
            "frac_bf16_peak": f_cand / (ms_k * 1e-3) / PEAK_BF16,
            "max_abs_diff_vs_candidate_rows_over_rms": diff}
        cand_rows["tflops_candidate_pairs"] = f_cand / (ms_c * 1e-3) / 1e12
        cand_rows["frac_bf16_peak"] = f_cand / (ms_c * 1e-3) / PEAK_BF16

    line = {
        "metric": METRIC,
        "value": T * args.steps / elapsed,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if spec.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "users": layout.num_users, "tokens": T,
                   "max_seqlen": layout.max_seqlen, "heads": H, "head_dim": dh, "d": d,
                   "rab_buckets": spec.rab_buckets, "pass": "fwd" if fwd_only else "fwd+bwd"},
        "tflops": tflops,
        "pct_bf16_peak": 100.0 * tflops * 1e12 / PEAK_BF16,
        "pct_of_path_peak": 100.0 * tflops * 1e12 / peak,
        "visible_pairs": pairs,
        "stage_ms": {s: round(v, 4) for s, v in stage_ms.items()},
        "stage_ms_how": f"HIP events around each stage; {dom} in the timed steps, the others in a pass of "
                        f"the same number of steps after them",
        "gln": {"bound": "hbm", "achieved_GBps": gln_bytes / (gln_ms * 1e-3) / 1e9, "peak_GBps": PEAK_HBM / 1e9},
        "roofline": roofline,
        "clock": clock,
        "parity_sampled_fwd": {"users": check_users, "max_err_over_rms": err_lit,
                               "max_err_over_rms_storage_adjusted": err_adj},
    }
    if graph is not None:
        line["graph_replay"] = graph
    if cand_rows is not None:
        line["serving_cand_rows"] = cand_rows
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(layout, args.cpu_seconds)
    print(json.dumps(line), flush=True)


def graph_replay(step, steps: int, tokens: int) -> dict:
    """The step captured once in a HIP graph (after a warm-up on a side stream) and replayed
    `steps` times, HIP events around the replays.  Reported, never fatal: a capture error is
    returned as a string."""
    import torch
    try:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        return {"ms_per_step": ms, "tokens_per_s": tokens / (ms * 1e-3),
                "how": "the timed step's stages captured once in a HIP graph, replayed `steps` times "
                       "after the timed region (HIP events around the replays)"}
    except RuntimeError as e:
        torch.cuda.synchronize()
        return {"error": str(e)[:200]}


def bench_layer(args, layout):
    """One encoder layer (Sec. 4.2) forward + backward on the workload's batch: synthetic
    bf16 input and seeded parameters; every step, the dense products included, runs in the
    library's kernels.  After the timed region each product is timed on its own (HIP events on
    the stream it runs on) against the dense bf16 MFMA peak."""
    import torch
    from paper_2505_18654_amd import layer, ops
    spec = layout.spec
    H, dh = spec.heads, spec.head_dim
    d, T = H * dh, layout.total_tokens
    G = 4
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    rnd = lambda *shape, scale=1.0: torch.randn(*shape, generator=g, device="cuda").mul_(scale)
    x = rnd(T, d).bfloat16()
    dxo = rnd(T, d).bfloat16()
    P = layer.LayerParams(1 + rnd(G, d, scale=0.1), rnd(G, d, scale=0.1), rnd(d, 4 * d, scale=d ** -0.5).bfloat16(),
                          rnd(4 * d, scale=0.1), 1 + rnd(G, d, scale=0.1), rnd(G, d, scale=0.1),
                          rnd(d, d, scale=d ** -0.5).bfloat16(), rnd(d, scale=0.1))
    jag = ops.Jagged.from_host(layout.offsets, layout.seg, layout.ts)
    q_like = torch.empty((T, H, dh), dtype=torch.bfloat16, device="cuda")
    ws = ops.attn_plan(q_like, jag, backward=True)
    fwd_only = spec.fwd_only

    def step():
        out, ctx = layer.layer_fwd(x, jag, P, H, workspace=ws, planned=True)
        if not fwd_only:
            layer.layer_bwd(dxo, ctx, jag, P, H, workspace=ws, planned=True)
        return out

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / args.steps
    pairs = int(visible_pairs(layout).sum())
    f_attn = (4.0 if fwd_only else 12.0) * dh * H * pairs
    f_gemm = (1 if fwd_only else 3) * 2.0 * T * d * 5 * d      # [d, 4d] and [d, d] products
    line = {"metric": "MTGR encoder layer fwd+bwd tokens/s, 1 MI355X", "value": T * args.steps / elapsed,
            "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": ms, "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": args.workload, "tokens": T, "heads": H, "head_dim": dh, "d": d,
                       "pass": "fwd" if fwd_only else "fwd+bwd", "layer": True},
            "tflops": (f_attn + f_gemm) / (ms * 1e-3) / 1e12,
            "flop_split": {"attention": f_attn, "gemm": f_gemm}}
    if not args.no_gemm_detail:
        line["gemm"] = layer_gemm_times(x, dxo, P, fwd_only)
        line["gemm_ms"] = sum(v["ms"] for v in line["gemm"].values())
    print(json.dumps(line), flush=True)


def layer_gemm_times(x, dxo, P, fwd_only, reps=20):
    """Each dense product of the layer timed alone: ms per call, TFLOP/s and the fraction of
    the 2.5 PFLOP/s dense bf16 MFMA peak."""
    import torch
    from paper_2505_18654_amd import ops
    T, d = x.shape
    h = torch.empty((T, 4 * d), dtype=torch.bfloat16, device="cuda")
    a = torch.empty_like(h)
    y = torch.empty_like(x)
    b_in = torch.empty(4 * d, device="cuda")
    b_out = torch.empty(d, device="cuda")
    ws = torch.empty(max(ops.hstu.mtgr_gemm_workspace_size(ops.hstu.MTGR_GEMM_TN, d, 4 * d, T), 256),
                     dtype=torch.uint8, device="cuda")
    cases = {"proj_fwd_nn_bias_silu": ((T, 4 * d, d), lambda: ops.gemm(y, P.w_in, "nn", out=h, bias=P.b_in,
                                                                          silu_out=a)),
             "out_fwd_nn_bias_residual": ((T, d, d), lambda: ops.gemm(y, P.w_out, "nn", bias=P.b_out, residual=x))}
    if not fwd_only:
        cases.update({
            "out_dgrad_nt": ((T, d, d), lambda: ops.gemm(dxo, P.w_out, "nt")),
            "out_wgrad_tn_colsum": ((d, d, T), lambda: ops.gemm(y, dxo, "tn", colsum=b_out, workspace=ws)),
            "proj_wgrad_tn_colsum": ((d, 4 * d, T), lambda: ops.gemm(y, a, "tn", colsum=b_in, workspace=ws)),
            "proj_dgrad_nt": ((T, d, 4 * d), lambda: ops.gemm(a, P.w_in, "nt")),
        })
    out = {}
    for name, ((M, N, K), fn) in cases.items():
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        tf = 2.0 * M * N * K / (ms * 1e-3) / 1e12
        out[name] = {"M": M, "N": N, "K": K, "ms": ms, "tflops": tf, "frac": tf / 2500.0}
    return out


def bench_embedding(args, layout):
    """Sparse-ID side of a training step on the workload's batch: every token carries
    EMB_FEATURES sparse IDs drawn Zipf(1.05) over 10^8 IDs (seeded, synthetic); a step is
    dedup + lookup with insertion + gather + SGD of those IDs on a bf16 table of dim 64."""
    import torch
    from paper_2505_18654_amd.embedding import DynamicEmbedding
    EMB_FEATURES, DIM, ROWS = 8, 64, 1 << 24
    T = layout.total_tokens
    n = T * EMB_FEATURES
    rng = np.random.default_rng(17)
    batches = []
    for i in range(4):   # distinct batches, cycled
        base = rng.zipf(1.05, n) % 100_000_000
        ids = (base.astype(np.uint64) * np.uint64(0x9E3779B97F4A7C15)).view(np.int64)
        batches.append(torch.from_numpy(ids).cuda())
    table = DynamicEmbedding(ROWS, DIM, dtype=torch.bfloat16)
    grad = torch.randn(n, DIM, device="cuda").bfloat16()
    now = [0]

    def step(i):
        now[0] += 1
        out, b = table.lookup(batches[i % len(batches)], now=now[0])
        table.sgd(b, grad, 1e-3)
        return b

    for i in range(max(args.warmup, len(batches))):
        b = step(i)
    torch.cuda.synchronize()
    nu = int(b.num_unique.item())
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for i in range(args.steps):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / args.steps
    st = table.stats()
    # gather alone, for its HBM roofline: reads and writes n rows of DIM bf16
    _, b = table.lookup(batches[0], now=now[0] + 1, gather=False)
    out = torch.empty(n, DIM, dtype=torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    g0.record()
    for _ in range(10):
        table.gather(b, out)
    g1.record()
    torch.cuda.synchronize()
    g_ms = g0.elapsed_time(g1) / 10
    g_bytes = n * DIM * 2 * 2 + n * 8
    line = {"metric": "dynamic embedding table step (dedup + lookup/insert + gather + SGD) IDs/s, 1 MI355X",
            "value": n * args.steps / elapsed, "unit": "ids/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "dtype": "bf16",
            "data": "synthetic",
            "config": {"workload": args.workload, "ids_per_step": n, "unique_per_step": nu,
                       "features_per_token": EMB_FEATURES, "dim": DIM, "row_capacity": ROWS,
                       "key_capacity": table.key_capacity, "live_keys": st["num_keys"], "embedding": True},
            "roofline": {"bound": "hbm", "kernel": "gather_kernel", "achieved": g_bytes / (g_ms * 1e-3) / 1e9,
                         "peak": 8000.0, "unit": "GB/s",
                         "frac": g_bytes / (g_ms * 1e-3) / 1e9 / 8000.0, "traffic": None}}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
