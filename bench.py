"""Benchmark of the group-batched step on one MI355X.

A step = jn_pack_group -> jn_backbone_forward -> jn_tenant_heads_fwd_bwd ->
jn_unpack over one group of requests with inputs resident in HBM.  Default
workload: 8 tenants x 32 samples on an 18-layer d2048 GeGLU (2B-shaped)
backbone with per-tenant 3-layer MLP heads (seeded synthetic inputs).

Reported in one JSON line: grouped samples/s (value), backbone tokens/s,
isolated per-tenant execution (the same calls once per tenant, same kernels
and tile rule) and the speedup over it, the GEMM roofline of the dominant
kernel measured with HIP events on the library stream, and the fp64 CPU
oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "grouped samples/s + backbone tokens/s at 1 GPU; speedup vs isolated; % MFMA peak"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


GEMM_SRC = os.path.join(ROOT, "paper_2607_16074_amd", "csrc", "k_gemm.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_geglu_traffic.json")


def source_hash(path: str) -> str:
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(config: int):
    """HBM bytes per launch of the dominant GEMM from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary (taken on the 8x32 2B-shaped workload), or
    None for another workload or once the kernel source changed."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if config != t.get("config", 3) or t.get("kernel_source_sha256_16") != source_hash(GEMM_SRC):
        return None
    return t.get("bytes_per_launch")


def copy_calibration(mib: int = 512):
    """A plain device copy of known size, for scaling the PMC byte counters."""
    import torch
    a = torch.empty(mib << 18, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    log(f"copy calibration: {mib} MiB device-to-device copy")
    del a, b


def copy_reference(mib: int = 1024, reps: int = 20) -> dict:
    """The practical rate of a stream that reads and writes HBM once: a plain
    device-to-device copy (torch copy_), timed with events after warm-up."""
    import torch
    a = torch.empty(mib << 18, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del a, b
    gbs = 2.0 * (mib << 20) / (ms * 1e-3) / 1e9
    return {"what": f"{mib} MiB device-to-device copy (torch copy_), read + write", "ms": ms, "GB_per_s": gbs,
            "frac_of_hbm": gbs / PEAK_HBM_GBS}


def gemm_flops_per_token(bb) -> dict:
    d, f = bb.d, bb.ffn
    up = 2 * (2 * f if bb.glu else f) * d
    return {"gemm_qkv": 2 * bb.qkv_rows * d, "gemm_o": 2 * d * d, "gemm_up": up, "gemm_down": 2 * f * d}


def kernel_rates(by_op, steps, spec, reqs, T, valid, N):
    """Attention against the bf16 MFMA peak and the HBM-bound kernels against
    8 TB/s, from their per-step event times and algorithmic work (valid rows
    only; bytes each kernel must move)."""
    bb = spec.backbone
    d, H, hd = bb.d, bb.heads, bb.d // bb.heads
    lens = np.concatenate([np.asarray(r.lengths, np.int64) for r in reqs])
    if bb.causal:
        att_flops = bb.layers * float(np.sum(2 * lens * (lens + 1) * d))   # keys <= query only
    else:
        att_flops = bb.layers * float(np.sum(4 * lens * lens * d))
    out = {}
    if "attention" in by_op:
        ms = by_op["attention"]["ms"] / steps
        out["attention"] = {"ms_per_step": ms, "tflops": att_flops / (ms * 1e-3) / 1e12,
                            "frac_of_bf16_peak": att_flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}
    # bytes per step: pack / unpack read and write every valid row once; the
    # first RMSNorm reads bf16 and writes the fp32 residual and the bf16 output,
    # the other 2L of them read fp32 and write bf16; pool reads every valid row
    # and writes N fp32 rows; the rotation reads and writes q and k
    kvh = bb.kv_heads or H
    nbytes = {"pack": 4.0 * valid * d, "unpack": 4.0 * valid * d,
              "rmsnorm": (8.0 + 6.0 * 2 * bb.layers) * T * d, "pool": 2.0 * valid * d + 4.0 * N * d,
              "rope": bb.layers * 4.0 * T * (H + kvh) * hd}
    for op, b in nbytes.items():
        if op in by_op:
            ms = by_op[op]["ms"] / steps
            out[op] = {"ms_per_step": ms, "GB_per_s": b / (ms * 1e-3) / 1e9,
                       "frac_of_hbm": b / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS}
    return out


def time_steps(steps, fn, ctx, warmup):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ctx.set_trace(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    trace = ctx.trace_read()
    ctx.set_trace(False)
    return (t1 - t0) / steps, trace


def cpu_oracle_baseline(wl, budget_s=25.0):
    """The fp64 oracle on a bounded sample: one sample's full backbone plus
    its tenant's head step; reported as oracle samples/s."""
    import oracle
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        threads = max([i.get("num_threads", 1) for i in info if i.get("user_api") == "blas"] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    req = wl.requests[0]
    key = (0, 0)
    t0 = time.perf_counter()
    res = oracle.step.isolated(wl, samples=[key], heads=False)
    ten = wl.spec.tenants[req.tenant]
    if ten.expert is None:
        n0 = ten.n_samples
        P = np.repeat(res["pooled"][key][None, :], n0, axis=0)
        oracle.step.tenant_from_pooled(wl, req.tenant, P)
        what = f"its tenant's head fwd/loss/grad over {n0} rows"
    else:
        # the sample's own expert forward, loss and gradients (one sample of its tenant)
        from oracle import expert as oexpert
        L_e, _, H_e, _ = ten.expert
        z = res["hidden"][key]
        ft = wl.flow_t[req.tenant] if getattr(wl, "flow_t", None) else None
        oexpert.expert_step(wl.experts[req.tenant], L_e, H_e, wl.spec.backbone.eps, [wl.noisy[req.tenant][0]], [z],
                            wl.targets[req.tenant][:1], flow_t=None if ft is None else ft[:1])
        what = "its tenant's action-expert fwd/loss/grad for that sample"
    dt = time.perf_counter() - t0
    L = int(req.lengths[0])
    return {"value": 1.0 / dt, "unit": "samples/s", "cores": int(threads), "kind": "oracle",
            "sample": f"1 of {sum(q.n for q in wl.requests)} samples ({L} tokens): full backbone forward in fp64 "
                      f"+ {what}; {dt:.1f} s on the host",
            "seconds": dt, "host_cpus": os.cpu_count(), "cpu_model": cpu_model()}


def cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo), or "" where unavailable."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


def local_batch_sweep(model, reqs, targets, steps, warmup, tenants_list=(2, 4, 6, 8), batches=(1, 2, 4, 8)):
    """Grouped vs isolated step time over tenants x local batch on one model:
    the first G tenants each submit their first n samples."""
    import torch
    from paper_2607_16074_amd import Context, Request
    from paper_2607_16074_amd import step as jstep
    ctx = Context()
    rows = []
    for G in tenants_list:
        for n in batches:
            sub = [Request(r.tenant, r.embeds[:n], r.lengths[:n]) for r in reqs if r.tenant < G]
            tg = {g: targets[g][:n] for g in range(G)}
            grouped = jstep.GroupStep(model, sub, tg, list(range(G)), 1, ctx)
            iso = jstep.isolated_runs(model, sub, tg, list(range(G)), 1, ctx)
            torch.cuda.synchronize()
            tg_s, _ = time_steps(steps, grouped.run, ctx, warmup)

            def run_iso():
                for st in iso:
                    st.run()
            ti_s, _ = time_steps(steps, run_iso, ctx, warmup)
            rows.append({"tenants": G, "local_batch": n, "grouped_ms": tg_s * 1e3, "isolated_ms": ti_s * 1e3,
                         "speedup": ti_s / tg_s})
            log(f"sweep G={G} n={n}: grouped {tg_s * 1e3:.2f} ms, isolated {ti_s * 1e3:.2f} ms, "
                f"{ti_s / tg_s:.2f}x")
            del grouped, iso
            torch.cuda.synchronize()
    return rows


def infer_latency(model, reqs, steps, warmup, tenants_list=(1, 2, 4, 8), per_tenant=(1, 4)):
    """Decode-only step latency (launch to completion, host clock) of a group
    of G tenants x n samples: eager launch vs replay of the captured HIP
    graph, and the same requests as G single-tenant steps (each replayed)."""
    import torch
    from paper_2607_16074_amd import Request
    from paper_2607_16074_amd import step as jstep

    def lat(fn, sync):
        for _ in range(warmup):
            fn()
        sync()
        ts = []
        for _ in range(steps):
            t0 = time.perf_counter()
            fn()
            sync()
            ts.append(time.perf_counter() - t0)
        return float(np.median(ts)) * 1e3

    rows = []
    for G in tenants_list:
        for n in per_tenant:
            sub = [Request(r.tenant, r.embeds[:n], r.lengths[:n]) for r in reqs if r.tenant < G]
            grp = jstep.InferStep(model, sub, list(range(G)))
            eager = lat(grp.launch, grp.synchronize)
            grp.capture()
            graph = lat(grp.replay, grp.synchronize)
            iso = []
            for g in range(G):
                st = jstep.InferStep(model, [q for q in sub if q.tenant == g], [g], stream=grp.stream)
                st.capture()
                iso.append(st)

            def run_iso():
                for st in iso:
                    st.replay()
            iso_ms = lat(run_iso, grp.synchronize)
            rows.append({"tenants": G, "samples_per_tenant": n, "eager_ms": eager, "graph_ms": graph,
                         "isolated_graph_ms": iso_ms, "speedup_vs_isolated": iso_ms / graph})
            log(f"infer G={G} n={n}: eager {eager:.2f} ms, graph {graph:.2f} ms, isolated (graphs) {iso_ms:.2f} ms")
            del grp, iso
            torch.cuda.synchronize()
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--align", type=int, default=1)
    ap.add_argument("--no-isolated", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-optimizer", action="store_true")
    ap.add_argument("--breakdown", action="store_true", help="print per-kernel time shares to stderr")
    ap.add_argument("--sweep", action="store_true",
                    help="grouped vs isolated over tenants {2,4,6,8} x local batch {1,2,4,8} (one JSON line)")
    ap.add_argument("--infer", action="store_true",
                    help="decode-only step latency of small groups: eager vs HIP-graph replay vs isolated (one JSON line)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run a 512 MiB device copy first (reference dispatch for PMC byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the step is sharded by "
              f"whole tenants across GPUs with no collective on the forward; run one process per GPU).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads as W
    from paper_2607_16074_amd import step as jstep

    if args.copy_calibration:
        copy_calibration()
    t0 = time.perf_counter()
    wl = W.make_workload(args.config)
    spec = wl.spec
    log(f"workload cfg{args.config} drawn in {time.perf_counter() - t0:.1f}s: {spec.name}")
    model, reqs, targets, noisy = jstep.from_workload(wl, "cuda", with_noisy=True)
    if args.infer:
        rows = infer_latency(model, reqs, args.steps, args.warmup)
        print(json.dumps({"infer_latency": "decode-only step, launch to completion (host clock, median)",
                          "config": f"config {args.config}: {spec.name}", "rows": rows}), flush=True)
        return
    if args.sweep:
        rows = local_batch_sweep(model, reqs, targets, args.steps, args.warmup)
        print(json.dumps({"sweep": "grouped vs isolated step time, tenants x local batch",
                          "config": f"config {args.config}: {spec.name}", "rows": rows}), flush=True)
        return
    G = spec.G
    experts = spec.tenants[0].expert is not None
    flow = jstep.flow_times(wl)
    grouped = jstep.GroupStep(model, reqs, targets, list(range(G)), args.align, noisy=noisy, flow_t=flow)
    torch.cuda.synchronize()
    N, valid = grouped.N, grouped.valid_tokens
    log(f"N={N} samples, {valid} valid tokens, T={grouped.T} packed rows")

    t_step, trace = time_steps(args.steps, grouped.run, grouped.ctx, args.warmup)
    log(f"grouped: {t_step * 1e3:.2f} ms/step")

    # per-kernel-class time from the trace
    by_op = {}
    for op, M, Nn, K, ms in trace:
        e = by_op.setdefault(op, {"ms": 0.0, "launches": 0})
        e["ms"] += ms
        e["launches"] += 1
    bb_ms = sum(v["ms"] for k, v in by_op.items() if k in ("rmsnorm", "gemm_qkv", "rope", "attention", "gemm_o",
                                                          "gemm_up", "gemm_down")) / args.steps
    fpt = gemm_flops_per_token(spec.backbone)
    gemm_stats = {}
    for op, per_tok in fpt.items():
        if op in by_op:
            avg = by_op[op]["ms"] / by_op[op]["launches"]
            flops = per_tok * valid
            gemm_stats[op] = {"avg_ms": avg, "tflops": flops / (avg * 1e-3) / 1e12,
                              "launches_per_step": by_op[op]["launches"] // args.steps}
    dom = max(gemm_stats, key=lambda k: gemm_stats[k]["avg_ms"] * gemm_stats[k]["launches_per_step"])
    gemm_total_ms = sum(by_op[k]["ms"] for k in fpt if k in by_op) / args.steps
    gemm_total_flops = sum(fpt[k] * valid * gemm_stats[k]["launches_per_step"] for k in gemm_stats)
    gemm_tflops = gemm_total_flops / (gemm_total_ms * 1e-3) / 1e12
    if args.breakdown:
        tot = sum(v["ms"] for v in by_op.values())
        for k, v in sorted(by_op.items(), key=lambda kv: -kv[1]["ms"]):
            log(f"  {k:10s} {v['ms'] / args.steps:9.3f} ms/step  {100 * v['ms'] / tot:5.1f}%  "
                f"launches/step {v['launches'] // args.steps}")
        for k, v in gemm_stats.items():
            log(f"  {k:10s} {v['avg_ms']:.3f} ms/launch  {v['tflops']:.0f} TFLOP/s")

    iso_ms = None
    if not args.no_isolated:
        iso = jstep.isolated_runs(model, reqs, targets, list(range(G)), args.align, ctx=grouped.ctx, noisy=noisy,
                                  flow_t=flow)
        torch.cuda.synchronize()

        def run_iso():
            for s in iso:
                s.run()
        t_iso, _ = time_steps(args.steps, run_iso, grouped.ctx, args.warmup)
        iso_ms = t_iso * 1e3
        log(f"isolated: {iso_ms:.2f} ms/step")
        del iso
        torch.cuda.synchronize()

    # the per-tenant AdamW step over the group's tenant parameters (not part of `value`)
    opt_stats = None
    if not args.no_optimizer:
        opt = jstep.TenantOptimizer(grouped, lr=1e-4, weight_decay=0.01)
        opt.step()
        torch.cuda.synchronize()
        grouped.ctx.set_trace(True)
        for _ in range(5):
            opt.step()
        torch.cuda.synchronize()
        tr = [e for e in grouped.ctx.trace_read() if e[0] == "optimizer"]
        grouped.ctx.set_trace(False)
        ms = sum(e[4] for e in tr) / max(1, len(tr))
        elems = sum(int(p.numel()) for ps, _, _ in opt.sets for p in ps)
        b16 = sum(int(p.numel()) for ps, _, b in opt.sets if b is not None for p in ps)
        nbytes = 28 * elems + 2 * b16
        opt_stats = {"ms": ms, "params": elems, "bytes": nbytes, "GB_per_s": nbytes / (ms * 1e-3) / 1e9,
                     "frac_of_hbm": nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS}
        log(f"optimizer: {ms:.3f} ms for {elems} parameters ({opt_stats['GB_per_s']:.0f} GB/s)")
        del opt
        torch.cuda.synchronize()

    cpu = None
    if not args.no_cpu:
        cpu = cpu_oracle_baseline(wl)
        log(f"cpu oracle: {cpu['value']:.4f} samples/s on {cpu['cores']} threads")

    gs = gemm_stats[dom]
    # reference rate for the HBM-bound kernels, measured after the timed steps
    copy_ref = copy_reference()
    kernels = kernel_rates(by_op, args.steps, spec, reqs, grouped.T, valid, N)
    for v in kernels.values():
        if "GB_per_s" in v:
            v["frac_of_copy"] = v["GB_per_s"] / copy_ref["GB_per_s"]
    if opt_stats is not None:
        opt_stats["frac_of_copy"] = opt_stats["GB_per_s"] / copy_ref["GB_per_s"]
    log(f"copy reference: {copy_ref['GB_per_s']:.0f} GB/s")
    result = {
        "metric": METRIC,
        "value": N / t_step,
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": t_step * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"config {args.config}: {spec.name}; per-tenant "
                               f"{'action experts' if experts else 'MLP heads'}, seed {spec.seed}",
                   "tenants": G, "samples": N, "valid_tokens": valid, "packed_rows": grouped.T,
                   "align": args.align},
        "backbone_tokens_per_s": valid / (bb_ms * 1e-3),
        "backbone_ms": bb_ms,
        "tenant_stage_ms": sum(v["ms"] for k, v in by_op.items()
                               if k in ("pool", "head_fwd", "loss", "head_bwd", "expert_gemm", "expert_attention",
                                        "expert_other")) / args.steps,
        "isolated_samples_per_s": (N / (iso_ms * 1e-3)) if iso_ms else None,
        "isolated_ms_per_step": iso_ms,
        "speedup_vs_isolated": (iso_ms / (t_step * 1e3)) if iso_ms else None,
        "backbone_gemm_tflops": gemm_tflops,
        "backbone_gemm_frac_of_bf16_peak": gemm_tflops / PEAK_BF16_TFLOPS,
        "roofline": {"bound": "mfma", "kernel": f"{dom} projection GEMM ({spec.backbone.d}-wide; gemm_ring_kernel tiles)",
                     "achieved": gs["tflops"], "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": gs["tflops"] / PEAK_BF16_TFLOPS, "traffic": measured_traffic(args.config),
                     "avg_launch_ms": gs["avg_ms"], "flops_per_launch": fpt[dom] * valid},
        "gemm_by_op": gemm_stats,
        "kernels": kernels,
        "copy_reference": copy_ref,
        "tenant_optimizer": opt_stats,
        "cpu_baseline": None if cpu is None else {k: cpu[k] for k in ("value", "unit", "cores", "kind", "sample",
                                                                      "host_cpus", "cpu_model")},
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
