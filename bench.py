#!/usr/bin/env python3
"""Throughput of multi-cartridge prefix attention, forward + backward, on one
MI355X.

One step is one pass of the whole path over one batch: cas_prefix_attn_fwd
(O, LSE) then cas_prefix_attn_bwd (dQ, self dK/dV and every cartridge's
dK/dV), through the C ABI. Default workload: bf16, batch 2, 32 query / 8 KV
heads of 128 channels, 16 cartridges of 2048 tokens per row (32K-token
prefix) and 2048 causal query tokens, seeded synthetic inputs resident in HBM
before timing.

value = algorithmic TFLOP/s: 12 * head_dim * visible (query, key) pairs per
step (forward 4d: QK^T and PV; backward 8d: dV, dP, dQ, dK) over the measured
step time.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X published dense peaks (bf16 MFMA 2.5 PFLOP/s; fp32 matrix; HBM3E).
PEAK_BF16_TFLOPS = 2500.0
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0

METRIC = "prefix-attn fwd+bwd TFLOP/s & MFMA util, 8B GQA shape, 16×2K cartridges"

# Algorithmic FLOPs per visible (query, key) pair per query head, in units of
# head_dim, that each kernel owns: forward QK^T and PV; dK/dV pass dV, dP and
# dK; dQ pass dQ (together 12d per pair).
KERNEL_FLOPS_PER_PAIR = {"fwd": 4, "dkdv": 6, "dq": 2}
# What each kernel executes, recomputation included (S in every backward
# kernel, dP again in the dQ pass).
KERNEL_EXEC_FLOPS_PER_PAIR = {"fwd": 4, "dkdv": 8, "dq": 6}


def kernel_hbm_bytes(wl, kernel: str):
    """Compulsory HBM bytes of one launch: every tensor the kernel must read
    once and every result it writes once (the algorithmic traffic; re-reads
    and workspace copies are not counted)."""
    es = 2 if wl.dtype == "bf16" else 4
    T = sum(wl.row_lens)
    qb = T * wl.num_q_heads * wl.head_dim * es                     # Q, O, dO or dQ
    kvs = T * wl.num_kv_heads * wl.head_dim * es                   # self K or V
    used = sorted({c for r in wl.rows for c in r})
    kvc = sum(wl.cart_lens[c] for c in used) * wl.num_kv_heads * wl.head_dim * es
    stat = T * wl.num_q_heads * 4                                  # one fp32 per query row
    if kernel == "fwd":       # Q, K, V in; O, LSE out
        return qb + 2 * (kvc + kvs) + qb + stat
    if kernel == "dkdv":      # Q, dO, K, V, LSE, D in; dK, dV out
        return 2 * qb + 2 * (kvc + kvs) + 2 * stat + 2 * (kvc + kvs)
    if kernel == "dq":        # Q, dO, K, V, LSE, D in; dQ out
        return 2 * qb + 2 * (kvc + kvs) + 2 * stat + qb
    return None


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """Hash of the bf16 kernel code the recorded HBM counters belong to
    (comments and blank lines are left out: they do not change the kernel)."""
    import hashlib
    import re
    csrc = os.path.join(ROOT, "paper_2606_04557_amd", "csrc")
    code = []
    for f in ("cas_bf16.hip", "cas_device.h"):
        text = open(os.path.join(csrc, f), encoding="utf-8").read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for line in text.splitlines():
            line = re.sub(r"//.*", "", line).rstrip()
            if line.strip():
                code.append(line)
    return hashlib.sha256("\n".join(code).encode()).hexdigest()[:16]


def cpu_baseline(wl, T, heads: int = 1):
    """The fp64 oracle, as it stands, on a bounded sample of the same workload:
    the full forward and backward of `heads` (batch row 0) query heads over
    that row's whole key axis."""
    import numpy as np
    import casgen
    import oracle
    try:
        from threadpoolctl import threadpool_info
        cores = max(i.get("num_threads", 1) for i in threadpool_info()) or 1
    except Exception:
        cores = 1
    try:
        # BLAS may start more threads than the CPUs this process may run on.
        cores = min(cores, len(os.sched_getaffinity(0)))
    except (AttributeError, OSError):
        pass
    f = lambda a: None if a is None else casgen.to_float(a, wl.dtype)
    # Batch row 0's query tokens in either layout.
    row0 = (lambda a: a[0:wl.row_lens[0]]) if wl.packed else (lambda a: a[0])
    q, ks, vs, do = (row0(f(T[n])) for n in ("q", "k_self", "v_self", "d_o"))
    ck = [f(a) for a in T["cart_k"]]
    cv = [f(a) for a in T["cart_v"]]
    Sq = wl.row_lens[0]
    t_all = np.arange(Sq)
    elapsed = 0.0
    pairs = 0
    for h in range(heads):
        kv = h // wl.group_size
        K, V, npre = oracle.row_keys(ck, cv, wl.rows[0], ks, vs, kv)
        qh = q[:, h, :].astype(np.float64)
        doh = do[:, h, :].astype(np.float64)
        t0 = time.perf_counter()
        o, lse, _ = oracle.head_forward(qh, K, V, npre, Sq, t_all, float(wl.scale))
        oracle.head_backward(qh, K, V, npre, Sq, t_all, float(wl.scale), doh, o, lse)
        elapsed += time.perf_counter() - t0
        pairs += Sq * npre + Sq * (Sq + 1) // 2
    tflops = 12.0 * wl.head_dim * pairs / elapsed / 1e12
    return {"value": tflops, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
            "sample": f"batch row 0, {heads} of {wl.num_q_heads} query heads: full fp64 forward+backward "
                      f"({Sq} queries x {npre + Sq} keys each), {elapsed:.1f} s"}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=3, help="workload 1-4 (5 is forward-only)")
    ap.add_argument("--packed", action="store_true",
                    help="the 8,192-token packed training layout instead of --config")
    ap.add_argument("--adam", action="store_true",
                    help="time the cartridge Adam step over the packed layout's 20-cartridge pool")
    ap.add_argument("--decode", action="store_true",
                    help="time one paged decode step of the retrieval mix (64 requests x 4 cartridges)")
    ap.add_argument("--pool", action="store_true",
                    help="time training steps (packed attention fwd+bwd, Adam) through the budget manager")
    ap.add_argument("--moment-dir", default=None,
                    help="--pool: directory of the moment file tier (default: the temporary directory)")
    ap.add_argument("--stage", action="store_true",
                    help="time the forward-only retrieval mix with the pool's second half staged "
                         "host->HBM (cas_cartridge_stage) on a side stream, overlapped with compute")
    ap.add_argument("--no-dist", action="store_true",
                    help="skip the per-step warm/cold distribution runs after the timed region "
                         "(profiler passes: keeps every dispatch of a kernel alike)")
    ap.add_argument("--cpu-heads", type=int, default=16, help="oracle heads timed for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--mfma-counters", default=os.path.join(ROOT, "profiles", "mfma_util_16x2k.json"),
                    help="JSON of rocprofv3 MFMA counters per launch (executed MFMA work, MFMA busy cycles, "
                         "clock); used only while the kernel sources still hash to the value recorded in it")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "hbm_traffic_16x2k.json"),
                    help="JSON of calibrated rocprofv3 FETCH_SIZE/WRITE_SIZE bytes per launch; used only "
                         "while the kernel sources still hash to the value recorded in it")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run 5 plain device copies of MIB MiB (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the library has no "
              "multi-GPU path", file=sys.stderr)
        sys.exit(2)

    import torch
    import casgen
    import paper_2606_04557_amd as cas

    cas.load()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n // 2, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "copies": 5}), flush=True)
        return
    if args.adam:
        return run_adam(args)
    if args.decode:
        return run_decode(args)
    if args.pool:
        return run_pool(args)
    if args.stage:
        return run_stage(args)
    wl = casgen.packed() if args.packed else casgen.config(args.config)
    if wl.forward_only:
        print("bench.py times forward+backward; pick config 1-4", file=sys.stderr)
        sys.exit(2)
    log(f"generating {wl.name}: {wl.description}")
    T = casgen.make_tensors(wl)
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32

    def dev(a):
        import numpy as np
        if wl.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(a).cuda()

    q, k_self, v_self, d_o = dev(T["q"]), dev(T["k_self"]), dev(T["v_self"]), dev(T["d_o"])
    used = sorted({c for r in wl.rows for c in r})
    K = {c: dev(T["cart_k"][c]) for c in used}
    V = {c: dev(T["cart_v"][c]) for c in used}
    dK = {c: torch.empty_like(K[c]) for c in used}
    dV = {c: torch.empty_like(V[c]) for c in used}
    rows = [[cas.Segment(K[c], V[c], dK[c], dV[c]) for c in r] for r in wl.rows]
    Hkv, g, scale = wl.num_kv_heads, wl.group_size, float(wl.scale)
    qo = wl.q_offsets if wl.packed else None
    o = torch.empty_like(q)
    lse_shape = (wl.num_q_heads, sum(wl.row_lens)) if wl.packed else (wl.batch, wl.num_q_heads, wl.q_len)
    lse = torch.empty(lse_shape, dtype=torch.float32, device="cuda")
    dq = torch.empty_like(q)
    dks, dvs = torch.empty_like(k_self), torch.empty_like(v_self)
    prob = cas.Problem.from_tensors(q, rows, Hkv, g, scale, qo)
    ws = torch.empty(max(cas.workspace_size(prob, False), cas.workspace_size(prob, True)),
                     dtype=torch.uint8, device="cuda")
    plan = cas.plan_info(prob)
    log("plan", plan)

    def step():
        cas.prefix_attn_fwd(q, k_self, v_self, rows, Hkv, g, scale, o=o, lse=lse, workspace=ws,
                            q_offsets=qo)
        cas.prefix_attn_bwd(q, k_self, v_self, rows, Hkv, g, scale, o, lse, d_o, dq=dq,
                            dk_self=dks, dv_self=dvs, workspace=ws, q_offsets=qo)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} done; timing {args.steps} steps")
    cas.timing_reset()
    cas.timing_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    cas.timing_enable(False)
    ktimes = cas.timing_read()
    ms = (t1 - t0) * 1e3 / args.steps
    flops_step = wl.flops(12)
    value = flops_step / (ms * 1e-3) / 1e12
    log("kernel times", ktimes)

    # Per-step distribution (HIP events around each step on the launch
    # stream), warm and cold: before each cold step a 1 GiB buffer is
    # rewritten, more than the 256 MiB Infinity Cache and the L2s, so the
    # step starts from HBM. Both run after the timed region above.
    def per_step(cold: bool):
        scrub = torch.empty(1 << 28, dtype=torch.float32, device="cuda") if cold else None
        out = []
        for i in range(args.steps):
            if cold:
                scrub.fill_(float(i))
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            step()
            b.record()
            b.synchronize()
            out.append(a.elapsed_time(b))
        out.sort()
        return [out[len(out) // 10], out[len(out) // 2], out[(9 * len(out)) // 10]]

    warm_dist = cold_dist = None
    if not args.no_dist:
        warm_dist, cold_dist = per_step(False), per_step(True)
        log("per-step ms p10/p50/p90 warm", warm_dist, "cold", cold_dist)

    # Dominant kernel: the one with the largest total time in the timed region.
    dom = max(ktimes, key=lambda k: ktimes[k][1])
    launches, total = ktimes[dom]
    avg_ms = total / launches
    per_pair = KERNEL_FLOPS_PER_PAIR.get(dom)
    exec_pair = KERNEL_EXEC_FLOPS_PER_PAIR.get(dom)
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_FP32_TFLOPS
    achieved = wl.flops(per_pair) / (avg_ms * 1e-3) / 1e12 if per_pair else None
    traffic = None
    if args.traffic and os.path.exists(args.traffic) and args.config == 3 and not args.packed:
        with open(args.traffic) as fh:
            rec = json.load(fh)
        if rec.get("source_sha256_16") == kernel_source_hash():
            traffic = rec["kernels"].get(dom, {}).get("bytes")
    algo_bytes = kernel_hbm_bytes(wl, dom)
    roofline = {"bound": "mfma", "kernel": dom, "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                "frac": (achieved / peak) if achieved else None, "traffic": traffic,
                "avg_launch_ms": avg_ms,
                "flops_per_launch": wl.flops(per_pair) if per_pair else None,
                "flops_per_pair": f"{per_pair}d" if per_pair else None,
                # recomputation included: what the matrix cores execute
                "executed_flops_per_launch": wl.flops(exec_pair) if exec_pair else None,
                "executed_tflops": wl.flops(exec_pair) / (avg_ms * 1e-3) / 1e12 if exec_pair else None,
                "hbm": {"algorithmic_bytes": algo_bytes,
                        "algorithmic_gbs": algo_bytes / (avg_ms * 1e-3) / 1e9 if algo_bytes else None,
                        "measured_bytes": traffic,
                        "measured_gbs": traffic / (avg_ms * 1e-3) / 1e9 if traffic else None,
                        "measured_frac_of_peak": traffic / (avg_ms * 1e-3) / 1e9 / PEAK_HBM_GBS
                        if traffic else None,
                        "peak_gbs": PEAK_HBM_GBS}}
    kernels = {}
    for k, (n, t) in ktimes.items():
        kernels[k] = {"launches": n, "avg_ms": t / n}
        if k in KERNEL_FLOPS_PER_PAIR:
            a = wl.flops(KERNEL_FLOPS_PER_PAIR[k]) / (t / n * 1e-3) / 1e12
            kernels[k]["algorithmic_tflops"] = a
            kernels[k]["frac_of_peak"] = a / peak
    # MFMA utilisation: the MFMA work each launch executes (counted by
    # SQ_INSTS_VALU_MFMA_MOPS_BF16, recompute and masked tile parts included)
    # over this run's live launch time, against the dense bf16 peak; and the
    # MFMA busy share of the SIMD cycles at the clock the counter run saw.
    mfma_util = None
    if args.mfma_counters and os.path.exists(args.mfma_counters) and args.config == 3 and not args.packed:
        with open(args.mfma_counters) as fh:
            rec = json.load(fh)
        if rec.get("source_sha256_16") == kernel_source_hash():
            mfma_util = {}
            for k, c in rec["kernels"].items():
                if k in kernels:
                    live = c["executed_tflop"] / (kernels[k]["avg_ms"] * 1e-3)
                    mfma_util[k] = {"executed_tflop_per_launch": c["executed_tflop"],
                                    "executed_tflops": live, "frac_of_peak": live / peak,
                                    "busy_frac_at_clock": c["mfma_busy_frac"],
                                    "clock_ghz": c["clock_ghz"]}

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded Gaussian Q/K/V/dO; no model weights or datasets)",
        "config": ({"workload": f"{wl.name}: {wl.description}", "batch": wl.batch,
                    "q_len": wl.q_len, "num_q_heads": wl.num_q_heads, "num_kv_heads": Hkv,
                    "head_dim": wl.head_dim, "cartridges_per_row": len(wl.rows[0]),
                    "prefix_tokens_per_row": wl.prefix_len(0), "parallelism": "single GPU"}
                   if not wl.packed else
                   {"workload": f"{wl.name}: {wl.description}", "samples": wl.batch,
                    "sample_tokens": wl.row_lens, "cartridges_per_sample": [len(r) for r in wl.rows],
                    "prefix_tokens_per_sample": [wl.prefix_len(b) for b in range(wl.batch)],
                    "num_q_heads": wl.num_q_heads, "num_kv_heads": Hkv, "head_dim": wl.head_dim,
                    "parallelism": "single GPU"}),
        "mfma_frac_of_step": value / peak,
        "tflops_fa14": wl.flops(14) / (ms * 1e-3) / 1e12,
        "query_tokens_per_s": sum(wl.row_lens) / (ms * 1e-3),
        "kv_tokens_per_s": sum(wl.prefix_len(b) + wl.row_lens[b] for b in range(wl.batch)) / (ms * 1e-3),
        "step_ms_p10_p50_p90": warm_dist,
        "cold_step_ms_p10_p50_p90": cold_dist,
        "kernels": kernels,
        "roofline": roofline,
        "mfma_util": mfma_util,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        log("timing the fp64 oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(wl, T, heads=args.cpu_heads)
    print(json.dumps(out), flush=True)


def run_adam(args):
    """One fused Adam step (cas_cartridge_adam) over the K and V of the 20
    cartridges of the packed training layout's GPU pool (8 KV heads x 128, bf16
    parameters and gradients, fp32 moments, one frozen token each). Bound by
    HBM: 22 bytes move per updated element (2 + 2 read, 2 written for the
    parameter and its gradient; 8 read and 8 written for the two moments)."""
    import numpy as np
    import torch
    import casgen
    import paper_2606_04557_amd as cas
    from casgen import rng
    wl = casgen.packed()
    Hkv, D = wl.num_kv_heads, wl.head_dim
    carts = []
    for c, L in enumerate(wl.cart_lens):
        t = {}
        for i, n in enumerate(("k", "v", "dk", "dv")):
            bits = rng.f64_to_bf16_bits(rng.normal(rng.stream_key(wl.seed, 30 + i, c), L * Hkv * D,
                                                   0.5 if len(n) == 1 else 1e-2))
            t[n] = torch.from_numpy(bits.view(np.int16).reshape(L, Hkv, D)).view(torch.bfloat16).cuda()
        for n in ("m1_k", "m2_k", "m1_v", "m2_v"):
            t[n] = torch.zeros((L, Hkv, D), dtype=torch.float32, device="cuda")
        carts.append(cas.AdamCartridge(**t, step=25, frozen_tokens=1))
    elems = sum(2 * (L - 1) * Hkv * D for L in wl.cart_lens)
    nbytes = 22 * elems
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    cfg = dict(lr=0.05, beta1=0.9, beta2=0.999, eps=1e-8, warmup_steps=20, warmup_buckets=4)
    for _ in range(args.warmup):
        cas.cartridge_adam(carts, workspace=ws, **cfg)
    torch.cuda.synchronize()
    cas.timing_reset()
    cas.timing_enable(True)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        cas.cartridge_adam(carts, workspace=ws, **cfg)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    cas.timing_enable(False)
    kt = cas.timing_read()
    n, tot = kt["adam"]
    avg = tot / n
    ms = (t1 - t0) * 1e3 / args.steps
    achieved = nbytes / (avg * 1e-3) / 1e9
    out = {
        "metric": "cartridge Adam step, HBM GB/s (20-cartridge pool, 8 KV heads x 128)",
        "value": nbytes / (ms * 1e-3) / 1e9, "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32 (moments) / bf16 (parameters)",
        "data": "synthetic (seeded Gaussian parameters and gradients)",
        "config": {"workload": "Adam over the packed layout's cartridge pool", "cartridges": len(wl.cart_lens),
                   "tokens": sum(wl.cart_lens), "updated_elements": elems, "parallelism": "single GPU"},
        "kernels": {"adam": {"launches": n, "avg_ms": avg}},
        "roofline": {"bound": "hbm", "kernel": "adam", "achieved": achieved, "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "traffic": None,
                     "avg_launch_ms": avg, "bytes_per_launch": nbytes},
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        import oracle
        h = {k: np.asarray(v.float().cpu().numpy()) for k, v in
             (("x", carts[0].k), ("g", carts[0].dk), ("m1", carts[0].m1_k), ("m2", carts[0].m2_k))}
        t0 = time.perf_counter()
        reps = 0
        while time.perf_counter() - t0 < 2.0:
            oracle.adam.adam_step(h["x"], h["g"], h["m1"], h["m2"], 25, frozen_tokens=1, **cfg)
            reps += 1
        el = time.perf_counter() - t0
        per = 22 * (h["x"].shape[0] - 1) * Hkv * D
        out["cpu_baseline"] = {"value": reps * per / el / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
                               "sample": f"cartridge 0's K ({h['x'].shape[0]} tokens), {reps} steps in {el:.1f} s"}
    print(json.dumps(out), flush=True)


def run_decode(args):
    """One decode step (cas_paged_decode_fwd) of the retrieval-selected mix: a
    pool of 256 cartridges of 1,024 tokens in 16-token pages (8 KV heads x 128,
    bf16); 64 requests, each over its 4 retrieved cartridges (the same seeded
    selection as the forward-only retrieval configuration) and its own 64-token
    prompt, generating one token (4,161 keys each). HBM-bound: the algorithmic
    bytes are every request's K and V (counted per request)."""
    import numpy as np
    import torch
    import paper_2606_04557_amd as cas
    from casgen import rng
    P, Hkv, g, D, pool, cart_len, own = 16, 8, 4, 128, 256, 1024, 65
    cp = cart_len // P
    sel = [rng.choose_distinct(rng.stream_key(5, rng.TAG_SELECT, r), pool, 4) for r in range(64)]
    own_pages = -(-own // P)
    npages = pool * cp + 64 * own_pages
    shape = (npages, P, Hkv, D)
    n_el = int(np.prod(shape))
    kp = torch.from_numpy(rng.f64_to_bf16_bits(rng.normal(rng.stream_key(5, 40), n_el, 0.5)).view(np.int16)
                          .reshape(shape)).view(torch.bfloat16).cuda()
    vp = torch.from_numpy(rng.f64_to_bf16_bits(rng.normal(rng.stream_key(5, 41), n_el, 0.5)).view(np.int16)
                          .reshape(shape)).view(torch.bfloat16).cuda()
    pages, kv_lens = [], []
    nxt = pool * cp
    for s_ in sel:
        pl = [c * cp + j for c in s_ for j in range(cp)] + list(range(nxt, nxt + own_pages))
        nxt += own_pages
        pages.append(pl)
        kv_lens.append(4 * cart_len + own)
    q_counts = [1] * 64
    Hq = Hkv * g
    q = torch.from_numpy(rng.f64_to_bf16_bits(rng.normal(rng.stream_key(5, 42), 64 * Hq * D, 1.0)).view(np.int16)
                         .reshape(64, Hq, D)).view(torch.bfloat16).cuda()
    scale = float(np.float32(1.0 / np.sqrt(D)))
    o = torch.empty_like(q)
    lse = torch.empty((Hq, 64), dtype=torch.float32, device="cuda")
    prob = cas.DecodeProblem(q_counts, kv_lens, pages, npages, P, Hkv, g, D, scale)
    import ctypes
    n = ctypes.c_size_t(0)
    cas._check(cas.load().cas_paged_decode_workspace_size(ctypes.byref(prob.c), ctypes.byref(n)))
    ws = torch.empty(max(n.value, 1), dtype=torch.uint8, device="cuda")

    def step():
        cas.paged_decode_fwd(q, kp, vp, q_counts, kv_lens, pages, Hkv, g, scale, o=o, lse=lse, workspace=ws,
                             problem=prob)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    cas.timing_reset()
    cas.timing_enable(True)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    cas.timing_enable(False)
    kt = cas.timing_read()
    ms = (t1 - t0) * 1e3 / args.steps
    kv_bytes = sum(kv_lens) * Hkv * D * 2 * 2
    dn, dtot = kt["decode"]
    avg = dtot / dn
    gpu_ms = avg + (kt["decode_merge"][1] / kt["decode_merge"][0] if "decode_merge" in kt else 0.0)
    achieved = kv_bytes / (avg * 1e-3) / 1e9
    out = {
        "metric": "paged decode step over retrieved cartridges, HBM GB/s of K/V (64 requests x 4 x 1K-token cartridges)",
        "value": kv_bytes / (ms * 1e-3) / 1e9, "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded Gaussian pages and queries; seeded retrieval selection)",
        "config": {"workload": "Cartridge-RAG decode: 64 requests, 4 of 256 cartridges of 1,024 tokens + "
                               "64-token prompt, 1 new token each", "page_size": P, "kv_len": kv_lens[0],
                   "num_q_heads": Hq, "num_kv_heads": Hkv, "head_dim": D, "parallelism": "single GPU"},
        "tokens_per_s": 64 / (ms * 1e-3),
        "gpu_ms": gpu_ms,
        "kernels": {k: {"launches": c, "avg_ms": t / c} for k, (c, t) in kt.items()},
        "roofline": {"bound": "hbm", "kernel": "decode", "achieved": achieved, "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "traffic": None, "avg_launch_ms": avg,
                     "bytes_per_launch": kv_bytes},
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        import oracle
        # The first 8 requests, over a compact copy of just their pages.
        used = sorted({pg for pl in pages[:8] for pg in pl})
        remap = {pg: i for i, pg in enumerate(used)}
        idx = torch.tensor(used, device="cuda")
        kpn = kp.index_select(0, idx).float().cpu().numpy()
        vpn = vp.index_select(0, idx).float().cpu().numpy()
        qh = q[:8].float().cpu().numpy()
        t0 = time.perf_counter()
        oracle.paged_decode_forward(qh, kpn, vpn, q_counts[:8], kv_lens[:8],
                                    [[remap[pg] for pg in pl] for pl in pages[:8]], scale, g)
        el = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": sum(kv_lens[:8]) * Hkv * D * 4 / el / 1e9, "unit": "GB/s", "cores": 1,
                               "kind": "oracle", "sample": f"8 of the 64 requests, {el:.1f} s"}
    print(json.dumps(out), flush=True)


def run_stage(args):
    """The forward-only retrieval-selected inference mix with cartridge
    staging: 64 requests of 64 causal queries (32 query / 8 KV heads x 128,
    bf16), each over its 4 seeded selections from a pool of 256 cartridges of
    1,024 tokens. Cartridges 0-127 are resident in HBM; 128-255 sit in pinned
    host memory and are staged inside the timed region by cas_cartridge_stage
    on a side stream, in 8 chunks of 16 cartridges (K and V, 64 MiB per chunk)
    with one event each. Requests are grouped by the last chunk they need and
    launched in that order: the resident-only group at once, every other group
    after its chunk's event. Reported: the wall time of the whole mix, the
    staging alone (GB/s against the host link), the compute alone, and the
    overlap (t_copy + t_compute - t_wall) / min(t_copy, t_compute)."""
    import ctypes
    import numpy as np
    import torch
    import casgen
    import paper_2606_04557_amd as cas
    wl = casgen.config(5)
    pool, L = len(wl.cart_lens), wl.cart_lens[0]
    half, chunk = pool // 2, 16
    B, Sq, Hq, Hkv, D, g = wl.batch, wl.q_len, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_size
    used = sorted({c for r in wl.rows for c in r})
    log(f"generating {wl.name}: {wl.description} ({len(used)} cartridges selected)")
    T = casgen.make_tensors(wl, carts=used)

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)

    kdev = torch.zeros((pool, L, Hkv, D), dtype=torch.bfloat16, device="cuda")
    vdev = torch.zeros_like(kdev)
    khost = torch.zeros((pool - half, L, Hkv, D), dtype=torch.bfloat16).pin_memory()
    vhost = torch.zeros_like(khost).pin_memory()
    for c in used:
        if c < half:
            kdev[c].copy_(bf(T["cart_k"][c]))
            vdev[c].copy_(bf(T["cart_v"][c]))
        else:
            khost[c - half].copy_(bf(T["cart_k"][c]))
            vhost[c - half].copy_(bf(T["cart_v"][c]))
    # Requests ordered by the last staged chunk they need (-1: resident only).
    need = [max([(c - half) // chunk for c in r if c >= half], default=-1) for r in wl.rows]
    order = sorted(range(B), key=lambda r: need[r])
    q = bf(T["q"][order]).cuda()
    ks = bf(T["k_self"][order]).cuda()
    vs = bf(T["v_self"][order]).cuda()
    o = torch.empty_like(q)
    lse = torch.empty((B, Hq, Sq), dtype=torch.float32, device="cuda")
    scale = float(wl.scale)
    lib = cas.load()
    groups = []   # (chunk waited for, problem, first row, last row, workspace)
    r0 = 0
    while r0 < B:
        r1 = r0
        while r1 < B and need[order[r1]] == need[order[r0]]:
            r1 += 1
        rows = [[cas.Segment(kdev[c], vdev[c]) for c in wl.rows[order[r]]] for r in range(r0, r1)]
        prob = cas.Problem.from_tensors(q[r0:r1], rows, Hkv, g, scale, None)
        ws = torch.empty(max(cas.workspace_size(prob, False), 1), dtype=torch.uint8, device="cuda")
        groups.append((need[order[r0]], prob, r0, r1, ws, rows))
        r0 = r1
    # All 64 requests as one forward call (every selected cartridge
    # resident): the kernel on this workload without the staging's grouping.
    rows_all = [[cas.Segment(kdev[c], vdev[c]) for c in wl.rows[order[r]]] for r in range(B)]
    prob_all = cas.Problem.from_tensors(q, rows_all, Hkv, g, scale, None)
    ws_all = torch.empty(max(cas.workspace_size(prob_all, False), 1), dtype=torch.uint8, device="cuda")
    compute = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    hs = cas._stream_handle(q.device, None)
    nchunks = (pool - half) // chunk
    copies = []
    for ci in range(nchunks):
        # K of the chunk's 16 cartridges, then their V: address order in both
        # pools, so the library moves each as one transfer.
        arr = (cas._lib.StageCopy * (2 * chunk))()
        for m, (hp, dp) in enumerate(((khost, kdev), (vhost, vdev))):
            for j in range(chunk):
                c = ci * chunk + j
                e = arr[m * chunk + j]
                e.host_src, e.dev_dst, e.bytes = hp[c].data_ptr(), dp[half + c].data_ptr(), hp[c].numel() * 2
        copies.append(arr)
    stage_bytes = (pool - half) * 2 * L * Hkv * D * 2
    events = [torch.cuda.Event() for _ in range(nchunks)]
    for e in events:
        e.record(side)   # torch creates its events lazily

    def launch(gr):
        _, prob, a, b_, ws, _ = gr
        o_, lse_ = o[a:b_], lse[a:b_]
        cas._check(lib.cas_prefix_attn_fwd(ctypes.byref(prob.c), q[a:b_].data_ptr(), ks[a:b_].data_ptr(),
                                           vs[a:b_].data_ptr(), o_.data_ptr(), lse_.data_ptr(),
                                           ws.data_ptr(), ws.numel(), hs))

    def stage_all():
        for ci in range(nchunks):
            cas._check(lib.cas_cartridge_stage(ctypes.cast(copies[ci], ctypes.POINTER(cas._lib.StageCopy)),
                                               2 * chunk, side.cuda_stream, events[ci].cuda_event))

    def wall():
        side.wait_stream(compute)
        stage_all()
        for gr in groups:
            if gr[0] >= 0:
                compute.wait_event(events[gr[0]])
            launch(gr)

    def timed(fn):
        # Both streams start after t0 and t1 follows both (the side stream's
        # copies are joined into the compute stream before t1).
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0.record(compute)
        fn()
        compute.wait_stream(side)
        t1.record(compute)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1)

    def compute_only():
        for gr in groups:
            launch(gr)

    def compute_one_launch():
        cas._check(lib.cas_prefix_attn_fwd(ctypes.byref(prob_all.c), q.data_ptr(), ks.data_ptr(), vs.data_ptr(),
                                           o.data_ptr(), lse.data_ptr(), ws_all.data_ptr(), ws_all.numel(), hs))

    def copy_only():
        side.wait_stream(compute)
        stage_all()

    for _ in range(args.warmup):
        timed(wall)
    cas.timing_reset()
    cas.timing_enable(True)
    t_comp = sorted(timed(compute_only) for _ in range(args.steps))
    cas.timing_enable(False)
    kt = cas.timing_read()
    t_one = sorted(timed(compute_one_launch) for _ in range(args.steps))
    t_copy = sorted(timed(copy_only) for _ in range(args.steps))
    t_wall = sorted(timed(wall) for _ in range(args.steps))
    med = lambda v: v[len(v) // 2]
    tc, tx, tw = med(t_comp), med(t_copy), med(t_wall)
    flops = wl.flops(4)
    fwd_n, fwd_ms = kt["fwd"]
    achieved = flops * args.steps / (fwd_ms * 1e-3) / 1e12
    out = {
        "metric": "retrieval inference mix: forward TFLOP/s with host->HBM cartridge staging overlapped "
                  "(64 requests x 4 of 256 1K-token cartridges)",
        "value": flops / (tw * 1e-3) / 1e12, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": tw, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded Gaussian Q/K/V; seeded retrieval selection)",
        "config": {"workload": f"{wl.name}: {wl.description}", "requests": B, "q_len": Sq,
                   "num_q_heads": Hq, "num_kv_heads": Hkv, "head_dim": D, "pool": pool,
                   "staged_cartridges": pool - half, "chunks": nchunks, "launch_groups": len(groups),
                   "parallelism": "single GPU"},
        "t_wall_ms": tw, "t_compute_ms": tc, "t_copy_ms": tx,
        "t_wall_ms_p10_p90": [t_wall[len(t_wall) // 10], t_wall[(9 * len(t_wall)) // 10]],
        "staging_gb_s": stage_bytes / (tx * 1e-3) / 1e9, "staging_bytes": stage_bytes,
        "overlap": (tx + tc - tw) / min(tx, tc),
        "compute_tflops": flops / (tc * 1e-3) / 1e12,
        "compute_one_launch_ms": med(t_one),
        "compute_one_launch_tflops": flops / (med(t_one) * 1e-3) / 1e12,
        "kernels": {k: {"launches": c, "avg_ms": t / c} for k, (c, t) in kt.items()},
        "roofline": {"bound": "mfma", "kernel": "fwd", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS, "traffic": None,
                     "avg_launch_ms": fwd_ms / fwd_n, "flops_per_launch": flops * args.steps / fwd_n},
        "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)


def run_pool(args):
    """Training steps through the budget manager with the paper's settings
    (B = 20 active of N = 60 cartridges, rotation every R = 10 steps swapping
    phi = 0.5 of the pool, least-trained first): per step one layer's packed
    8,192-token attention forward and backward over the active cartridges
    (the packed layout's samples, their cartridge slots mapped onto the active
    set), the fused Adam step, and cas_pool_end_step. The same loop with
    phi = 0 (no rotation) gives the cost of the rotations' copies, which run
    on the pool's stream behind the compute. The rotating loop runs twice:
    with the offloaded cartridges' Adam moments in pinned host memory, and
    with them in a file under --moment-dir (the NVMe tier; its reads and
    writes run on the pool's thread)."""
    import numpy as np
    import torch
    import casgen
    import paper_2606_04557_amd as cas
    from casgen import rng
    wl = casgen.packed()
    Hkv, g, D = wl.num_kv_heads, wl.group_size, wl.head_dim
    lens = [wl.cart_lens[c % len(wl.cart_lens)] for c in range(60)]
    T = casgen.make_tensors(wl, carts=[])
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    q, ks, vs, do = dev(T["q"]), dev(T["k_self"]), dev(T["v_self"]), dev(T["d_o"])
    qo, scale = wl.q_offsets, float(wl.scale)
    o, dq = torch.empty_like(q), torch.empty_like(q)
    lse = torch.empty((wl.num_q_heads, sum(wl.row_lens)), dtype=torch.float32, device="cuda")
    dks, dvs = torch.empty_like(ks), torch.empty_like(vs)
    cfg = dict(lr=0.05, beta1=0.9, beta2=0.999, eps=1e-8, warmup_steps=20, warmup_buckets=4)
    import tempfile
    mdir = args.moment_dir or tempfile.gettempdir()
    res = {}
    steps = args.steps if args.steps >= 20 else 40
    for key in ("file", 0.5, 0.0):
        phi = 0.5 if key == "file" else key
        pl = cas.CartridgePool(lens, Hkv, D, 20, 10, phi, frozen_tokens=1,
                               moment_dir=mdir if key == "file" else None)
        for c, L in enumerate(lens):
            h = pl.host(c)
            for i, name in enumerate(("k", "v")):
                h[name][...] = rng.f64_to_bf16_bits(rng.normal(rng.stream_key(60, c, i), L * Hkv * D, 0.5)
                                                    ).view(np.int16).reshape(L, Hkv, D)
        pl.load()

        def step():
            act = pl.active()
            views = [a for _, a in act]
            rows = [[cas.Segment(views[i].k, views[i].v, views[i].dk, views[i].dv) for i in r] for r in wl.rows]
            cas.prefix_attn_fwd(q, ks, vs, rows, Hkv, g, scale, o=o, lse=lse, q_offsets=qo)
            cas.prefix_attn_bwd(q, ks, vs, rows, Hkv, g, scale, o, lse, do, dq=dq, dk_self=dks, dv_self=dvs,
                                q_offsets=qo)
            cas.cartridge_adam(views, **cfg)
            pl.end_step()

        for _ in range(5):
            step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        res[key] = (time.perf_counter() - t0) * 1e3 / steps
        pl.flush()
        pl.close()
        log(f"pool {key}: {res[key]:.3f} ms per step")
    per_cart = [L * Hkv * D * (2 * 2 + 4 * 4) for L in lens]
    moved = 2 * 10 * (sum(per_cart) / len(per_cart))         # 10 evicted + 10 admitted per rotation
    out = {
        "metric": "training step through the budget manager, ms per step (packed 8K attention fwd+bwd + Adam)",
        "value": res[0.5], "unit": "ms", "n_gpus": 1, "steps": steps, "warmup": 5, "ms_per_step": res[0.5],
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded Gaussian cartridges and samples)",
        "config": {"workload": "N = 60 cartridges, B = 20 active, rotation every 10 steps swapping 10 "
                               "(least-trained first); one attention layer of the packed 8,192-token layout",
                   "parallelism": "single GPU"},
        "ms_per_step_without_rotation": res[0.0],
        "rotation_overhead_frac": res[0.5] / res[0.0] - 1.0,
        "bytes_moved_per_rotation": moved,
        "moment_file_tier": {"ms_per_step": res["file"], "overhead_frac": res["file"] / res[0.0] - 1.0,
                             "directory": mdir,
                             "file_bytes_per_rotation": 2 * 10 * sum(L * Hkv * D * 16 for L in lens) / len(lens),
                             "pinned_host_bytes": {"host_tier": sum(per_cart),
                                                   "file_tier": sum(L * Hkv * D * 4 for L in lens)
                                                   + 3 * 10 * 4 * max(lens) * Hkv * D * 4}},
        "roofline": None, "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
