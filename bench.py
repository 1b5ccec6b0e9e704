"""Benchmark: head-chunked causal GQA attention fwd+bwd on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input:
upipe_attn_fwd followed by upipe_attn_bwd (pack, flash forward, unpack,
backward pre-pass, dK/dV, dQ, unpack, for every head chunk) on the
Llama3-8B per-GPU share at 8-way Ulysses (S = 131072, 4 query heads, 1 kv
head, d = 128), inputs resident in HBM.  Prints one JSON line.
`--workload qwen32b_share|llama8b_4m|tiny` times the other attention
shares; `--workload llama8b_layer` times upipe_layer_fwd + upipe_layer_bwd.

Throughput counts only algorithmic work: 4 d flops per visible causal
(query, key, head) triple for the forward and 2.5x that for the backward;
for the layer also 2 flops per multiply-add of the QKV and output
projections, 3x (forward, data gradient, weight gradient; the backward's
recomputation of K, V and Q is not credited).
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = ("attention fwd+bwd TFLOP/s (causal) per MI355X; "
          "peak activation GB vs chunk size U")
KERNEL_SOURCES = {"attn_fwd": ("attn_fwd.hip", "common.h"),
                  "attn_bwd_dkdv": ("attn_bwd.hip", "common.h"),
                  "attn_bwd_dq": ("attn_bwd.hip", "common.h")}
PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 4096 flop/clk x 2.4 GHz, dense bf16
PEAK_HBM_GBS = 8000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=5)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--workload", default="llama8b_share")
    p.add_argument("--U", type=int, default=1)
    p.add_argument("--no-sweep", action="store_true",
                   help="skip the per-U throughput/memory sweep")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--batch", type=int, default=1,
                   help="sequences per step (each of the workload's length S), run "
                        "through one workspace")
    p.add_argument("--checkpointing", choices=("selective", "full"), default="selective",
                   help="layer workloads: keep the attention output for the backward "
                        "(selective) or recompute it there (full)")
    p.add_argument("--rope-base", type=float, default=None,
                   help="layer workloads: rotary base (0 = none); default: the workload's")
    p.add_argument("--cpu-seconds", type=float, default=15.0,
                   help="target CPU time of the oracle sample")
    p.add_argument("--ceiling", action="store_true",
                   help="instead of the workload: the sustained bf16 MFMA rate of a large "
                        "plain GEMM (the library's projection GEMM and torch.matmul), "
                        "each run back to back for --ceiling-seconds")
    p.add_argument("--ceiling-size", type=int, default=8192)
    p.add_argument("--ceiling-seconds", type=float, default=3.0)
    return p.parse_args()


def kernel_flops(S, Hq, B, d, fwd_passes=1, causal=True):
    """Algorithmic flops per step of each attention kernel family, over all
    Hq heads of B sequences (independent of how the library splits the heads
    into launches; per launch it is this over the launch count when the
    launches are equal).  fwd_passes = 2 when the backward recomputes the
    forward (full checkpointing)."""
    pairs = S * (S + 1) // 2 if causal else S * S
    heads = Hq * B
    return {
        "attn_fwd": 4 * d * pairs * heads * fwd_passes,   # Q K^T and P V
        "attn_bwd_dkdv": 8 * d * pairs * heads,           # S, dP recompute + dV, dK
        "attn_bwd_dq": 2 * d * pairs * heads,             # dQ (S, dP recomputed again)
    }


def source_sha(kernel):
    """Hash of the sources a kernel is built from (traffic records go stale
    when they change)."""
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2602_21196_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, workload, U):
    """HBM bytes per launch from profiles/traffic.json (rocprofv3 FETCH_SIZE
    and WRITE_SIZE, calibrated on a copy kernel), if they were taken on the
    current source of that kernel for this workload; else None."""
    import json as _json
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            rec = _json.load(f).get(f"{workload}/U{U}/{kernel}")
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_sha") != source_sha(kernel):
        return None
    return rec["fetch_bytes"] + rec["write_bytes"]


def measured_clock(kernel, workload, U):
    """Sustained shader clock (GHz) under a kernel from profiles/clock.json
    (rocprofv3 GRBM_COUNT per dispatch over its kernel-trace duration, per
    XCD), if it was taken on the current source of that kernel for this
    workload; else None."""
    import json as _json
    path = os.path.join(ROOT, "profiles", "clock.json")
    try:
        with open(path) as f:
            rec = _json.load(f).get(f"{workload}/U{U}/{kernel}")
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_sha") != source_sha(kernel):
        return None
    return rec["clock_ghz"]


def host_info():
    """(BLAS threads in use, BLAS library, CPU model) of this host."""
    cores, blas = os.cpu_count(), "unknown"
    try:
        from threadpoolctl import threadpool_info
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"] or threadpool_info()
        if info:
            cores = max(i.get("num_threads", 1) for i in info)
            blas = ",".join(sorted({str(i.get("internal_api", "?")) for i in info}))
    except Exception:  # pragma: no cover
        pass
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    return cores, blas, cpu


def cpu_baseline(w, q, k, v, do, target_s):
    """Oracle (float64 numpy) on a bounded causal prefix of the workload.

    The first S' tokens of a causal sequence form a causal attention problem
    of their own with exactly the same rows; the oracle runs forward and
    backward for one query head on that prefix and its rate is reported in
    the metric's unit (TFLOP/s of algorithmic work).
    """
    import numpy as np
    from oracle import attention as A
    cores, blas, cpu = host_info()

    def run(sp):
        f = lambda t, h: t[:sp, :h].float().double().numpy()  # noqa: E731
        args = (f(q, 1), f(k, 1), f(v, 1), f(do, 1))
        t0 = time.perf_counter()
        A.attn_fwd(*args[:3])
        A.attn_bwd(*args)
        return time.perf_counter() - t0

    # Time grows ~ S'^2 once the fixed overheads are amortised: grow S' from
    # a small probe until one run takes at least 0.6 x target_s.
    sp = 2048
    t = run(sp)
    for _ in range(4):
        if t >= 0.6 * target_s or sp >= w.S:
            break
        scale = (target_s / max(t, 1e-3)) ** 0.5
        sp = int(min(w.S, max(sp + 128, (sp * scale) // 128 * 128)))
        t = run(sp)
    pairs = sp * (sp + 1) // 2
    flops = 3.5 * 4 * w.d * pairs
    full_pairs = w.S * (w.S + 1) // 2 * w.Hq
    return {"value": round(flops / t / 1e12, 6), "unit": "TFLOP/s",
            "cores": cores, "kind": "oracle", "blas": blas, "cpu": cpu,
            "sample": f"causal prefix S'={sp} of {w.name}, 1 query head "
                      f"(kv head 0), fwd+bwd, float64 numpy, {t:.1f} s",
            "extrapolated_full_s": round(t * full_pairs / pairs, 1),
            "extrapolated_note": "whole workload (all heads, full S) at the "
                                 "sampled rate; extrapolated, not run"}


def workspace_model_gb(S, Hq, Hkv, d, U):
    """Attention-only backward workspace model A + B U (the larger of the two
    workspaces): resident packed K, V (none when one key/value head of a
    length that is a multiple of 128 is read in place), fp32 dK, dV carries
    when a key/value group spans chunks, and, per chunk head, Q, dO, dQ
    (bf16) and lse, D."""
    Sp = (S + 127) // 128 * 128
    G = Hq // Hkv   # a group spans chunks when its first and last heads differ in h // U
    carry = any((g * G) // U != ((g + 1) * G - 1) // U for g in range(Hkv))
    packed_kv = not (Hkv == 1 and S % 128 == 0)
    fixed = (2 * Sp * Hkv * d * 2 if packed_kv else 0) + (2 * Sp * Hkv * d * 4 if carry else 0)
    return (fixed + U * Sp * (3 * d * 2 + 2 * 4)) / 1e9


def linear_fit(xs, ys):
    """Least-squares y = A + B x and R^2."""
    n = len(xs)
    mx, my = sum(xs) / n, sum(ys) / n
    sxx = sum((x - mx) ** 2 for x in xs)
    B = sum((x - mx) * (y - my) for x, y in zip(xs, ys)) / sxx if sxx else 0.0
    A = my - B * mx
    ss_tot = sum((y - my) ** 2 for y in ys)
    ss_res = sum((y - (A + B * x)) ** 2 for x, y in zip(xs, ys))
    return A, B, (1.0 - ss_res / ss_tot) if ss_tot else 1.0


def ceiling_bench(args):
    """Sustained bf16 dense MFMA rate on an MFMA-bound plain GEMM (M = N = K =
    --ceiling-size, N(0,1) operands, so the matrix units see realistic bit
    patterns): the library's projection GEMM and torch.matmul (hipBLASLt),
    each launched back to back for --ceiling-seconds of wall time after a
    warm-up, so that the chip reaches its sustained (power-limited) clock."""
    import torch
    from paper_2602_21196_amd import upipe
    n = args.ceiling_size
    g = torch.Generator().manual_seed(77)
    a = torch.randn((n, n), generator=g).to(torch.bfloat16).to("cuda:0")
    b = torch.randn((n, n), generator=g).to(torch.bfloat16).to("cuda:0")
    c = torch.empty((n, n), dtype=torch.bfloat16, device="cuda:0")
    flops = 2.0 * n * n * n
    st = torch.cuda.current_stream().cuda_stream
    pa, pb, pc = a.data_ptr(), b.data_ptr(), c.data_ptr()

    def ours():
        if upipe.upipe_gemm_bf16(pa, pb, pc, n, n, n, st) != 0:
            raise RuntimeError("upipe_gemm_bf16 failed")

    def blas():
        torch.matmul(a, b, out=c)

    res = {}
    for name, fn in (("upipe_gemm_bf16", ours), ("torch.matmul (hipBLASLt)", blas)):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        # launches per second from a short probe, then one timed run of the
        # requested length (no host sync inside)
        t0 = time.perf_counter()
        for _ in range(10):
            fn()
        torch.cuda.synchronize()
        per = (time.perf_counter() - t0) / 10
        reps = max(10, int(args.ceiling_seconds / per))
        t0 = time.perf_counter()
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        res[name] = {"tflops": round(flops * reps / el / 1e12, 1), "launches": reps,
                     "seconds": round(el, 2), "ms_per_launch": round(el / reps * 1e3, 3),
                     "frac_of_peak": round(flops * reps / el / 1e12 / PEAK_BF16_TFLOPS, 4)}
    best = max(v["tflops"] for v in res.values())
    out = {"metric": "sustained bf16 dense GEMM TFLOP/s per MI355X (attainable MFMA ceiling)",
           "value": best, "unit": "TFLOP/s", "n_gpus": 1, "higher_is_better": True,
           "dtype": "bf16", "data": "synthetic N(0,1)",
           "config": {"workload": f"gemm M=N=K={n}", "seconds_per_kernel": args.ceiling_seconds},
           "peak": PEAK_BF16_TFLOPS, "frac_of_peak": round(best / PEAK_BF16_TFLOPS, 4),
           "kernels": res}
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: this library has no multi-GPU "
              f"path (asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)
    if args.ceiling:
        return ceiling_bench(args)
    import torch
    import workloads as W
    from paper_2602_21196_amd import upipe

    w = W.WORKLOADS[args.workload]
    if w.extra.get("ring"):
        return ring_bench(args, w)
    dev = "cuda:0"
    S, Hq, Hkv, d, U, B = w.S, w.Hq, w.Hkv, w.d, args.U, args.batch
    fwd_flops, bwd_flops = W.attention_flops(S, Hq, d)
    step_flops = B * (fwd_flops + bwd_flops)
    if w.is_layer:
        dm = w.d_model
        if B == 1:
            x, wqkv, wo, dy = (t.to(dev) for t in W.inputs_for(w))
        else:
            x, wqkv, wo, dy = (t.to(dev) for t in
                               W.batch_layer_inputs(S, dm, Hq, Hkv, d, w.seed, B))
        proj_fwd = 2 * S * dm * (Hq + 2 * Hkv) * d + 2 * S * Hq * d * dm
        step_flops += 3 * proj_fwd * B
        ws_f = upipe.workspace(upipe.upipe_layer_fwd_workspace_size(S, dm, Hq, Hkv, d, U), dev)
        ws_b = upipe.workspace(upipe.upipe_layer_bwd_workspace_size(S, dm, Hq, Hkv, d, U), dev)

        rope_base = (args.rope_base if args.rope_base is not None
                     else w.extra.get("rope_base", 0.0))

        full_ac = args.checkpointing == "full"
        # Tensors the forward leaves for the backward besides x and the
        # weights: the attention output and its lse under selective
        # checkpointing, nothing under full checkpointing.
        kept_bytes = 0 if full_ac else B * (2 * S * Hq * d + 4 * Hq * S)

        def step():
            y, o, lse = upipe.layer_fwd(x, wqkv, wo, Hq, Hkv, d, U=U, ws=ws_f,
                                        rope_base=rope_base)
            if full_ac:
                o = lse = None
            upipe.layer_bwd(x, wqkv, wo, o, lse, dy, Hq, Hkv, d, U=U, ws=ws_b,
                            rope_base=rope_base)
    else:
        if B == 1:
            q, k, v, do = W.attention_inputs(S, Hq, Hkv, d, w.seed)
        else:
            q, k, v, do = W.batch_attention_inputs(S, Hq, Hkv, d, w.seed, B)
        qd, kd, vd, dod = (t.to(dev) for t in (q, k, v, do))
        ws_f = upipe.workspace(upipe.upipe_attn_fwd_workspace_size(S, Hq, Hkv, d, U), dev)
        ws_b = upipe.workspace(upipe.upipe_attn_bwd_workspace_size(S, Hq, Hkv, d, U), dev)

        def step():
            o, lse = upipe.attn_fwd(qd, kd, vd, causal=True, U=U, ws=ws_f)
            upipe.attn_bwd(qd, kd, vd, o, lse, dod, causal=True, U=U, ws=ws_b)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        # progress on stderr (a long workload runs for minutes before its line)
        print(f"bench: warmup step {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)
    upipe.upipe_profile_reset()
    upipe.upipe_profile_enable(1)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    upipe.upipe_profile_enable(0)
    ms_per_step = elapsed / args.steps * 1e3
    value = step_flops / (elapsed / args.steps) / 1e12

    full_ckpt = w.is_layer and args.checkpointing == "full"
    kflops = kernel_flops(S, Hq, B, d, fwd_passes=2 if full_ckpt else 1)
    kernels = {}
    for name in upipe.upipe_profile_names():
        n, ms = upipe.upipe_profile_query(name)
        if n == 0:
            continue
        entry = {"launches_per_step": n // args.steps,
                 "ms_per_step": round(ms / args.steps, 4),
                 "avg_launch_ms": round(ms / n, 4)}
        if name in kflops:
            entry["tflops"] = round(kflops[name] / (ms / args.steps / 1e3) / 1e12, 2)
        kernels[name] = entry
    dom = max(kernels, key=lambda n: kernels[n]["ms_per_step"])
    achieved = kernels[dom].get("tflops")
    roofline = {"kernel": dom, "bound": "mfma",
                "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4) if achieved else None,
                "traffic": (measured_traffic(dom, w.name, U)
                            if dom in KERNEL_SOURCES else None),
                "traffic_unit": "bytes per launch",
                "clock_ghz_est": (measured_clock(dom, w.name, U)
                                  if dom in KERNEL_SOURCES else None),
                "clock_note": "sustained shader clock under this kernel (rocprofv3 "
                              "GRBM_COUNT / duration / 8 XCDs, profiles/clock.json); "
                              "the peak assumes 2.4 GHz"}
    upipe.upipe_profile_reset()

    out = {"metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s",
           "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(ms_per_step, 3), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic",
           "config": {"workload": w.name, "S": S, "Hq": Hq, "Hkv": Hkv,
                      "d": d, "U": U, "causal": True, "seed": w.seed, "batch": B,
                      **({"d_model": w.d_model, "rope_base": rope_base,
                          "checkpointing": args.checkpointing} if w.is_layer else {})},
           "frac_of_peak": round(value / PEAK_BF16_TFLOPS, 4),
           "roofline": roofline, "kernels": kernels}
    if w.is_layer:
        out["layer_memory_gb"] = {
            "kept_for_backward": round(kept_bytes / 1e9, 4),
            "fwd_workspace": round(upipe.upipe_layer_fwd_workspace_size(S, w.d_model, Hq, Hkv,
                                                                         d, U) / 1e9, 4),
            "bwd_workspace": round(upipe.upipe_layer_bwd_workspace_size(S, w.d_model, Hq, Hkv,
                                                                         d, U) / 1e9, 4)}

    if not args.no_sweep and w.is_layer and B == 1:
        del ws_f, ws_b
        torch.cuda.synchronize()
        out.update(layer_sweep(args, w, x, wqkv, wo, dy, rope_base, step_flops))

    if not args.no_sweep and not w.is_layer and B == 1:
        del ws_f, ws_b
        torch.cuda.synchronize()
        # outputs of one fwd+bwd: o, dq [S,Hq,d] bf16, dk, dv [S,Hkv,d] bf16,
        # lse [Hq,S] fp32; everything else allocated in between is workspace.
        out_bytes = 2 * (2 * S * Hq * d) + 2 * (2 * S * Hkv * d) + 4 * Hq * S
        sweep_mem, sweep_tf = {}, {}
        for u in w.U_sweep:
            torch.cuda.empty_cache()
            torch.cuda.reset_peak_memory_stats()
            base = torch.cuda.memory_allocated()
            o, lse = upipe.attn_fwd(qd, kd, vd, U=u)
            g = upipe.attn_bwd(qd, kd, vd, o, lse, dod, U=u)
            torch.cuda.synchronize()
            peak = torch.cuda.max_memory_allocated() - base
            sweep_mem[str(u)] = round((peak - out_bytes) / 1e9, 4)
            del o, lse, g
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            for _ in range(2):
                o, lse = upipe.attn_fwd(qd, kd, vd, U=u)
                g = upipe.attn_bwd(qd, kd, vd, o, lse, dod, U=u)
            torch.cuda.synchronize()
            sweep_tf[str(u)] = round(step_flops / ((time.perf_counter() - t1) / 2) / 1e12, 2)
            del o, lse, g
        out["peak_activation_gb_vs_U"] = sweep_mem
        out["peak_activation_model_gb_vs_U"] = {
            str(u): round(workspace_model_gb(S, Hq, Hkv, d, u), 4) for u in w.U_sweep}
        us = [int(u) for u in sweep_mem]
        fit_a, fit_b, r2 = linear_fit(us, [sweep_mem[str(u)] for u in us])
        out["peak_activation_fit"] = {"A_gb": round(fit_a, 4), "B_gb_per_U": round(fit_b, 4),
                                      "r2": round(r2, 4)}
        out["peak_activation_note"] = (
            "max_memory_allocated during one fwd+bwd above the resident "
            "inputs, minus the outputs o, lse, dq, dk, dv: the workspaces; "
            "the model drops the fp32 dK/dV carries once U is a multiple of "
            "the group size, so the fit over all U is not exactly linear")
        out["tflops_vs_U"] = sweep_tf

    if not args.no_cpu_baseline and not w.is_layer and B == 1:
        out["cpu_baseline"] = cpu_baseline(w, q, k, v, do, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def layer_sweep(args, w, x, wqkv, wo, dy, rope_base, step_flops):
    """Throughput and peak activation memory of the layer share for every U.

    Peak = torch.cuda.max_memory_allocated over one forward + backward above
    the resident inputs (x, weights, dY), minus the caller-owned outputs (y,
    final_out, lse, dX, dWqkv, dWo): the two workspaces and the kept
    attention output's lifetime overlap, as a training step would see them.
    Only the U-dependent chunk buffers change with U (per chunk head the
    projected Q, the recomputed output and the fp32 lse, D rows), and the
    dK/dV fp32 carries while a key/value group spans chunks."""
    import torch
    from paper_2602_21196_amd import upipe
    S, Hq, Hkv, d, dm = w.S, w.Hq, w.Hkv, w.d, w.d_model
    full_ac = args.checkpointing == "full"
    out_bytes = 2 * S * dm + 2 * S * Hq * d + 4 * Hq * S + 2 * S * dm + \
        2 * dm * (Hq + 2 * Hkv) * d + 2 * Hq * d * dm
    mem, tf, ws = {}, {}, {}
    for u in w.U_sweep:
        torch.cuda.empty_cache()
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        y, o, lse = upipe.layer_fwd(x, wqkv, wo, Hq, Hkv, d, U=u, rope_base=rope_base)
        g = upipe.layer_bwd(x, wqkv, wo, None if full_ac else o, None if full_ac else lse, dy,
                            Hq, Hkv, d, U=u, rope_base=rope_base)
        torch.cuda.synchronize()
        mem[str(u)] = round((torch.cuda.max_memory_allocated() - base - out_bytes) / 1e9, 4)
        ws[str(u)] = {"fwd": round(upipe.upipe_layer_fwd_workspace_size(S, dm, Hq, Hkv, d, u)
                                   / 1e9, 4),
                      "bwd": round(upipe.upipe_layer_bwd_workspace_size(S, dm, Hq, Hkv, d, u)
                                   / 1e9, 4)}
        del y, o, lse, g
        wf = upipe.workspace(upipe.upipe_layer_fwd_workspace_size(S, dm, Hq, Hkv, d, u), "cuda:0")
        wb = upipe.workspace(upipe.upipe_layer_bwd_workspace_size(S, dm, Hq, Hkv, d, u), "cuda:0")
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(2):
            y, o, lse = upipe.layer_fwd(x, wqkv, wo, Hq, Hkv, d, U=u, ws=wf, rope_base=rope_base)
            g = upipe.layer_bwd(x, wqkv, wo, None if full_ac else o, None if full_ac else lse,
                                dy, Hq, Hkv, d, U=u, ws=wb, rope_base=rope_base)
        torch.cuda.synchronize()
        tf[str(u)] = round(step_flops / ((time.perf_counter() - t1) / 2) / 1e12, 2)
        del y, o, lse, g, wf, wb
    us = [int(u) for u in mem]
    fit_a, fit_b, r2 = linear_fit(us, [mem[str(u)] for u in us])
    return {"peak_activation_gb_vs_U": mem, "workspace_gb_vs_U": ws,
            "peak_activation_fit": {"A_gb": round(fit_a, 4), "B_gb_per_U": round(fit_b, 4),
                                    "r2": round(r2, 4)},
            "peak_activation_note": (
                "max_memory_allocated during one layer fwd+bwd above the resident "
                "inputs, minus the outputs y, final_out, lse, dX, dWqkv, dWo"),
            "tflops_vs_U": tf}


def ring_cpu_baseline(w, q, k, v, delta, target_s):
    """Oracle ring step (float64 numpy) on a bounded block: the first n query
    rows against the first n keys at the workload's offsets, one query head."""
    import numpy as np
    from oracle import ring as R
    import workloads as W

    def run(n):
        f = lambda t, m: t[:m, :1].float().double().numpy()  # noqa: E731
        args = (f(q, n), f(k, n), f(v, n))
        t0 = time.perf_counter()
        R.attn_fwd_offset(*args, delta, True)
        return time.perf_counter() - t0

    n = 1024
    t = run(n)
    for _ in range(4):
        if t >= 0.6 * target_s or n >= min(w.S, w.extra["kv_len"]):
            break
        n = int(min(w.S, w.extra["kv_len"], max(n + 128, n * (target_s / max(t, 1e-3)) ** 0.5)))
        t = run(n)
    pairs = W.ring_pairs(n, n, delta)
    cores, blas, cpu = host_info()
    return {"value": round(4 * w.d * pairs / t / 1e12, 6), "unit": "TFLOP/s", "cores": cores,
            "kind": "oracle", "blas": blas, "cpu": cpu,
            "sample": f"first {n} query rows x first {n} keys of {w.name}, 1 query head, "
                      f"ring-step forward, float64 numpy, {t:.1f} s"}


def ring_bench(args, w):
    """One ring step (query block against one key/value block at its offset)
    plus the merge of its partial result into the running one."""
    import torch
    import workloads as W
    from paper_2602_21196_amd import upipe
    dev = "cuda:0"
    Sq, Skv, Hq, Hkv, d, U = w.S, w.extra["kv_len"], w.Hq, w.Hkv, w.d, args.U
    qo, ko = w.extra["q_offset"], w.extra["kv_offset"]
    q, k, v = W.inputs_for(w)
    qd, kd, vd = (t.to(dev) for t in (q, k, v))
    ws = upipe.workspace(upipe.upipe_attn_fwd_ring_workspace_size(Sq, Skv, Hq, Hkv, d, U), dev)
    # the running result before this step: the query block's own causal block
    o_acc, lse_acc = upipe.attn_fwd_ring(qd, qd[:, :Hkv].contiguous(), qd[:, :Hkv].contiguous(),
                                         qo, qo, causal=True, U=U)
    flops = 4 * d * Hq * W.ring_pairs(Sq, Skv, qo - ko)

    def step():
        o_p, lse_p = upipe.attn_fwd_ring(qd, kd, vd, qo, ko, causal=True, U=U, ws=ws)
        upipe.lse_merge(o_acc, lse_acc, o_p, lse_p)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    upipe.upipe_profile_reset()
    upipe.upipe_profile_enable(1)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    upipe.upipe_profile_enable(0)
    kernels = {}
    for name in upipe.upipe_profile_names():
        n, ms = upipe.upipe_profile_query(name)
        if n:
            kernels[name] = {"launches_per_step": n // args.steps,
                             "ms_per_step": round(ms / args.steps, 4),
                             "avg_launch_ms": round(ms / n, 4)}
    upipe.upipe_profile_reset()
    fw = kernels.get("attn_fwd", {})
    fwd_tf = flops / (fw["ms_per_step"] * 1e-3) / 1e12 if fw else None
    if fw:
        fw["tflops"] = round(fwd_tf, 2)
    mg = kernels.get("lse_merge")
    merge_bytes = 3 * Sq * Hq * d * 2 + 3 * Hq * Sq * 4    # o, o_p read, o written; lse likewise
    if mg:
        mg["gb_per_s"] = round(merge_bytes / (mg["avg_launch_ms"] * 1e-3) / 1e9, 1)
    value = flops / (elapsed / args.steps) / 1e12
    out = {"metric": "ring step: attention forward over one key/value block + LSE merge, "
                     "TFLOP/s per MI355X",
           "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(elapsed / args.steps * 1e3, 3),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic",
           "config": {"workload": w.name, "Sq": Sq, "Skv": Skv, "q_offset": qo,
                      "kv_offset": ko, "Hq": Hq, "Hkv": Hkv, "d": d, "U": U, "causal": True,
                      "seed": w.seed},
           "frac_of_peak": round(value / PEAK_BF16_TFLOPS, 4),
           "roofline": {"kernel": "attn_fwd", "bound": "mfma",
                        "achieved": round(fwd_tf, 2) if fwd_tf else None,
                        "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                        "frac": round(fwd_tf / PEAK_BF16_TFLOPS, 4) if fwd_tf else None,
                        "traffic": None, "traffic_unit": "bytes per launch"},
           "merge_roofline": {"kernel": "lse_merge", "bound": "hbm",
                              "achieved": mg["gb_per_s"] if mg else None, "peak": PEAK_HBM_GBS,
                              "unit": "GB/s",
                              "frac": round(mg["gb_per_s"] / PEAK_HBM_GBS, 4) if mg else None,
                              "bytes_per_launch": merge_bytes},
           "kernels": kernels}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = ring_cpu_baseline(w, q, k, v, qo - ko, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
