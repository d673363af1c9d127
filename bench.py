"""Benchmark of the LCE hot path (forward + backward) on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload llama8b] [--no-cpu-baseline]
                [--variant lce|adamw_fused|adamw_two_phase|vocab_shard|kd|kd_fused] [--shards 8]

One step is one lce_forward + lce_backward (which reuses the valid-row list and
gathered rows the forward left in the shared workspace) over the whole batch of the named
workload (default: the Llama-3.1-8B vocabulary head, N = 8 x 2048 tokens,
D = 4096, V = 128256, 25% of targets masked). Inputs are seeded synthetic
tensors already resident in HBM; outputs and workspace are allocated once
before the timed region. The script prints one JSON line on stdout.

The optimizer variants add one AdamW step on W per step (paper Sec. 4.1):
``adamw_fused`` runs lce_forward + lce_backward_adamw (the step inside the
backward, no dW buffer), ``adamw_two_phase`` runs lce_forward + lce_backward +
lce_adamw_step (the standard path). Both keep fp32 moments and an fp32 master
copy of W.

``vocab_shard`` times one device's share of G-way vocabulary parallelism (loss
parallel, paper Sec. 5): lce_forward_shard + lce_combine_shards +
lce_backward_shard on N tokens x V/G ids (shard 0). The [G, N] partials that
an all-gather would bring from the other devices are stood in for by copies of
this shard's own, and no collective runs; the line reports N / step time, the
whole job's rate when G devices each run their share in parallel.

``kd`` times the fused linear knowledge-distillation loss (lce_kd_forward +
lce_kd_backward, temperature 2) distilling the Llama-3.1-8B head (teacher,
D = 4096) into the Llama-3.2-1B head (student, D = 2048) over 8 x 2048 tokens;
its MFMA work per step is 6 Nv V Dt + 10 Nv V Ds (teacher statistics and two
probability passes; student statistics, Q pass, G recompute, dW and dH).
``kd_fused`` runs the same step as one lce_kd_forward_backward call: 4 Nv V Dt
+ 8 Nv V Ds (one teacher probability pass, one student pass for G and Q).

Two diagnostics put the contractions' rate in context; neither is the benchmark:
``--data zeros`` runs the same launches on all-zero H and W (the workload's targets and mask),
so that the operands toggle no bits and the chip's power limit holds its clock near the maximum;
``--gemm-reference`` times torch.matmul (the vendor BLAS) on the forward's logits product,
[Nv, D] x [D, V] in bf16, with the workload's data, and prints its own JSON line instead.
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

PEAK_BF16_TFLOPS = 2500.0        # MI355X dense bf16 MFMA peak
PEAK_HBM_GBS = 8000.0
METRIC = "LCE fwd+bwd tokens/sec, % bf16 MFMA peak, peak HBM bytes (1 GPU)"
GEMM_KERNELS = ("fwd_stats", "bwd_g", "bwd_dw", "bwd_dh")


def _cpu_baseline(inp, seconds_target=10.0):
    """The CPU oracle, as it stands, on a bounded sample of the workload's tokens."""
    from oracle import lce_oracle as O
    try:
        import threadpoolctl
        threads = max(i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()) or 1
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    valid = np.nonzero(inp.targets != inp.ignore_index)[0]
    # double the token sample until one oracle run takes at least `seconds_target`
    sample = 32
    while True:
        t0 = time.perf_counter()
        O.lce(inp.h_bits[valid[:sample]], inp.w_bits, inp.targets[valid[:sample]])
        dt = time.perf_counter() - t0
        if dt >= seconds_target or sample >= len(valid):
            break
        sample = min(len(valid), max(2 * sample, int(sample * 1.2 * seconds_target / max(dt, 1e-3))))
    return {"value": sample / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{sample} valid tokens of the {inp.workload.name} batch, full D and V, "
                      f"fp64 forward+backward ({dt:.1f} s)"}


def _host_info():
    """The host the CPU oracle ran on: CPU model, cores visible to this process, BLAS build."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), None)
    except OSError:  # pragma: no cover
        pass
    try:
        blas = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        blas = f"{blas.get('name')} {blas.get('version')}"
    except Exception:  # pragma: no cover
        blas = None
    return {"cpu_model": model, "affinity_cores": len(os.sched_getaffinity(0)), "os_cpu_count": os.cpu_count(),
            "blas": blas}


def _event_summary(events):
    """Median / min step time and the median forward and backward parts, from per-step
    (start, after forward, end) events recorded on the stream the step runs on."""
    steps = [a.elapsed_time(c) for a, _, c in events]
    fwd = [a.elapsed_time(b) for a, b, _ in events]
    bwd = [b.elapsed_time(c) for _, b, c in events]
    return {"median": float(np.median(steps)), "min": float(np.min(steps)),
            "fwd_median": float(np.median(fwd)), "bwd_median": float(np.median(bwd))}


def _copy_calibration(gib=1.0, reps=3):
    """A plain device copy of a known size, for scaling the HBM byte counters (FETCH_SIZE,
    WRITE_SIZE) of a profiled run: each copy reads and writes exactly `gib` GiB."""
    import torch
    n = int(gib * (1 << 30))
    a = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_per_launch": n, "launches": reps}), flush=True)


def _gemm_reference(args, wl, h, w, inp):
    """torch.matmul of the valid rows of H by W^T ([Nv, D] x [D, V] -> [Nv, V] bf16): the forward's
    logits product as one plain library GEMM, timed with HIP events over `steps` launches. It
    materialises the logits, which the LCE path never does; it is a yardstick, not a step."""
    import torch
    valid = torch.from_numpy(np.flatnonzero(inp.targets != inp.ignore_index)).to(h.device)
    hv = h.index_select(0, valid).contiguous()
    out = torch.empty((hv.shape[0], w.shape[0]), dtype=torch.bfloat16, device=h.device)
    for _ in range(args.warmup):
        torch.matmul(hv, w.t(), out=out)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        torch.matmul(hv, w.t(), out=out)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    tflops = 2.0 * hv.shape[0] * wl.d * wl.v / (ms * 1e-3) / 1e12
    print(json.dumps({"metric": "bf16 GEMM rate of torch.matmul on the forward logits product (context)",
                      "value": tflops, "unit": "TFLOP/s", "frac": tflops / PEAK_BF16_TFLOPS, "ms": ms,
                      "steps": args.steps, "warmup": args.warmup,
                      "shape": {"m": int(hv.shape[0]), "n": wl.v, "k": wl.d},
                      "data": "synthetic" if args.data == "random" else "synthetic, all-zero H and W",
                      "config": {"workload": wl.name}}), flush=True)


def _source_hash():
    import hashlib
    src = os.path.join(ROOT, "paper_2605_21442_amd", "csrc", "lce.hip")
    return hashlib.sha256(open(src, "rb").read()).hexdigest()


def _kernel_breakdown(B, step, steps):
    """Per-kernel totals over `steps` more steps with the library's per-launch HIP events on (a pass
    of its own, so that the headline's timed region carries no extra events)."""
    import torch
    torch.cuda.synchronize()
    B.lce_timing_enable(True)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    kernels = {}
    for k, name in enumerate(B.lce_timing_kernel_names()):
        ms, cnt = B.lce_timing_read(k)
        if cnt:
            kernels[name] = {"total_ms": ms, "launches": cnt, "avg_ms": ms / cnt}
    B.lce_timing_enable(False)
    return kernels, steps


def _traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed counter summary of `workload`, or None
    when there is none or it was taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("lce.hip sha256") != _source_hash():
        return None
    key = f"{kernel} bytes per launch"
    return float(kv[key]) if key in kv else None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama8b")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--variant", default="lce",
                    choices=("lce", "adamw_fused", "adamw_two_phase", "vocab_shard", "kd", "kd_fused"))
    ap.add_argument("--shards", type=int, default=8, help="vocabulary shards (vocab_shard variant)")
    ap.add_argument("--data", default="random", choices=("random", "zeros"),
                    help="zeros: all-zero H and W, a power diagnostic (not the benchmark)")
    ap.add_argument("--gemm-reference", action="store_true",
                    help="time only torch.matmul on the forward logits product, for context")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a 1 GiB device copy (for scaling HBM byte counters)")
    args = ap.parse_args()
    if args.copy_calibration:
        _copy_calibration()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}); the LCE path here has no "
              f"multi-GPU mode", file=sys.stderr)
        sys.exit(2)

    if args.variant in ("kd", "kd_fused"):
        bench_kd(args, fused=args.variant == "kd_fused")
        return

    import torch
    from paper_2605_21442_amd import binding as B
    from paper_2605_21442_amd import workloads as WL

    wl = WL.WORKLOADS[args.workload]
    t_gen = time.perf_counter()
    inp = WL.generate(wl, args.seed)
    print(f"[bench] {wl.name}: N={wl.n} D={wl.d} V={wl.v} Nv={wl.n_valid()} "
          f"(inputs drawn in {time.perf_counter() - t_gen:.1f} s)", file=sys.stderr, flush=True)
    dev = torch.device("cuda:0")
    h = torch.from_numpy(inp.h_bits.view(np.int16)).view(torch.bfloat16).to(dev)
    sharded = args.variant == "vocab_shard"
    # shard 0 of the vocabulary-parallel variant holds ids [0, ceil(V / G)); only its rows go to the GPU
    v_rows = (wl.v + args.shards - 1) // args.shards if sharded else wl.v
    w = torch.from_numpy(inp.w_bits[:v_rows].view(np.int16)).view(torch.bfloat16).to(dev)
    t = torch.from_numpy(inp.targets).to(dev)
    if args.data == "zeros":
        h.zero_()
        w.zero_()
    n, d, v = wl.n, wl.d, wl.v
    if args.gemm_reference:
        _gemm_reference(args, wl, h, w, inp)
        return
    v_total = v
    if sharded:
        v = v_rows
        shard = B.LceShard(v_total, 0)
        p_full = B.problem(n, d, v_total, ignore_index=inp.ignore_index, reduction="mean", target_bytes=4)
        comb_bytes, _ = B.lce_workspace_size(p_full)
    p = B.problem(n, d, v, ignore_index=inp.ignore_index, reduction="mean", target_bytes=4)
    # the backward reuses the valid-row list and gathered rows the forward left in the workspace
    pb = B.problem(n, d, v, ignore_index=inp.ignore_index, reduction="mean", target_bytes=4,
                   flags=B.LCE_FLAG_REUSE_FORWARD)
    fwd_bytes, bwd_bytes = B.lce_workspace_size(p)
    if sharded:
        fwd_bytes = max(fwd_bytes, comb_bytes)
    torch.cuda.synchronize()
    base_alloc = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()

    loss = torch.empty((), dtype=torch.float32, device=dev)
    lse = torch.empty(n, dtype=torch.float32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    grad = torch.ones(1, dtype=torch.float32, device=dev)
    dh = torch.empty((n, d), dtype=torch.bfloat16, device=dev)
    fused = args.variant == "adamw_fused"
    dw = None if fused else torch.empty((v, d), dtype=torch.bfloat16, device=dev)
    if sharded:
        dh = torch.empty((n, d), dtype=torch.float32, device=dev)      # this shard's fp32 dH term
        lse_part = torch.empty(n, dtype=torch.float32, device=dev)
        tgt_part = torch.empty(n, dtype=torch.float32, device=dev)
        lse_parts = torch.empty((args.shards, n), dtype=torch.float32, device=dev)
        tgt_parts = torch.empty((args.shards, n), dtype=torch.float32, device=dev)
    ws = torch.empty(max(fwd_bytes, bwd_bytes), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    opt_ptrs = None
    if args.variant != "lce":
        m1 = torch.zeros((v, d), dtype=torch.float32, device=dev)
        m2 = torch.zeros((v, d), dtype=torch.float32, device=dev)
        master = w.float()
        opt_ptrs = (m1.data_ptr(), m2.data_ptr(), master.data_ptr())
        step_no = [0]

    def adamw():
        step_no[0] += 1
        return B.adamw(1e-5, 0.9, 0.95, 1e-8, 0.1, step_no[0])

    def shard_step(mid=None):
        B.lce_forward_shard(p, shard, h.data_ptr(), w.data_ptr(), t.data_ptr(), lse_part.data_ptr(),
                            tgt_part.data_ptr(), nv.data_ptr(), status.data_ptr(), ws.data_ptr(), fwd_bytes, stream)
        # stand-in for the all-gather of every shard's partials
        lse_parts.copy_(lse_part.expand(args.shards, n))
        tgt_parts.copy_(tgt_part.expand(args.shards, n))
        B.lce_combine_shards(p_full, args.shards, lse_parts.data_ptr(), tgt_parts.data_ptr(), t.data_ptr(),
                             loss.data_ptr(), lse.data_ptr(), nv.data_ptr(), status.data_ptr(), ws.data_ptr(),
                             fwd_bytes, stream)
        if mid is not None:
            mid.record()
        B.lce_backward_shard(pb, shard, h.data_ptr(), w.data_ptr(), t.data_ptr(), lse.data_ptr(), nv.data_ptr(),
                             grad.data_ptr(), dh.data_ptr(), dw.data_ptr(), ws.data_ptr(), bwd_bytes, stream)

    def step(mid=None):
        if sharded:
            shard_step(mid)
            return
        B.lce_forward(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), loss.data_ptr(), lse.data_ptr(),
                      nv.data_ptr(), status.data_ptr(), ws.data_ptr(), fwd_bytes, stream)
        if mid is not None:
            mid.record()
        if fused:
            B.lce_backward_adamw(pb, h.data_ptr(), w.data_ptr(), t.data_ptr(), lse.data_ptr(), nv.data_ptr(),
                                 grad.data_ptr(), dh.data_ptr(), *opt_ptrs, adamw(), ws.data_ptr(), bwd_bytes,
                                 stream)
            return
        B.lce_backward(pb, h.data_ptr(), w.data_ptr(), t.data_ptr(), lse.data_ptr(), nv.data_ptr(),
                       grad.data_ptr(), dh.data_ptr(), dw.data_ptr(), ws.data_ptr(), bwd_bytes, stream)
        if opt_ptrs is not None:
            B.lce_adamw_step(v, d, 0, w.data_ptr(), dw.data_ptr(), *opt_ptrs, adamw(), stream)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        print(f"[bench] warmup {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)
    peak = torch.cuda.max_memory_allocated()
    # inputs, outputs and (optimizer variants) the optimizer state; dW only where it exists
    def nbytes(x):
        return x.numel() * x.element_size() if x is not None else 0
    resident = nbytes(h) + nbytes(w) + nbytes(t) + nbytes(dh) + nbytes(dw) + n * 4 \
        + (3 * v * d * 4 if opt_ptrs is not None else 0)

    # the headline: K steps with no per-kernel events in the stream
    events = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1, e2 in events:
        e0.record()
        step(e1)
        e2.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    print(f"[bench] timed {args.steps} steps in {elapsed:.3f} s; loss={loss.item():.6f} "
          f"Nv={int(nv.item())}", file=sys.stderr, flush=True)
    # a second pass, after the timed region: per-kernel launch times from HIP events that the
    # library records on the launch stream around each of its kernels
    kernels, kpass = _kernel_breakdown(B, step, args.steps)

    nvalid = int(nv.item())
    ms_step = elapsed * 1e3 / args.steps
    flops_step = 8.0 * nvalid * d * v
    dom = max((k for k in kernels if k in GEMM_KERNELS), key=lambda k: kernels[k]["total_ms"])
    launches_per_step = kernels[dom]["launches"] / kpass
    flops_launch = 2.0 * nvalid * d * v / launches_per_step
    achieved = flops_launch / (kernels[dom]["avg_ms"] * 1e-3) / 1e12
    for k, r in sorted(kernels.items(), key=lambda kv: -kv[1]["total_ms"]):
        extra = ""
        if k in GEMM_KERNELS:
            tf = 2.0 * nvalid * d * v / (r["launches"] / kpass) / (r["avg_ms"] * 1e-3) / 1e12
            extra = f" {tf:7.1f} TFLOP/s ({100 * tf / PEAK_BF16_TFLOPS:4.1f}% of peak)"
        print(f"[bench]   {k:12s} {r['total_ms'] / kpass:8.3f} ms/step  {r['launches']:5d} launches"
              f"  avg {r['avg_ms']:.4f} ms{extra}", file=sys.stderr)

    out = {
        "metric": METRIC,
        "value": n * args.steps / elapsed,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic" if args.data == "random" else "synthetic, all-zero H and W (power diagnostic)",
        "config": {"workload": wl.name, "n_tokens": n, "hidden": d, "vocab": v, "n_valid": nvalid,
                   "global_batch": wl.batch, "seq_len": wl.seq_len, "parallelism": "none",
                   "reduction": "mean", "ignore_index": inp.ignore_index, "variant": args.variant,
                   **({"shards": args.shards, "vocab_total": v_total} if sharded else {})},
        "valid_tokens_per_s": nvalid * args.steps / elapsed,
        "mfma_frac_step": flops_step / (ms_step * 1e-3) / (PEAK_BF16_TFLOPS * 1e12),
        # the same step counted without the backward's recompute of the logits (6 Nv D V)
        "mfma_frac_step_no_recompute": 0.75 * flops_step / (ms_step * 1e-3) / (PEAK_BF16_TFLOPS * 1e12),
        "step_ms": _event_summary(events),
        "peak_hbm_bytes": int(peak),
        "peak_hbm_bytes_transient": int(peak - resident),
        "workspace_bytes": int(max(fwd_bytes, bwd_bytes)),
        "logits_bytes_avoided_fp32": int(n) * int(v) * 4,
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS, "traffic": _traffic(dom, wl.name) if args.variant == "lce" else None,
                     "flops_per_launch": flops_launch, "avg_launch_ms": kernels[dom]["avg_ms"]},
        "kernels_ms_per_step": {k: r["total_ms"] / kpass for k, r in kernels.items()},
        "kernel_timing": f"second pass of {kpass} steps after the timed region, HIP events around each launch",
        "lce_hip_sha256": _source_hash(),
    }
    if not args.no_cpu_baseline and args.data == "random":
        print("[bench] timing the CPU oracle on a token sample ...", file=sys.stderr, flush=True)
        out["cpu_baseline"] = _cpu_baseline(inp)
        out["host"] = _host_info()
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


def _kd_cpu_baseline(inp, temperature, seconds_target=10.0):
    """The KD oracle, as it stands, on a bounded token sample (forward + backward)."""
    from oracle import kd_oracle as K
    try:
        import threadpoolctl
        threads = max(i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()) or 1
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    valid = np.nonzero(inp.targets != inp.ignore_index)[0]
    sample = 16
    while True:
        r = valid[:sample]
        t0 = time.perf_counter()
        K.kd_bits(inp.hs_bits[r], inp.ws_bits, inp.ht_bits[r], inp.wt_bits, inp.targets[r], temperature=temperature)
        dt = time.perf_counter() - t0
        if dt >= seconds_target or sample >= len(valid):
            break
        sample = min(len(valid), max(2 * sample, int(sample * 1.2 * seconds_target / max(dt, 1e-3))))
    return {"value": sample / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{sample} valid tokens of the {inp.name} batch, full Ds, Dt and V, fp64 KD "
                      f"forward+backward ({dt:.1f} s)"}


def bench_kd(args, fused=False):
    """The KD variants: one step = lce_kd_forward + lce_kd_backward (or one lce_kd_forward_backward)
    on the 8B-to-1B heads."""
    import torch
    from paper_2605_21442_amd import binding as B
    from paper_2605_21442_amd import workloads as WL

    name, T = "kd_8b_to_1b", 2.0
    inp = WL.kd_generate(name, args.seed)
    k = WL.KD_WORKLOADS[name]
    n, ds, dt, v = k["n"], k["ds"], k["dt"], k["v"]
    dev = torch.device("cuda:0")
    to = lambda b: torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).to(dev)
    hs, ws, ht, wt = to(inp.hs_bits), to(inp.ws_bits), to(inp.ht_bits), to(inp.wt_bits)
    t = torch.from_numpy(inp.targets).to(dev)
    p = B.kd_problem(n, ds, dt, v, temperature=T, ignore_index=inp.ignore_index)
    fwd_bytes, bwd_bytes = B.lce_kd_workspace_size(p)
    if fused:
        fwd_bytes = bwd_bytes = B.lce_kd_workspace_size_fused(p)
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    loss = torch.empty((), dtype=torch.float32, device=dev)
    lse_s = torch.empty(n, dtype=torch.float32, device=dev)
    lse_t = torch.empty(n, dtype=torch.float32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    grad = torch.ones(1, dtype=torch.float32, device=dev)
    dh = torch.empty((n, ds), dtype=torch.bfloat16, device=dev)
    dw = torch.empty((v, ds), dtype=torch.bfloat16, device=dev)
    wsp = torch.empty(max(fwd_bytes, bwd_bytes), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream

    def step(mid=None):
        if fused:
            B.lce_kd_forward_backward(p, hs.data_ptr(), ws.data_ptr(), ht.data_ptr(), wt.data_ptr(), t.data_ptr(),
                                      grad.data_ptr(), loss.data_ptr(), lse_s.data_ptr(), lse_t.data_ptr(),
                                      nv.data_ptr(), status.data_ptr(), dh.data_ptr(), dw.data_ptr(), wsp.data_ptr(),
                                      fwd_bytes, stream)
            return
        B.lce_kd_forward(p, hs.data_ptr(), ws.data_ptr(), ht.data_ptr(), wt.data_ptr(), t.data_ptr(),
                         loss.data_ptr(), lse_s.data_ptr(), lse_t.data_ptr(), nv.data_ptr(), status.data_ptr(),
                         wsp.data_ptr(), fwd_bytes, stream)
        if mid is not None:
            mid.record()
        B.lce_kd_backward(p, hs.data_ptr(), ws.data_ptr(), ht.data_ptr(), wt.data_ptr(), t.data_ptr(),
                          lse_s.data_ptr(), lse_t.data_ptr(), nv.data_ptr(), grad.data_ptr(), dh.data_ptr(),
                          dw.data_ptr(), wsp.data_ptr(), bwd_bytes, stream)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        print(f"[bench] kd warmup {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)
    peak = torch.cuda.max_memory_allocated()
    events = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1, e2 in events:
        e0.record()
        step(e1)
        if fused:           # one call: no forward / backward boundary to mark
            e1.record()
        e2.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    kernels, kpass = _kernel_breakdown(B, step, args.steps)
    nvalid = int(nv.item())
    # MFMA work per step and kernel (see the module docstring)
    work = {"fwd_stats": 2.0 * nvalid * v * (ds + dt), "kd_teacher_p": (2.0 if fused else 4.0) * nvalid * v * dt,
            "bwd_g": 2.0 * nvalid * v * ds, "bwd_dw": 2.0 * nvalid * v * ds, "bwd_dh": 2.0 * nvalid * v * ds}
    if not fused:
        work["kd_q"] = 2.0 * nvalid * v * ds
    flops_step = sum(work.values())
    ms_step = elapsed * 1e3 / args.steps
    for kname, r in sorted(kernels.items(), key=lambda kv: -kv[1]["total_ms"]):
        extra = ""
        if kname in work:
            tf = work[kname] / (r["total_ms"] / kpass * 1e-3) / 1e12
            extra = f" {tf:7.1f} TFLOP/s ({100 * tf / PEAK_BF16_TFLOPS:4.1f}% of peak)"
        print(f"[bench]   {kname:12s} {r['total_ms'] / kpass:8.3f} ms/step  {r['launches']:5d} launches"
              f"  avg {r['avg_ms']:.4f} ms{extra}", file=sys.stderr)
    dom = max((kk for kk in kernels if kk in work), key=lambda kk: kernels[kk]["total_ms"])
    per_launch = work[dom] / (kernels[dom]["launches"] / kpass)
    achieved = per_launch / (kernels[dom]["avg_ms"] * 1e-3) / 1e12
    out = {
        "metric": METRIC, "value": n * args.steps / elapsed, "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": name, "n_tokens": n, "student_hidden": ds, "teacher_hidden": dt, "vocab": v,
                   "n_valid": nvalid, "temperature": T, "parallelism": "none", "reduction": "mean",
                   "variant": "kd_fused" if fused else "kd"},
        "valid_tokens_per_s": nvalid * args.steps / elapsed,
        "mfma_frac_step": flops_step / (ms_step * 1e-3) / (PEAK_BF16_TFLOPS * 1e12),
        "step_ms": _event_summary(events),
        "peak_hbm_bytes": int(peak), "workspace_bytes": int(max(fwd_bytes, bwd_bytes)),
        "logits_bytes_avoided_fp32": 2 * int(n) * int(v) * 4,
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS, "traffic": None,
                     "flops_per_launch": per_launch, "avg_launch_ms": kernels[dom]["avg_ms"]},
        "kernels_ms_per_step": {kk: r["total_ms"] / kpass for kk, r in kernels.items()},
        "kernel_timing": f"second pass of {kpass} steps after the timed region, HIP events around each launch",
        "lce_hip_sha256": _source_hash(),
        "cpu_baseline": None if args.no_cpu_baseline else _kd_cpu_baseline(inp, T),
    }
    if not args.no_cpu_baseline:
        out["host"] = _host_info()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
