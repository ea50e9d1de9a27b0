#!/usr/bin/env python3
"""Causal attention forward+backward throughput on one MI355X.

One step = attn_fwd + attn_bwd (every kernel of the hot path) over one packed
batch whose inputs are already resident in HBM.  Prints ONE JSON line with
the counted-FLOP throughput (TFLOP/s), the roofline of the dominant kernel
(timed with HIP events on its own stream inside the library) and the fp64 CPU
oracle timed on a bounded sample of the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

WORKLOADS = {
    "single131072": 3,   # one 131,072-token sequence, 4 heads (one GPU's head share), d=128
    "packed65536": 2,    # 65,536 tokens, log-uniform lengths in [128, 8192], 32 heads
    "single638976": 4,   # one 638,976-token ("624K") sequence, 4 heads
    "single512": 1,      # 512 tokens, 8 heads, d=64
}

METRIC = "causal attn fwd+bwd TFLOP/s and % bf16 MFMA peak vs seq length (1 GPU)"

# the sequence-length sweep timed in the same run as the main line: single
# sequences over 4 heads (one GPU's share of a 32-head layer over 8 GPUs)
# from 4K to the 638,976-token ("624K") length, and the packed 65,536-token
# batch over 32 heads; (label, lengths, heads, steps, warmup, events in the
# timed steps: off for sub-millisecond steps, where recording them would be
# part of what is timed)
SWEEP = [
    ("single4096_h4_d128", [4096], 4, 50, 5, False),
    ("single16384_h4_d128", [16384], 4, 20, 3, False),
    ("single131072_h4_d128", [131072], 4, 5, 2, True),
    ("single638976_h4_d128", [638976], 4, 3, 1, True),
    ("packed65536_loguniform128-8192_h32_d128", None, 32, 10, 3, True),
]


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="single131072")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the sequence-length sweep timed after the main line")
    ap.add_argument("--cpu-sample-tokens", type=int, default=40960,
                    help="causal prefix length the CPU oracle is timed on")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (3 times), for "
                         "calibrating HBM byte counters, and exit")
    return ap.parse_args()


def copy_calibration(mib: int):
    """A plain device-to-device copy of known size: its FETCH_SIZE / WRITE_SIZE
    counters give the scale between counter kilobytes and real bytes."""
    import torch
    n = mib << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(7)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n, "launches": 3}), flush=True)


def cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo), or the machine type."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def cpu_baseline(w, inputs, sample_tokens: int):
    """Time the fp64 oracle (as it stands) on the causal prefix of head 0:
    its full forward + backward over the first `sample_tokens` tokens.  The
    full workload's oracle time is extrapolated from the measured rate."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import attention as ora
    from paper_2511_13198_amd import accounting as acc
    S = min(sample_tokens, w.total_tokens)
    hk = 0
    q = inputs["q"][:S, 0:1].cpu().double().numpy()
    k = inputs["k"][:S, hk:hk + 1].cpu().double().numpy()
    v = inputs["v"][:S, hk:hk + 1].cpu().double().numpy()
    do = inputs["do"][:S, 0:1].cpu().double().numpy()
    cu = np.array([0, S], dtype=np.int64)
    t0 = time.perf_counter()
    ora.backward(q, k, v, do, cu, w.causal, w.softmax_scale)
    dt = time.perf_counter() - t0
    flops = acc.fwd_bwd_flops([S], 1, w.head_dim, w.causal)
    full = acc.fwd_bwd_flops(w.lengths, w.heads_q, w.head_dim, w.causal)
    rate = flops / dt
    threads = max([p.get("num_threads", 1) for p in threadpool_info()
                   if p.get("user_api") == "blas"] or [1])
    return {
        "value": rate / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "cpu_model": cpu_model(),
        "sample": (f"fp64 forward+backward of the causal prefix of the first {S} tokens of "
                   f"query head 0 of the {w.name} workload ({flops:.3e} counted FLOPs in "
                   f"{dt:.2f} s)"),
        "full_workload_s_extrapolated": round(full / rate, 1),
        "extrapolation": (f"{full:.3e} counted FLOPs of one full step at the sample's "
                          f"measured rate (extrapolated, not run)"),
    }


def recorded_traffic(workload_name: str, kernel: str):
    """HBM bytes per launch of `kernel` (FETCH_SIZE + WRITE_SIZE, each scaled
    by a plain-copy calibration) from the committed rocprofv3 summary of this
    workload, or None when there is none or the kernel sources changed since
    the counters were taken."""
    from paper_2511_13198_amd import profiling
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles",
                        f"{workload_name}_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("source_sha256") != profiling.source_hash():
        return None
    k = rec.get("kernels", {}).get(kernel, {})
    if "fetch_bytes" not in k or "write_bytes" not in k:
        return None
    return k["fetch_bytes"] + k["write_bytes"]


def time_steps(w, steps: int, warmup: int, events_in_timed: bool = True):
    """Mean wall time (ms) of `steps` fwd+bwd steps of workload w with inputs
    resident in HBM, after `warmup` untimed steps, and the library's
    per-kernel times (HIP events recorded on each launch's stream): over the
    timed steps themselves, or (events_in_timed=False, for sub-millisecond
    steps where recording two events per launch would be part of what is
    timed) over as many further steps after the timed ones."""
    import torch

    from paper_2511_13198_amd import pdyattn
    from paper_2511_13198_amd import workloads as wl
    T, hq, hkv, d = w.total_tokens, w.heads_q, w.heads_kv, w.head_dim
    dev = torch.device("cuda:0")
    inputs = wl.device_inputs(T, hq, hkv, d, device="cuda")
    q, k, v, do = inputs["q"], inputs["k"], inputs["v"], inputs["do"]
    cu = torch.from_numpy(w.cu_seqlens()).to(dev)
    maxlen, scale, causal = w.max_seqlen, w.softmax_scale, w.causal
    o = torch.empty_like(q)
    lse = torch.empty((hq, T), dtype=torch.float32, device=dev)
    dq = torch.empty((T, hq, d), dtype=torch.float32, device=dev)
    dk = torch.empty((T, hkv, d), dtype=torch.float32, device=dev)
    dv = torch.empty((T, hkv, d), dtype=torch.float32, device=dev)
    n = w.num_seqs
    wsf = torch.empty(max(256, pdyattn.fwd_workspace_size(T, n, maxlen, hq, hkv, d)),
                      dtype=torch.uint8, device=dev)
    wsb = torch.empty(max(256, pdyattn.bwd_workspace_size(T, n, maxlen, hq, hkv, d)),
                      dtype=torch.uint8, device=dev)

    def step():
        pdyattn.attn_fwd(q, k, v, cu, maxlen, causal, scale, out=o, lse=lse, workspace=wsf)
        pdyattn.attn_bwd(q, k, v, o, lse, do, cu, maxlen, causal, scale, dq=dq, dk=dk, dv=dv,
                         workspace=wsb)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    if events_in_timed:
        pdyattn.profile_start()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if not events_in_timed:
        pdyattn.profile_start()
        for _ in range(steps):
            step()
    prof = pdyattn.profile_stop()
    kernels_ms = {name: tot / cnt for name, (cnt, tot) in prof.items()}
    return (t1 - t0) / steps * 1e3, kernels_ms, inputs


def sweep(main_name: str, main_ms: float, main_kms: dict, main_steps: int, main_warmup: int):
    """The sweep lines: fwd+bwd TFLOP/s and % of peak per length (the main
    workload's line is the main measurement itself)."""
    import torch

    from paper_2511_13198_amd import accounting as acc
    from paper_2511_13198_amd import workloads as wl
    out = []
    for label, lengths, heads, steps, warmup, events in SWEEP:
        w = wl.config(2) if lengths is None else wl.Workload(label, lengths, heads, heads, 128)
        if w.name == main_name:
            ms, kms, steps, warmup = main_ms, main_kms, main_steps, main_warmup
        else:
            ms, kms, inputs = time_steps(w, steps, warmup, events_in_timed=events)
            del inputs
            torch.cuda.empty_cache()
        flops = acc.fwd_bwd_flops(w.lengths, w.heads_q, w.head_dim, w.causal)
        tf = flops / (ms / 1e3) / 1e12
        out.append({"workload": w.name, "tokens": w.total_tokens, "segments": w.num_seqs,
                    "max_seqlen": w.max_seqlen, "heads_q": w.heads_q, "heads_kv": w.heads_kv,
                    "steps": steps, "warmup": warmup, "ms_per_step": round(ms, 4),
                    "tflops": round(tf, 2),
                    "pct_of_peak": round(100.0 * tf / acc.PEAK_BF16_TFLOPS, 2),
                    "kernels_ms": {kk: round(vv, 4) for kk, vv in kms.items()}})
        print(f"[bench] sweep {w.name}: {ms:.3f} ms/step, {tf:.1f} TFLOP/s", file=sys.stderr,
              flush=True)
    return out


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, "
              f"WORLD_SIZE={world}): the library computes one GPU's share of the "
              f"attention, and sharding it over several GPUs is not implemented",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2511_13198_amd import accounting as acc
    from paper_2511_13198_amd import pdyattn
    from paper_2511_13198_amd import workloads as wl

    if args.copy_calibration_mib > 0:
        copy_calibration(args.copy_calibration_mib)
        return
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    pdyattn.lib()  # fail loudly if the HIP library is missing

    w = wl.config(WORKLOADS[args.workload])
    T, hq, hkv, d = w.total_tokens, w.heads_q, w.heads_kv, w.head_dim
    n, maxlen, causal = w.num_seqs, w.max_seqlen, w.causal
    print(f"[bench] {w.name}: {args.warmup} warmup + {args.steps} timed steps", file=sys.stderr,
          flush=True)
    ms, kernels_ms, inputs = time_steps(w, args.steps, args.warmup)
    flops = acc.fwd_bwd_flops(w.lengths, hq, d, causal)
    value = flops / (ms / 1e3) / 1e12

    dom = max((kname for kname in kernels_ms if kname in acc.KERNEL_PRODUCTS),
              key=lambda kname: kernels_ms[kname])
    dom_flops = acc.kernel_flops(dom, w.lengths, hq, d, causal)
    achieved = dom_flops / (kernels_ms[dom] / 1e3) / 1e12
    roofline = {
        "kernel": dom,
        "bound": "mfma",
        "achieved": round(achieved, 2),
        "peak": acc.PEAK_BF16_TFLOPS,
        "unit": "TFLOP/s",
        "frac": round(achieved / acc.PEAK_BF16_TFLOPS, 4),
        "traffic": recorded_traffic(w.name, dom),
    }
    print(f"[bench] {ms:.3f} ms/step, {value:.1f} TFLOP/s; kernels (avg ms): "
          + ", ".join(f"{kk}={vv:.3f}" for kk, vv in kernels_ms.items()),
          file=sys.stderr, flush=True)

    per_kernel = {kname: {"algorithmic_tflops": round(acc.kernel_flops(kname, w.lengths, hq, d, causal)
                                                      / (kms / 1e3) / 1e12, 2),
                          "issued_tflops": round(acc.kernel_issued_flops(kname, w.lengths, hq, d,
                                                                         causal)
                                                 / (kms / 1e3) / 1e12, 2)}
                  for kname, kms in kernels_ms.items() if kname in acc.KERNEL_PRODUCTS}
    lengths = None
    if not args.no_sweep:
        lengths = sweep(w.name, ms, kernels_ms, args.steps, args.warmup)

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, inputs, args.cpu_sample_tokens)

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 q/k/v/dO)",
        "config": {
            "workload": w.name,
            "tokens": T,
            "segments": n,
            "max_seqlen": maxlen,
            "heads_q": hq,
            "heads_kv": hkv,
            "head_dim": d,
            "causal": causal,
            "counted_flops_per_step": flops,
        },
        "pct_of_peak": round(100.0 * value / acc.PEAK_BF16_TFLOPS, 2),
        "kernels_ms": {kk: round(vv, 4) for kk, vv in kernels_ms.items()},
        "kernels_tflops": per_kernel,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "vs_seq_length": lengths,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
