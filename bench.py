#!/usr/bin/env python3
"""Benchmark of the RDN training step of the sequence-mixing layer on one GPU.

One step = rdn_forward + rdn_backward (the whole hot path) on the workload
B=4, T=4096, H=16, d_k=d_v=128, bf16 inputs, fp32 accumulation and fp32
outputs (o, dq, dk, dv), gates fp32, clip 1, zero initial states, dO ~ N(0,1).
Inputs are seeded synthetic data (datagen) resident in HBM before timing.
As in training, the forward saves its chunk states and clip masks in the
workspace and the backward reads them instead of recomputing the forward.

Prints ONE JSON line with the throughput (tokens/s, whole job), the roofline
of the dominant kernel (algorithmic MFMA flops per launch / its launch time,
measured with HIP events recorded on the launch stream around each kernel
stage), and the fp64 CPU oracle timed on a bounded sample of the same
workload on this host.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

CHUNK = 64
PEAK_MFMA_TFLOPS = 2500.0   # MI355X dense fp16/bf16 MFMA
PEAK_HBM_GBS = 8000.0


def stage_flops_per_chunk_head(stage: str, d: int, C: int = CHUNK, rdn: bool = True) -> float:
    """Algorithmic matrix-product flops of one (chunk, head) for each kernel
    stage of the RDN fwd+bwd path (d = d_k = d_v).  Each product is counted
    once as 2*m*n*k, whatever precision splitting the kernel uses."""
    cd2, c2d = 2.0 * C * d * d, 2.0 * C * C * d
    if stage == "prep":           # G = K K^T, P = Q K^T
        return 2 * c2d
    if stage == "fwd_scan":       # KS QS KR QR, T^S Y MG U MP U T^R YR MR UR, S/R updates
        return 6 * cd2 + 5 * c2d
    if stage == "fwd_scan_ckpt":  # KS KR, T^S Y MG U T^R YR, S/R updates
        return 4 * cd2 + 3 * c2d
    if stage == "bwd_scan":       # K dS K dR, 5 transposed C x C products, dS/dR updates (4)
        return 6 * cd2 + 5 * c2d
    if stage == "bwd_grad":       # recompute 4+4, bwd 2+5, dQ/dK 6, W1..W5, G P, 4 final
        return 12 * cd2 + 14 * c2d + 6 * c2d
    raise KeyError(stage)


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seed", type=int, default=None)
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the operator shards by (sequence, head) with no "
              "exchange, and multi-GPU runs are not part of this build; use --gpus 1.",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch
    import datagen
    import paper_2509_25223_amd as rla

    dev = torch.device("cuda:0")
    wl = datagen.WORKLOADS[datagen.TRAINING]
    B, T, H, d = wl.B, wl.T, wl.H, wl.dk
    seed = datagen.SEEDS[wl.name] if args.seed is None else args.seed
    inp = datagen.make_inputs(wl, seed=seed, grads=True)

    def to_dev(name, dtype):
        a = np.ascontiguousarray(inp[name], dtype=np.float32)
        t = torch.from_numpy(a).to(device=dev, dtype=dtype)
        return t.view(B, T, *a.shape[1:])

    q, k, v, dO = (to_dev(n, torch.bfloat16) for n in ("q", "k", "v", "dO"))
    gates = [to_dev(n, torch.float32) for n in ("alpha_s", "beta", "alpha_r", "gamma")]
    prob = rla.make_problem(q, v, clip=wl.clip)
    ws_b = torch.empty(rla.rla_workspace_size(prob, rla.RLA_OP_RDN_BACKWARD), dtype=torch.uint8, device=dev)
    o = torch.empty(v.shape, dtype=torch.float32, device=dev)
    grads = rla.rdn_backward(q, k, v, *gates, dO, clip=wl.clip, workspace=ws_b)

    def fwd():
        rla.rdn_forward(q, k, v, *gates, clip=wl.clip, out=o, workspace=ws_b, return_states=False,
                        save_for_backward=True)

    def bwd():
        rla.rdn_backward(q, k, v, *gates, dO, clip=wl.clip, workspace=ws_b, grads=grads,
                         use_saved=True)

    def step():
        fwd()
        bwd()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # ---- timed region: K steps, synchronized on both sides ----
    if torch.distributed.is_available() and torch.distributed.is_initialized():
        torch.distributed.barrier()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed = t1 - t0
    tokens = B * T * args.steps
    value = tokens / elapsed
    ms_per_step = elapsed * 1e3 / args.steps

    # ---- per-kernel launch times with HIP events on the launch stream ----
    fwd_stages = ["prep", "fwd_scan"]
    bwd_stages = ["bwd_scan", "bwd_grad"]
    ev_f = [[torch.cuda.Event(enable_timing=True) for _ in range(len(fwd_stages) + 1)]
            for _ in range(args.steps)]
    ev_b = [[torch.cuda.Event(enable_timing=True) for _ in range(len(bwd_stages) + 1)]
            for _ in range(args.steps)]
    torch.cuda.synchronize()
    for s in range(args.steps):
        rla.rla_set_stage_events(ev_f[s])
        fwd()
        rla.rla_set_stage_events(ev_b[s])
        bwd()
    rla.rla_set_stage_events(None)
    torch.cuda.synchronize()
    stage_ms = {}
    for names, evs, tag in ((fwd_stages, ev_f, "fwd."), (bwd_stages, ev_b, "bwd.")):
        for i, name in enumerate(names):
            stage_ms[tag + name] = float(np.mean([e[i].elapsed_time(e[i + 1]) for e in evs]))
    units = B * ((T + CHUNK - 1) // CHUNK) * H   # (chunk, head) pairs per launch
    dom = max(stage_ms, key=stage_ms.get)
    dom_flops = stage_flops_per_chunk_head(dom.split(".", 1)[1], d) * units
    achieved = dom_flops / (stage_ms[dom] * 1e-3) / 1e12
    kernel_names = {"prep": "prep_kernel", "fwd_scan": "fwd_scan_kernel (saving)",
                    "fwd_scan_ckpt": "fwd_scan_kernel (checkpointing)",
                    "bwd_scan": "bwd_scan_kernel", "bwd_grad": "bwd_grad_kernel"}
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_MFMA_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_MFMA_TFLOPS, 4), "traffic": None,
                "kernel": kernel_names[dom.split(".", 1)[1]], "stage": dom,
                "flops_per_launch": dom_flops, "launch_ms": round(stage_ms[dom], 4)}

    # ---- CPU baseline: the fp64 oracle on a bounded sample of the workload ----
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        sample_T = T
        sub = {n: inp[n][:sample_T] for n in ("q", "k", "v", "alpha_s", "beta", "alpha_r",
                                               "gamma", "dO")}
        c0 = time.perf_counter()
        oracle.forward("rdn", sub["q"], sub["k"], sub["v"], sub["alpha_s"], sub["beta"],
                       sub["alpha_r"], sub["gamma"], clip=wl.clip)
        oracle.backward("rdn", sub["q"], sub["k"], sub["v"], sub["alpha_s"], sub["beta"],
                        sub["alpha_r"], sub["gamma"], sub["dO"], clip=wl.clip)
        c1 = time.perf_counter()
        cpu = {"value": round(sample_T / (c1 - c0), 2), "unit": "tokens/s",
               "cores": oracle.threads(), "kind": "oracle",
               "sample": "sequence 0 (%d tokens, all %d heads), fwd+bwd, fp64 (%.1f s wall)"
                         % (sample_T, H, c1 - c0)}

    line = {
        "metric": "RDN fwd+bwd tokens/sec on 1 MI355X (H=16,d=128,T=4096)",
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 in, fp16/bf16 MFMA, fp32 acc+out",
        "data": "synthetic",
        "config": {"workload": wl.name, "B": B, "T": T, "H": H, "d_k": d, "d_v": d,
                   "chunk": CHUNK, "clip": wl.clip, "outputs": "fp32",
                   "parallelism": "single GPU"},
        "stage_ms": {k_: round(v_, 4) for k_, v_ in stage_ms.items()},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
