#!/usr/bin/env python3
"""Benchmark of the RDN training step of the sequence-mixing layer on one GPU.

One step = rdn_forward + rdn_backward (the whole hot path) on the workload
B=4, T=4096, H=16, d_k=d_v=128, bf16 inputs, fp32 accumulation and fp32
outputs (o, dq, dk, dv), gates fp32, clip 1, zero initial states, dO ~ N(0,1).
Inputs are seeded synthetic data (datagen) resident in HBM before timing.
As in training, the forward saves what the backward needs (chunk states,
clip masks, the U, UR, r blocks) in the workspace and the backward reads it
instead of recomputing the forward.

Prints ONE JSON line with the throughput (tokens/s, whole job) and the
metric's second figure, the step's share of the dense bf16 MFMA peak (the
chunked method's count model, ~1.52 Mflop per token-head, over the step
time); per-stage launch times (HIP events recorded on the launch stream
around each kernel stage) with their algorithmic TFLOP/s and GB/s (bytes:
only the operator's own inputs and outputs each kernel touches); the roofline
of the dominant kernel (HBM or MFMA by its algorithmic intensity against the
ridge), with the design's bytes (intermediates included) and the counter
traffic beside the algorithmic bytes; and the fp64 CPU oracle timed on the
same workload on this host.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
                    [--copy-calibration-mib M] [--op fwdbwd|decode]

--op decode instead times the recurrent decoding step (one token for each of
256 sequences, H=16, d=128, states resident in HBM and updated in place),
an HBM-bound kernel reported against the 8 TB/s peak.
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


# HBM bytes per launch of each kernel on this workload, from rocprofv3
# FETCH_SIZE / WRITE_SIZE runs scaled by a 1 GiB device copy's counts (the
# numbers and commands are in profiles/), keyed by a hash of the kernel's
# sources: a kernel changed since its counters were taken reports null.
MEASURED_TRAFFIC = {
    "prep": ("6d1faa0c02a5a94f", ('prep.hip', 'common.hpp', 'kernels.hpp'), 168030112, 109707264),
    "grad_absmax": ("4b44d1d3f6c4cf05", ('grad_scale.hip', 'common.hpp', 'kernels.hpp'), 67196357, 131370),
    "bwd_scan": ("89cbf6b2fe761bee", ('bwd_scan.hip', 'common.hpp', 'kernels.hpp'), 344435965, 613594794),
    "bwd_grad": ("08848c41c5e9ad23", ('bwd_grad.hip', 'common.hpp', 'kernels.hpp'), 1232656230, 302521893),
    "fwd_scan": ("017ad91aed089cd7", ('fwd_scan.hip', 'common.hpp', 'kernels.hpp'), 310649896, 638591833),
    "decode": ("a6d19635132fd623", ('decode.hip', 'common.hpp', 'kernels.hpp'), 542746720, 539558630),
}


def measured_traffic(stage: str):
    """Counter-derived HBM bytes per launch, or None if the kernel changed."""
    import hashlib
    if stage not in MEASURED_TRAFFIC:
        return None
    digest, files, read, written = MEASURED_TRAFFIC[stage]
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2509_25223_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return read + written if h.hexdigest()[:16] == digest else None


def kernel_flops(stage: str, d: int, C: int = CHUNK) -> float:
    """Algorithmic flops of one (chunk, head) for each kernel of the RDN
    fwd+bwd path, d_k = d_v = d: every matrix product the kernel's chunk
    algebra needs, counted once as 2*m*n*k (split-precision repeats are not
    counted), products restricted to a triangle over its C(C+1)/2 entries."""
    cd2, c2d, tri = 2.0 * C * d * d, 2.0 * C * C * d, float(C * (C + 1)) * d
    if stage == "prep":           # G = K K^T, P = Q K^T, two triangular inverses
        return 2 * c2d + 2 * (C ** 3) / 3.0
    if stage == "fwd_scan":       # KS QS KR QR, S/R updates; T^S Y, MG U, MP U, T^R YR, MR UR
        return 6 * cd2 + 5 * c2d
    if stage == "bwd_scan":       # K dS, K dR, dS/dR updates (4); 5 transposed C x C products
        return 6 * cd2 + 5 * c2d
    if stage == "bwd_grad":       # 7 state products, W1..W5 G P (lower), dP K, dP^T Q, (dG+dG^T) K
        return 7 * cd2 + 7 * tri + 3 * c2d
    if stage == "grad_absmax":    # a maximum over dO: no products
        return 0.0
    raise KeyError(stage)


def kernel_io_bytes(stage: str, d: int, C: int = CHUNK) -> int:
    """Algorithmic HBM bytes of one (chunk, head): only the operator's own
    inputs and outputs that the kernel must read or write (bf16 q, k, v, dO;
    fp32 gates; fp32 o, dq, dk, dv and gate gradients as this benchmark
    writes them).  Intermediates of the design (matrices, checkpoints, saved
    blocks, masks) are not algorithmic and are not counted here."""
    row_in, row_out, gate = d * 2, d * 4, 4
    if stage == "prep":           # q, k, four gates
        return C * (2 * row_in + 4 * gate)
    if stage == "fwd_scan":       # q, k, v, four gates in; o out
        return C * (3 * row_in + 4 * gate + row_out)
    if stage == "bwd_scan":       # q, k, dO, four gates in; dv out
        return C * (3 * row_in + 4 * gate + row_out)
    if stage == "bwd_grad":       # q, k, v, dO, four gates in; dq, dk, four gate gradients out
        return C * (4 * row_in + 4 * gate + 2 * row_out + 4 * gate)
    if stage == "grad_absmax":    # dO in
        return C * row_in
    raise KeyError(stage)


def design_bytes(stage: str, d: int, C: int = CHUNK) -> int:
    """HBM bytes of one (chunk, head) that the kernel moves by design,
    intermediates included: the algorithmic bytes plus prep's five fp16 64x64
    matrices and gate block, the fp16 chunk-start states S, R and chunk-end
    gradient states dS, dR with their tile scales, the clip mask (one byte per
    element) and the fp16 token blocks U, UR, r, dX, dY, dYR.  This is the
    traffic the counters should read; the excess over kernel_io_bytes is the
    price of the split into four kernels."""
    tok_h = C * d * 2
    mats, gate_blk = 5 * C * C * 2, 256 * 4
    state = d * d * 2 + (d // 16) * (d // 32) * 4
    if stage == "prep":
        return kernel_io_bytes(stage, d, C) + mats + gate_blk
    if stage == "fwd_scan":       # + matrices, gate block in; S R, mask, U UR r out
        return kernel_io_bytes(stage, d, C) + mats + gate_blk + 2 * state + C * d + 3 * tok_h
    if stage == "bwd_scan":       # + matrices, gate block, mask in; dS dR, dX dY dYR out
        return kernel_io_bytes(stage, d, C) + mats + gate_blk + C * d + 2 * state + 3 * tok_h
    if stage == "bwd_grad":       # + S0 R0 dS1 dR1, U UR r dX dY dYR, gate block in
        return kernel_io_bytes(stage, d, C) + 4 * state + 6 * tok_h + gate_blk
    if stage == "grad_absmax":    # + one maximum out
        return kernel_io_bytes(stage, d, C) + 4
    raise KeyError(stage)


def step_flops_per_token_head(d: int, C: int = CHUNK) -> float:
    """The count model of the RDN chunked method per token-head: forward =
    state-independent intra-chunk work 10Cd + 2C^2/3 (Gram, scores, UT
    transform, W and U0 formation) + state-dependent intra-chunk work 8Cd +
    state products 14d^2; forward + backward = 4x the forward (the backward
    recomputes the forward and takes two gradient products per forward
    product).  ~1.52 Mflop at C = 64, d = 128."""
    fwd = 10.0 * C * d + 2.0 * C * C / 3.0 + 8.0 * C * d + 14.0 * d * d
    return 4.0 * fwd


RIDGE = PEAK_MFMA_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)   # flop per byte


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--op", choices=("fwdbwd", "decode"), default="fwdbwd",
                    help="fwdbwd: the RDN training step (default); decode: the RDN recurrent "
                         "step, one token for each of 256 sequences from resident states")
    ap.add_argument("--variants", default="",
                    help="comma list of operator variants to switch on: tanh (log-cosh "
                         "residual), ungated (output), decayed (residual), or all")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="first run one device-to-device copy of this many MiB (a kernel of "
                         "known traffic, for scaling hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the operator shards by (sequence, head) with no "
              "exchange, and multi-GPU runs are not part of this build; use --gpus 1.",
              file=sys.stderr)
        return 2

    if args.op == "decode":
        return run_decode(args)
    return run_fwdbwd(args)


def variant_bits(spec: str) -> tuple:
    """(flag bits, names) for --variants."""
    import paper_2509_25223_amd as rla
    table = {"tanh": rla.RLA_FLAG_RESIDUAL_TANH, "ungated": rla.RLA_FLAG_UNGATED_OUTPUT,
             "decayed": rla.RLA_FLAG_DECAYED_RESIDUAL}
    names = sorted(table) if spec == "all" else [x for x in spec.split(",") if x]
    for n in names:
        if n not in table:
            raise SystemExit("unknown variant %r (choose from %s or all)" % (n, ", ".join(table)))
    return sum(table[n] for n in names), names


def copy_calibration(mib: int, dev) -> None:
    """One device-to-device copy of known size, for scaling byte counters."""
    import torch
    if mib <= 0:
        return
    n = mib * (1 << 20) // 4
    src_ = torch.ones(n, dtype=torch.float32, device=dev)
    dst_ = torch.empty_like(src_)
    dst_.copy_(src_)
    torch.cuda.synchronize()


def run_fwdbwd(args) -> int:
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
    vbits, vnames = variant_bits(args.variants)
    prob = rla.make_problem(q, v, clip=wl.clip)
    ws_b = torch.empty(rla.rla_workspace_size(prob, rla.RLA_OP_RDN_BACKWARD), dtype=torch.uint8, device=dev)
    o = torch.empty(v.shape, dtype=torch.float32, device=dev)
    grads = rla.rdn_backward(q, k, v, *gates, dO, clip=wl.clip, workspace=ws_b, variants=vbits)

    def fwd():
        rla.rdn_forward(q, k, v, *gates, clip=wl.clip, out=o, workspace=ws_b, return_states=False,
                        save_for_backward=True, variants=vbits)

    def bwd():
        rla.rdn_backward(q, k, v, *gates, dO, clip=wl.clip, workspace=ws_b, grads=grads,
                         use_saved=True, variants=vbits)

    def step():
        fwd()
        bwd()

    copy_calibration(args.copy_calibration_mib, dev)

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
    bwd_stages = ["grad_absmax", "bwd_scan", "bwd_grad"]
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
    stages = {}
    for key, ms in stage_ms.items():
        name = key.split(".", 1)[1]
        fl, by, dby = kernel_flops(name, d), kernel_io_bytes(name, d), design_bytes(name, d)
        tf = fl * units / (ms * 1e-3) / 1e12
        gb = by * units / (ms * 1e-3) / 1e9
        traffic = None if vnames else measured_traffic(name)
        stages[key] = {"ms": round(ms, 4), "tflops": round(tf, 2), "gbs": round(gb, 1),
                       "mfma_frac": round(tf / PEAK_MFMA_TFLOPS, 4),
                       "hbm_frac": round(gb / PEAK_HBM_GBS, 4),
                       "intensity": round(fl / by, 1),
                       "design_bytes": dby * units,
                       "traffic": traffic,
                       "traffic_over_algorithmic": None if traffic is None else round(traffic / (by * units), 2)}
    dom = max(stage_ms, key=stage_ms.get)
    ds = stages[dom]
    dname = dom.split(".", 1)[1]
    kernel_names = {"prep": "prep_kernel", "fwd_scan": "fwd_scan_kernel (saving)",
                    "grad_absmax": "grad_absmax_kernel", "bwd_scan": "bwd_scan_kernel",
                    "bwd_grad": "bwd_grad_kernel"}
    fl, by = kernel_flops(dname, d), kernel_io_bytes(dname, d)
    # the binding roof of the dominant kernel: HBM below the ridge intensity, MFMA above it
    if fl / by < RIDGE:
        roofline = {"bound": "hbm", "achieved": ds["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": ds["hbm_frac"], "traffic": ds["traffic"],
                    "bytes_per_launch": by * units, "flops_per_launch": fl * units,
                    "mfma_frac": ds["mfma_frac"]}
    else:
        roofline = {"bound": "mfma", "achieved": ds["tflops"], "peak": PEAK_MFMA_TFLOPS,
                    "unit": "TFLOP/s", "frac": ds["mfma_frac"], "traffic": ds["traffic"],
                    "flops_per_launch": fl * units, "bytes_per_launch": by * units,
                    "hbm_frac": ds["hbm_frac"]}
    roofline.update({"kernel": kernel_names[dname], "stage": dom, "launch_ms": ds["ms"],
                     "units_per_launch": units, "design_bytes_per_launch": ds["design_bytes"],
                     "traffic_over_algorithmic": ds["traffic_over_algorithmic"]})
    # the metric's own fraction: the count model's flops of the whole step over
    # the step time, against the dense bf16 MFMA peak
    step_flops = step_flops_per_token_head(d) * B * T * H
    step_tflops = step_flops / (ms_per_step * 1e-3) / 1e12
    step_roofline = {"bound": "mfma", "achieved": round(step_tflops, 2), "peak": PEAK_MFMA_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(step_tflops / PEAK_MFMA_TFLOPS, 4),
                     "flops_per_step": step_flops,
                     "flops_per_token_head": step_flops_per_token_head(d)}

    # ---- CPU baseline: the fp64 oracle on the same workload ----
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        names = ("q", "k", "v", "alpha_s", "beta", "alpha_r", "gamma", "dO")
        cu = wl.cu_seqlens()
        oflags = sum(f for n, f in (("tanh", oracle.TANH), ("ungated", oracle.UNGATED),
                                    ("decayed", oracle.DECAYED)) if n in vnames)
        c0 = time.perf_counter()
        oracle.forward("rdn", *[inp[n] for n in names[:7]], clip=wl.clip, cu_seqlens=cu, flags=oflags)
        oracle.backward("rdn", *[inp[n] for n in names], clip=wl.clip, cu_seqlens=cu, flags=oflags)
        c1 = time.perf_counter()
        cpu = {"value": round(B * T / (c1 - c0), 2), "unit": "tokens/s",
               "cores": oracle.threads(), "kind": "oracle",
               "sample": "the whole workload (%d sequences x %d tokens, %d heads), forward then "
                         "backward, fp64 token recurrence (%.1f s wall)" % (B, T, H, c1 - c0)}

    line = {
        "metric": "RDN fwd+bwd tokens/sec on 1 MI355X (H=16,d=128,T=4096); % bf16 MFMA peak",
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
        "config": dict({"workload": wl.name, "B": B, "T": T, "H": H, "d_k": d, "d_v": d,
                        "chunk": CHUNK, "clip": wl.clip, "outputs": "fp32",
                        "parallelism": "single GPU"}, **({"variants": vnames} if vnames else {})),
        # the metric's second figure: % of the dense bf16 MFMA peak of the whole step
        "pct_bf16_mfma_peak": round(100.0 * step_roofline["frac"], 2),
        "step_roofline": step_roofline,
        "stages": stages,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    return 0


DECODE_B = 256   # sequences decoded together (one token each per step)


def decode_bytes(dk: int, dv: int) -> int:
    """Algorithmic HBM bytes of one (sequence, head) of a one-token decode
    step: S and R read and written (fp32), q k v in (bf16), o out (fp32), four
    fp32 gates."""
    return 4 * dk * dv * 4 + (2 * dk + dv) * 2 + dv * 4 + 4 * 4


def run_decode(args) -> int:
    import numpy as np
    import torch
    import datagen
    import paper_2509_25223_amd as rla

    dev = torch.device("cuda:0")
    B, H, d = DECODE_B, 16, 128
    wl = datagen.small("rdn_fwd", "bf16", [1] * B, H=H, d=d, varlen=False)
    seed = 6 if args.seed is None else args.seed
    inp = datagen.make_inputs(wl, seed=seed)
    S0, R0 = datagen.random_states(seed, B, H, d, d)

    def to_dev(a, dtype, shape):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev, dtype).view(*shape)

    q, k, v = (to_dev(inp[n], torch.bfloat16, (B, 1, H, d)) for n in ("q", "k", "v"))
    gates = [to_dev(inp[n], torch.float32, (B, 1, H)) for n in ("alpha_s", "beta", "alpha_r", "gamma")]
    S, R = to_dev(S0, torch.float32, S0.shape), to_dev(R0, torch.float32, R0.shape)
    o = torch.empty(v.shape, dtype=torch.float32, device=dev)
    copy_calibration(args.copy_calibration_mib, dev)

    def step():   # in place: the states advance by one token per step
        rla.rdn_decode(q, k, v, *gates, clip=wl.clip, S_in=S, R_in=R, S_out=S, R_out=R, out=o)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed * 1e3 / args.steps

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    for s_ in range(args.steps):
        rla.rla_set_stage_events(ev[s_])
        step()
    rla.rla_set_stage_events(None)
    torch.cuda.synchronize()
    kms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    units = B * H
    by = decode_bytes(d, d) * units
    gbs = by / (kms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": measured_traffic("decode"),
                "bytes_per_launch": by,
                "kernel": "decode_kernel", "launch_ms": round(kms, 4), "units_per_launch": units}

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        names = ("q", "k", "v", "alpha_s", "beta", "alpha_r", "gamma")
        reps = 0
        c0 = time.perf_counter()
        while True:   # repeat the same step for about 10 s of oracle time
            oracle.forward("rdn", *[inp[n] for n in names], clip=wl.clip, S0=S0, R0=R0,
                           cu_seqlens=wl.cu_seqlens())
            reps += 1
            if time.perf_counter() - c0 > 10.0:
                break
        c1 = time.perf_counter()
        cpu = {"value": round(B * reps / (c1 - c0), 2), "unit": "tokens/s",
               "cores": oracle.threads(), "kind": "oracle",
               "sample": "%d repetitions of the whole decode step (%d sequences x 1 token, %d "
                         "heads, states in and out), fp64 token recurrence (%.1f s wall)"
                         % (reps, B, H, c1 - c0)}

    line = {
        "metric": "RDN decode-step tokens/sec on 1 MI355X (B=256 sequences, H=16, d=128)",
        "value": round(B / (ms_per_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 in, fp32 states and arithmetic, fp32 out",
        "data": "synthetic",
        "config": {"workload": "rdn_decode_bf16_B256_H16_d128", "B": B, "T": 1, "H": H,
                   "d_k": d, "d_v": d, "clip": wl.clip, "states": "fp32, updated in place",
                   "parallelism": "single GPU"},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
