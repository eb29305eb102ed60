"""Helpers shared by the GPU parity tests: moving seeded inputs to the device,
running the library through its C ABI, and the error metric.

Error metric (per tensor): max |gpu - oracle| / RMS(oracle).  Bounds: 1e-4 for
fp32 inputs, 2e-2 for bf16 inputs with fp32 accumulation."""
import numpy as np

import oracle
import paper_2509_25223_amd as rla

TOL = {"f32": 1e-4, "bf16": 2e-2}

# library variant bits -> the oracle's own variant bits
LIB_TO_ORACLE = ((rla.RLA_FLAG_RESIDUAL_TANH, oracle.TANH), (rla.RLA_FLAG_UNGATED_OUTPUT, oracle.UNGATED),
                 (rla.RLA_FLAG_DECAYED_RESIDUAL, oracle.DECAYED))


def oracle_flags(variants):
    return sum(o for lib, o in LIB_TO_ORACLE if variants & lib)


def torch_dtype(dt):
    import torch
    return torch.float32 if dt == "f32" else torch.bfloat16


def dev(a, dtype, device):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.float32)))
    return t.to(device=device, dtype=dtype)


def host(t):
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def rel_err(x, ref):
    ref = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref)))
    if rms == 0.0:
        return float(np.max(np.abs(x))) if x.size else 0.0
    return float(np.max(np.abs(np.asarray(x, np.float64) - ref))) / rms


def gpu_forward(variant, inp, dtype, device, clip=1.0, S0=None, R0=None, dense_B=None, variants=0):
    """Runs rla_forward / rdn_forward on packed inputs [ntok, H, d].  With
    dense_B the tokens are viewed as [B, T, H, d] (equal lengths), else
    cu_seqlens from inp is used."""
    import torch
    td = torch_dtype(dtype)
    q, k, v = (dev(inp[n], td, device) for n in ("q", "k", "v"))
    gates = [dev(inp[n], torch.float32, device) for n in ("alpha_s", "beta", "alpha_r", "gamma")]
    S0d = None if S0 is None else dev(S0, torch.float32, device)
    R0d = None if R0 is None else dev(R0, torch.float32, device)
    cu = None
    if dense_B:
        B = dense_B
        T = q.shape[0] // B
        q, k, v = (x.view(B, T, *x.shape[1:]) for x in (q, k, v))
        gates = [g.view(B, T, -1) for g in gates]
    else:
        cu = torch.from_numpy(np.asarray(inp["cu_seqlens"], dtype=np.int32)).to(device)
    fn = rla.rdn_forward if variant == "rdn" else rla.rla_forward
    o, Sf, Rf = fn(q, k, v, *gates, clip=clip, S0=S0d, R0=R0d, cu_seqlens=cu, variants=variants)
    torch.cuda.synchronize()
    return host(o).reshape(-1, *o.shape[-2:]), host(Sf), host(Rf)


def oracle_forward(variant, inp, clip=1.0, S0=None, R0=None, variants=0):
    return oracle.forward(variant, inp["q"], inp["k"], inp["v"], inp["alpha_s"], inp["beta"],
                          inp["alpha_r"], inp["gamma"], clip=clip, S0=S0, R0=R0,
                          cu_seqlens=inp["cu_seqlens"], flags=oracle_flags(variants))


def select(inp, seqs, heads):
    """Sub-problem of the given sequences and heads (for sampled checks)."""
    cu = inp["cu_seqlens"]
    idx = np.concatenate([np.arange(cu[n], cu[n + 1]) for n in seqs]).astype(np.int64)
    out = {}
    for key, val in inp.items():
        if key == "cu_seqlens":
            continue
        out[key] = val[idx][:, heads]
    lens = [cu[n + 1] - cu[n] for n in seqs]
    out["cu_seqlens"] = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    return out


def gpu_backward(variant, inp, dtype, device, clip=1.0, S0=None, R0=None, dS_final=None,
                 dR_final=None, dense_B=None, out_dtype=None, variants=0):
    """Runs rla_backward / rdn_backward on packed inputs; returns numpy grads."""
    import torch
    td = torch_dtype(dtype)
    q, k, v, dO = (dev(inp[n], td, device) for n in ("q", "k", "v", "dO"))
    gates = [dev(inp[n], torch.float32, device) for n in ("alpha_s", "beta", "alpha_r", "gamma")]
    opt = lambda a: None if a is None else dev(a, torch.float32, device)
    cu = None
    if dense_B:
        B = dense_B
        T = q.shape[0] // B
        q, k, v, dO = (x.view(B, T, *x.shape[1:]) for x in (q, k, v, dO))
        gates = [g.view(B, T, -1) for g in gates]
    else:
        cu = torch.from_numpy(np.asarray(inp["cu_seqlens"], dtype=np.int32)).to(device)
    fn = rla.rdn_backward if variant == "rdn" else rla.rla_backward
    g = fn(q, k, v, *gates, dO, clip=clip, S0=opt(S0), R0=opt(R0), dS_final=opt(dS_final),
           dR_final=opt(dR_final), cu_seqlens=cu, out_dtype=out_dtype, variants=variants)
    torch.cuda.synchronize()
    out = {}
    for key, t in g.items():
        a = host(t)
        if key in ("dq", "dk", "dv"):
            a = a.reshape(-1, *a.shape[-2:])
        elif key not in ("dS0", "dR0"):
            a = a.reshape(-1, a.shape[-1])
        out[key] = a
    return out


def oracle_backward(variant, inp, clip=1.0, S0=None, R0=None, dS_final=None, dR_final=None,
                    variants=0):
    return oracle.backward(variant, inp["q"], inp["k"], inp["v"], inp["alpha_s"], inp["beta"],
                           inp["alpha_r"], inp["gamma"], inp["dO"], clip=clip, S0=S0, R0=R0,
                           dS_final=dS_final, dR_final=dR_final, cu_seqlens=inp["cu_seqlens"],
                           flags=oracle_flags(variants))


def nudge(variant, inp, dtype, clip=1.0, S0=None, R0=None, margin=None, variants=0):
    """Moves v (on its dtype's grid) so no pre-clip residual is within `margin`
    of the clip kink; masks taken in two precisions then agree."""
    if margin is None:
        margin = 1e-2 if dtype == "bf16" else 1e-4
    v, moved = oracle.nudge_margin(variant, inp["q"], inp["k"], inp["v"], inp["alpha_s"],
                                   inp["beta"], inp["alpha_r"], inp["gamma"], clip=clip, S0=S0,
                                   R0=R0, cu_seqlens=inp["cu_seqlens"], margin=margin,
                                   grid="bf16" if dtype == "bf16" else "f32",
                                   flags=oracle_flags(variants))
    out = dict(inp)
    out["v"] = v.astype(np.float32)
    return out, moved


GRAD_KEYS = ("dq", "dk", "dv", "dalpha_s", "dbeta", "dalpha_r", "dgamma", "dS0", "dR0")
