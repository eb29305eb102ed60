"""Helpers shared by the GPU parity tests: moving seeded inputs to the device,
running the library through its C ABI, and the error metric.

Error metric (per tensor): max |gpu - oracle| / RMS(oracle).  Bounds: 1e-4 for
fp32 inputs, 2e-2 for bf16 inputs with fp32 accumulation."""
import numpy as np

import oracle
import paper_2509_25223_amd as rla

TOL = {"f32": 1e-4, "bf16": 2e-2}


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


def gpu_forward(variant, inp, dtype, device, clip=1.0, S0=None, R0=None, dense_B=None):
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
    o, Sf, Rf = fn(q, k, v, *gates, clip=clip, S0=S0d, R0=R0d, cu_seqlens=cu)
    torch.cuda.synchronize()
    return host(o).reshape(-1, *o.shape[-2:]), host(Sf), host(Rf)


def oracle_forward(variant, inp, clip=1.0, S0=None, R0=None):
    return oracle.forward(variant, inp["q"], inp["k"], inp["v"], inp["alpha_s"], inp["beta"],
                          inp["alpha_r"], inp["gamma"], clip=clip, S0=S0, R0=R0,
                          cu_seqlens=inp["cu_seqlens"])


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
