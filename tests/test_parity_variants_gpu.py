"""GPU parity of the operator's variants (log-cosh residual, ungated output,
decayed residual, and all three together) against the fp64 oracle with the
same variant flags: forward, backward (recomputing and saved paths) and the
decoding step, element by element on seeded inputs."""
import math

import numpy as np
import pytest

import datagen
import paper_2509_25223_amd as rla
from tests.gpu_util import (GRAD_KEYS, TOL, gpu_backward, gpu_forward, nudge, oracle_backward,
                            oracle_forward, rel_err)

pytestmark = pytest.mark.gpu

TANH, UNG, DEC = (rla.RLA_FLAG_RESIDUAL_TANH, rla.RLA_FLAG_UNGATED_OUTPUT,
                  rla.RLA_FLAG_DECAYED_RESIDUAL)
FLAGS = [TANH, UNG, DEC, TANH | UNG | DEC]
NAMES = {TANH: "tanh", UNG: "ungated", DEC: "decayed", TANH | UNG | DEC: "all"}


def report(tag, errs, tol):
    print("[%s] %s" % (tag, " ".join("%s=%.2e" % kv for kv in errs.items())), flush=True)
    for key, e in errs.items():
        assert e <= tol, (key, e)


@pytest.mark.parametrize("flags", FLAGS, ids=[NAMES[f] for f in FLAGS])
@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("dtype,d", [("f32", 64), ("bf16", 128)])
def test_forward(device, variant, dtype, d, flags):
    lens = [1, 63, 0, 64, 65, 200]
    wl = datagen.small(variant + "_fwd", dtype, lens, H=2, d=d)
    inp = datagen.make_inputs(wl, seed=301)
    S0, R0 = datagen.random_states(31, len(lens), 2, d, d)
    for clip in (1.0, math.inf, 0.0):
        o, Sf, Rf = gpu_forward(variant, inp, dtype, device, clip=clip, S0=S0, R0=R0, variants=flags)
        ro, rS, rR = oracle_forward(variant, inp, clip=clip, S0=S0, R0=R0, variants=flags)
        report("fwd %s %s %s c=%s" % (variant, dtype, NAMES[flags], clip),
               dict(o=rel_err(o, ro), S=rel_err(Sf, rS), R=rel_err(Rf, rR)), TOL[dtype])


@pytest.mark.parametrize("flags", FLAGS, ids=[NAMES[f] for f in FLAGS])
@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("dtype,d", [("f32", 64), ("bf16", 128)])
def test_backward(device, variant, dtype, d, flags):
    lens = [64, 130, 5]
    wl = datagen.small(variant + "_fwdbwd", dtype, lens, H=2, d=d)
    inp = datagen.make_inputs(wl, seed=302)
    S0, R0 = datagen.random_states(32, len(lens), 2, d, d)
    rng = np.random.default_rng(33)
    dSf = (rng.standard_normal(S0.shape) * 0.3).astype(np.float32)
    dRf = (rng.standard_normal(R0.shape) * 0.3).astype(np.float32)
    inp, _ = nudge(variant, inp, dtype, S0=S0, R0=R0, variants=flags)
    g = gpu_backward(variant, inp, dtype, device, S0=S0, R0=R0, dS_final=dSf, dR_final=dRf,
                     variants=flags)
    ref = oracle_backward(variant, inp, S0=S0, R0=R0, dS_final=dSf, dR_final=dRf, variants=flags)
    report("bwd %s %s %s" % (variant, dtype, NAMES[flags]),
           {key: rel_err(g[key], ref[key]) for key in GRAD_KEYS}, TOL[dtype])


@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_saved_forward_path_is_identical(device, variant):
    """A saving forward with the variant flags, then the backward reading the
    workspace, gives bit-identical gradients to the recomputing backward."""
    import torch
    from tests.gpu_util import dev
    flags = TANH | UNG | DEC
    wl = datagen.small(variant + "_fwdbwd", "bf16", [200, 200], H=2, d=128, varlen=False)
    inp = datagen.make_inputs(wl, seed=303)
    q, k, v, dO = (dev(inp[n], torch.bfloat16, device).view(2, 200, 2, 128)
                   for n in ("q", "k", "v", "dO"))
    gates = [dev(inp[n], torch.float32, device).view(2, 200, 2)
             for n in ("alpha_s", "beta", "alpha_r", "gamma")]
    fwd = rla.rdn_forward if variant == "rdn" else rla.rla_forward
    bwd = rla.rdn_backward if variant == "rdn" else rla.rla_backward
    prob = rla.make_problem(q, v)
    op = rla.RLA_OP_RDN_BACKWARD if variant == "rdn" else rla.RLA_OP_RLA_BACKWARD
    ws = torch.empty(rla.rla_workspace_size(prob, op), dtype=torch.uint8, device=device)
    fwd(q, k, v, *gates, workspace=ws, save_for_backward=True, variants=flags)
    g1 = bwd(q, k, v, *gates, dO, workspace=ws, use_saved=True, variants=flags)
    g2 = bwd(q, k, v, *gates, dO, variants=flags)
    torch.cuda.synchronize()
    for key in GRAD_KEYS:
        assert torch.equal(g1[key], g2[key]), key


@pytest.mark.parametrize("flags", FLAGS, ids=[NAMES[f] for f in FLAGS])
@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_decode(device, variant, flags):
    from tests.test_parity_decode_gpu import gpu_decode
    B, H, d, T = 3, 2, 128, 7
    wl = datagen.small(variant + "_fwd", "bf16", [T] * B, H=H, d=d, varlen=False)
    inp = datagen.make_inputs(wl, seed=304)
    S0, R0 = datagen.random_states(34, B, H, d, d)
    for clip in (1.0, math.inf):
        o, Sf, Rf = gpu_decode(variant, inp, "bf16", device, B, clip=clip, S0=S0, R0=R0,
                               steps=T, in_place=True, variants=flags)
        ro, rS, rR = oracle_forward(variant, inp, clip=clip, S0=S0, R0=R0, variants=flags)
        report("decode %s %s c=%s" % (variant, NAMES[flags], clip),
               dict(o=rel_err(o, ro), S=rel_err(Sf, rS), R=rel_err(Rf, rR)), TOL["bf16"])


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_full_training_workload_all_variants(device):
    """The benchmarked training shape (B=4, T=4096, H=16, d=128, bf16) with all
    three variants on: forward and backward on the GPU at full size, every
    element of every (sequence, head) pair against the oracle (the log-cosh
    residual has no kink, so no input is moved)."""
    import torch
    from tests.gpu_util import dev, host
    from tests.test_parity_full_gpu import check_all
    flags = TANH | UNG | DEC
    wl = datagen.WORKLOADS[datagen.TRAINING]
    inp = datagen.make_inputs(wl, seed=305)
    B, T, H, d = wl.B, wl.T, wl.H, wl.dk
    q, k, v, dO = (dev(inp[n], torch.bfloat16, device).view(B, T, H, d) for n in ("q", "k", "v", "dO"))
    gates = [dev(inp[n], torch.float32, device).view(B, T, H)
             for n in ("alpha_s", "beta", "alpha_r", "gamma")]
    o, Sf, Rf = rla.rdn_forward(q, k, v, *gates, variants=flags)
    g = rla.rdn_backward(q, k, v, *gates, dO, variants=flags)
    torch.cuda.synchronize()
    got = dict(o=host(o).reshape(-1, H, d), S=host(Sf), R=host(Rf))
    for key in ("dq", "dk", "dv"):
        got[key] = host(g[key]).reshape(-1, H, d)
    for key in ("dalpha_s", "dbeta", "dalpha_r", "dgamma"):
        got[key] = host(g[key]).reshape(-1, H)
    for key in ("dS0", "dR0"):
        got[key] = host(g[key])
    ro, rS, rR = oracle_forward("rdn", inp, variants=flags)
    ref = oracle_backward("rdn", inp, variants=flags)
    want = dict(o=ro, S=rS, R=rR, **{key: ref[key] for key in GRAD_KEYS})
    check_all("full training shape, all variants", got, want, inp["cu_seqlens"], TOL["bf16"],
              token_keys=("o", "dq", "dk", "dv", "dalpha_s", "dbeta", "dalpha_r", "dgamma"))
