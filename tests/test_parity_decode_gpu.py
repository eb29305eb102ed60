"""GPU parity of the recurrent (decoding) step: rla_decode / rdn_decode through
the C ABI against the fp64 oracle's token recurrence on identical seeded
inputs, element by element (o, S_out, R_out)."""
import math

import numpy as np
import pytest

import datagen
from tests.gpu_util import TOL, dev, host, oracle_forward, rel_err, torch_dtype

pytestmark = pytest.mark.gpu


def gpu_decode(variant, inp, dtype, device, B, clip=1.0, S0=None, R0=None, steps=1,
               out_dtype=None, in_place=False, variants=0):
    """Runs the packed inputs (B sequences of equal length T) through `steps`
    decode calls of T / steps tokens each, carrying the states between calls."""
    import torch
    import paper_2509_25223_amd as rla
    td = torch_dtype(dtype)
    q, k, v = (dev(inp[n], td, device) for n in ("q", "k", "v"))
    gates = [dev(inp[n], torch.float32, device) for n in ("alpha_s", "beta", "alpha_r", "gamma")]
    T = q.shape[0] // B
    q, k, v = (x.view(B, T, *x.shape[1:]) for x in (q, k, v))
    gates = [g.view(B, T, -1) for g in gates]
    Sd = None if S0 is None else dev(S0, torch.float32, device)
    Rd = None if R0 is None else dev(R0, torch.float32, device)
    fn = rla.rdn_decode if variant == "rdn" else rla.rla_decode
    per = T // steps
    assert per * steps == T
    outs = []
    for s in range(steps):
        sl = slice(s * per, (s + 1) * per)
        args = [x[:, sl].contiguous() for x in (q, k, v)] + [g[:, sl].contiguous() for g in gates]
        if in_place and Sd is not None:
            o, Sd, Rd = fn(*args, clip=clip, S_in=Sd, R_in=Rd, S_out=Sd, R_out=Rd,
                           out_dtype=out_dtype, variants=variants)
        else:
            o, Sd, Rd = fn(*args, clip=clip, S_in=Sd, R_in=Rd, out_dtype=out_dtype,
                           variants=variants)
        outs.append(o)
    o = torch.cat(outs, dim=1) if outs else torch.empty(0)
    torch.cuda.synchronize()
    return host(o).reshape(-1, *o.shape[-2:]), host(Sd), host(Rd)


def check(variant, inp, dtype, device, B, clip=1.0, S0=None, R0=None, steps=1, label="",
          tol=None, **kw):
    o, Sf, Rf = gpu_decode(variant, inp, dtype, device, B, clip=clip, S0=S0, R0=R0, steps=steps, **kw)
    ro, rS, rR = oracle_forward(variant, inp, clip=clip, S0=S0, R0=R0)
    errs = dict(o=rel_err(o, ro), S=rel_err(Sf, rS), R=rel_err(Rf, rR))
    print("[decode %s %s %s] %s" % (variant, dtype, label, " ".join("%s=%.2e" % kv for kv in errs.items())))
    bound = TOL[dtype] if tol is None else tol
    for key, e in errs.items():
        assert e <= bound, (key, e)
    return errs


def inputs(variant, dtype, B, T, H, d, dv=None, seed=0):
    wl = datagen.small(variant + "_fwd", dtype, [T] * B, H=H, d=d, dv=dv, varlen=False,
                       decay_mu=3.0 if variant == "rla" else 2.0)
    return datagen.make_inputs(wl, seed=seed)


@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("dtype,d,dv", [("f32", 64, 64), ("f32", 128, 128), ("f32", 64, 128),
                                        ("bf16", 128, 128), ("bf16", 128, 64), ("bf16", 64, 128)])
def test_one_token(device, variant, dtype, d, dv):
    """One generated token per sequence from random states: the serving step."""
    B, H = 5, 3
    inp = inputs(variant, dtype, B, 1, H, d, dv, seed=201)
    S0, R0 = datagen.random_states(21, B, H, d, dv)
    check(variant, inp, dtype, device, B, S0=S0, R0=R0, label="T1 d%d dv%d" % (d, dv))


@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("dtype,d", [("f32", 64), ("bf16", 128)])
def test_several_tokens_clip_variants(device, variant, dtype, d):
    """T = 7 tokens per call; no clipping and c = 0 as well as c = 1."""
    B, H = 3, 2
    inp = inputs(variant, dtype, B, 7, H, d, seed=202)
    S0, R0 = datagen.random_states(22, B, H, d, d)
    check(variant, inp, dtype, device, B, S0=S0, R0=R0, label="T7")
    check(variant, inp, dtype, device, B, clip=math.inf, S0=S0, R0=R0, label="T7 noclip")
    check(variant, inp, dtype, device, B, clip=0.0, S0=S0, R0=R0, label="T7 clip0")
    check(variant, inp, dtype, device, B, label="T7 zero states")


@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_in_place_generation_matches_chunked_forward(device, variant):
    """150 single-token steps updating the states in place equal the oracle
    over the 150 tokens and the chunked GPU forward (three chunks, ragged)."""
    import torch
    import paper_2509_25223_amd as rla
    B, H, d, T = 2, 2, 128, 150
    inp = inputs(variant, "bf16", B, T, H, d, seed=203)
    S0, R0 = datagen.random_states(23, B, H, d, d)
    o, Sf, Rf = gpu_decode(variant, inp, "bf16", device, B, S0=S0, R0=R0, steps=T, in_place=True)
    ro, rS, rR = oracle_forward(variant, inp, S0=S0, R0=R0)
    errs = dict(o=rel_err(o, ro), S=rel_err(Sf, rS), R=rel_err(Rf, rR))
    print("[decode %s in place x%d] %s" % (variant, T, " ".join("%s=%.2e" % kv for kv in errs.items())))
    for key, e in errs.items():
        assert e <= TOL["bf16"], (key, e)
    # the chunked forward on the same device inputs agrees within both bounds
    td = torch.bfloat16
    q, k, v = (dev(inp[n], td, device).view(B, T, H, d) for n in ("q", "k", "v"))
    gates = [dev(inp[n], torch.float32, device).view(B, T, H)
             for n in ("alpha_s", "beta", "alpha_r", "gamma")]
    fn = rla.rdn_forward if variant == "rdn" else rla.rla_forward
    oc, Sc, Rc = fn(q, k, v, *gates, S0=dev(S0, torch.float32, device), R0=dev(R0, torch.float32, device))
    torch.cuda.synchronize()
    assert rel_err(o, host(oc).reshape(-1, H, d)) <= 2 * TOL["bf16"]
    assert rel_err(Sf, host(Sc)) <= 2 * TOL["bf16"]


def test_bf16_output_and_empty_cases(device):
    import torch
    import paper_2509_25223_amd as rla
    B, H, d = 4, 2, 128
    inp = inputs("rdn", "bf16", B, 1, H, d, seed=204)
    S0, R0 = datagen.random_states(24, B, H, d, d)
    ro, _, _ = oracle_forward("rdn", inp, S0=S0, R0=R0)
    # bf16 output rounding adds at most 2^-8 max|o| / RMS(o)
    rms = float(np.sqrt(np.mean(ro * ro)))
    extra = 2.0 ** -8 * float(np.max(np.abs(ro))) / rms
    check("rdn", inp, "bf16", device, B, S0=S0, R0=R0, label="bf16 out",
          tol=TOL["bf16"] + extra, out_dtype=torch.bfloat16)
    # T = 0: the states are copied through and nothing else is written
    z = torch.zeros(B, 0, H, d, dtype=torch.bfloat16, device=device)
    zg = torch.zeros(B, 0, H, dtype=torch.float32, device=device)
    Sd, Rd = dev(S0, torch.float32, device), dev(R0, torch.float32, device)
    o, So, Ro = rla.rdn_decode(z, z, z, zg, zg, zg, zg, S_in=Sd, R_in=Rd)
    torch.cuda.synchronize()
    assert o.numel() == 0
    assert torch.equal(So, Sd) and torch.equal(Ro, Rd)
    # B = 0: nothing to do
    e = torch.zeros(0, 1, H, d, dtype=torch.bfloat16, device=device)
    eg = torch.zeros(0, 1, H, dtype=torch.float32, device=device)
    o, So, Ro = rla.rdn_decode(e, e, e, eg, eg, eg, eg)
    assert o.numel() == 0 and So.numel() == 0


@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_full_serving_batch(device, variant):
    """The benchmarked decode shape: 256 sequences x 16 heads, d = 128, bf16,
    one token each from random states, every output checked."""
    B, H, d = 256, 16, 128
    inp = inputs(variant, "bf16", B, 1, H, d, seed=205)
    S0, R0 = datagen.random_states(25, B, H, d, d)
    check(variant, inp, "bf16", device, B, S0=S0, R0=R0, label="B256 H16 d128")
