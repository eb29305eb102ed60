"""GPU backward parity: rdn_backward / rla_backward through the C ABI against
the oracle's hand-derived adjoint (itself pinned to finite differences), on
identical seeded inputs, for all nine gradient tensors.

Clip masks are a step function of the residual; the inputs are moved (on the
input dtype's grid) so no residual lies within 1e-2 (bf16) / 1e-4 (fp32) of
the kink, so both sides take the same mask."""
import math

import numpy as np
import pytest

import datagen
from tests.gpu_util import GRAD_KEYS, TOL, gpu_backward, nudge, oracle_backward, rel_err

pytestmark = pytest.mark.gpu


def check(variant, inp, dtype, device, clip=1.0, S0=None, R0=None, dSf=None, dRf=None,
          dense_B=None, label="", out_dtype=None):
    inp, moved = nudge(variant, inp, dtype, clip=clip, S0=S0, R0=R0)
    g = gpu_backward(variant, inp, dtype, device, clip=clip, S0=S0, R0=R0, dS_final=dSf,
                     dR_final=dRf, dense_B=dense_B, out_dtype=out_dtype)
    ref = oracle_backward(variant, inp, clip=clip, S0=S0, R0=R0, dS_final=dSf, dR_final=dRf)
    errs = {key: rel_err(g[key], ref[key]) for key in GRAD_KEYS}
    if out_dtype is not None:   # dq, dk, dv rounded once to bf16 on the way out
        for key in ("dq", "dk", "dv"):
            errs[key] = rel_err_rounded(g[key], ref[key], 2.0 ** -8)
    print("[%s %s %s moved=%d] %s" % (variant, dtype, label, moved,
                                      " ".join("%s=%.1e" % kv for kv in errs.items())))
    for key, e in errs.items():
        assert e <= TOL[dtype], (key, e)


def rel_err_rounded(x, ref, half_ulp):
    """max(|x - ref| - half_ulp |ref|, 0) / RMS(ref): what is left of the error
    once each value's own rounding to the output format (relative half-ulp
    half_ulp: 2^-8 for bf16's 8 significant bits) is set aside.  A plain
    max|x - ref| / RMS would be dominated by that rounding of the largest
    gradients (about 10x the RMS), which the computation cannot avoid."""
    ref = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref)))
    d = np.abs(np.asarray(x, np.float64) - ref) - half_ulp * np.abs(ref)
    return float(np.max(np.maximum(d, 0.0))) / rms


@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("dtype,d,dv", [("f32", 64, 64), ("bf16", 128, 128), ("bf16", 64, 64),
                                        ("bf16", 64, 128), ("bf16", 128, 64)])
def test_dense_ragged(device, variant, dtype, d, dv):
    wl = datagen.small(variant + "_fwdbwd", dtype, [150, 150], H=2, d=d, dv=dv, varlen=False)
    inp = datagen.make_inputs(wl, seed=201)
    check(variant, inp, dtype, device, dense_B=2, label="B2 T150 d%d dv%d" % (d, dv))


@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("dtype,d", [("f32", 64), ("bf16", 128)])
def test_states_in_and_out(device, variant, dtype, d):
    """Non-zero S0, R0 and upstream gradients on the final states."""
    wl = datagen.small(variant + "_fwdbwd", dtype, [100], H=2, d=d, varlen=False)
    inp = datagen.make_inputs(wl, seed=202)
    S0, R0 = datagen.random_states(9, 1, 2, d, d)
    dSf, dRf = datagen.random_states(10, 1, 2, d, d, scale=1.0)
    check(variant, inp, dtype, device, S0=S0, R0=R0, dSf=dSf, dRf=dRf, dense_B=1, label="states")
    check(variant, inp, dtype, device, clip=math.inf, S0=S0, R0=R0, dense_B=1, label="noclip")


@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("dtype,d", [("f32", 64), ("bf16", 128)])
def test_varlen_edges(device, variant, dtype, d):
    lens = [1, 63, 0, 64, 65, 130]
    wl = datagen.small(variant + "_fwdbwd", dtype, lens, H=2, d=d)
    inp = datagen.make_inputs(wl, seed=203)
    S0, R0 = datagen.random_states(11, len(lens), 2, d, d)
    check(variant, inp, dtype, device, S0=S0, R0=R0, label="varlen")


@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("scale", ["2^-30", "2^-20", "2^12", "chunkwise"])
def test_upstream_gradient_scale(device, variant, scale):
    """The upstream gradients dO, dS_T, dR_T multiplied by 2^-30, 2^-20, 2^12
    (exact in bf16 and fp32; bf16 training without loss scaling sees the small
    ones), or dO shrinking 4x per chunk along each sequence: every gradient
    scales with them, so the relative bound applies unchanged.  Unscaled fp16
    operands would flush the small cases to zero and overflow the large one."""
    lens = [300, 70]
    wl = datagen.small(variant + "_fwdbwd", "bf16", lens, H=2, d=128)
    inp = datagen.make_inputs(wl, seed=205)
    S0, R0 = datagen.random_states(12, len(lens), 2, 128, 128)
    dSf, dRf = datagen.random_states(13, len(lens), 2, 128, 128, scale=1.0)
    if scale == "chunkwise":
        cu = inp["cu_seqlens"]
        f = np.concatenate([4.0 ** -(np.arange(cu[n + 1] - cu[n]) // 64) for n in range(len(lens))])
        inp["dO"] = (inp["dO"] * f[:, None, None]).astype(np.float32)
        dSf = dRf = None
    else:
        f = 2.0 ** int(scale[2:])
        inp["dO"] = (inp["dO"] * f).astype(np.float32)
        dSf, dRf = (dSf * f).astype(np.float32), (dRf * f).astype(np.float32)
    check(variant, inp, "bf16", device, S0=S0, R0=R0, dSf=dSf, dRf=dRf, label="dO x %s" % scale)


@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_bf16_outputs(device, variant):
    """dq, dk, dv returned in bf16 (out_dtype): the same gradients rounded once
    to bf16, compared with the bound after setting that rounding aside
    (rel_err_rounded); ragged lengths, so the row masks of the dv stores and
    the partial chunks are hit."""
    import torch
    lens = [1, 63, 130, 64]
    wl = datagen.small(variant + "_fwdbwd", "bf16", lens, H=2, d=128)
    inp = datagen.make_inputs(wl, seed=204)
    check(variant, inp, "bf16", device, out_dtype=torch.bfloat16, label="bf16 out")


@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("varlen", [False, True])
def test_saved_forward_path_is_identical(device, variant, varlen):
    """forward(save_for_backward) + backward(use_saved) gives bit-identical
    outputs and gradients to the self-contained calls (same kernels, same
    arithmetic; the backward only skips recomputing what the forward left)."""
    import torch
    import paper_2509_25223_amd as rla
    from tests.gpu_util import dev
    lens = [70, 0, 130] if varlen else [150, 150]
    wl = datagen.small(variant + "_fwdbwd", "bf16", lens, H=2, d=128, varlen=varlen)
    inp = datagen.make_inputs(wl, seed=204)
    q, k, v, dO = (dev(inp[n], torch.bfloat16, device) for n in ("q", "k", "v", "dO"))
    g = [dev(inp[n], torch.float32, device) for n in ("alpha_s", "beta", "alpha_r", "gamma")]
    cu = None
    if varlen:
        cu = torch.from_numpy(inp["cu_seqlens"].astype(np.int32)).to(device)
    else:
        q, k, v, dO = (x.view(2, 150, *x.shape[1:]) for x in (q, k, v, dO))
        g = [x.view(2, 150, -1) for x in g]
    fwd = rla.rdn_forward if variant == "rdn" else rla.rla_forward
    bwd = rla.rdn_backward if variant == "rdn" else rla.rla_backward
    o1, S1, R1 = fwd(q, k, v, *g, cu_seqlens=cu)
    ref = bwd(q, k, v, *g, dO, cu_seqlens=cu)
    prob = rla.make_problem(q, v, cu)
    ws = torch.empty(rla.rla_workspace_size(prob, rla.RLA_OP_RDN_BACKWARD if variant == "rdn"
                                            else rla.RLA_OP_RLA_BACKWARD),
                     dtype=torch.uint8, device=device)
    o2, S2, R2 = fwd(q, k, v, *g, cu_seqlens=cu, workspace=ws, save_for_backward=True)
    got = bwd(q, k, v, *g, dO, cu_seqlens=cu, workspace=ws, use_saved=True)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(S1, S2) and torch.equal(R1, R2)
    for key in GRAD_KEYS:
        assert torch.equal(ref[key], got[key]), key
