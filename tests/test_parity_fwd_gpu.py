"""GPU forward parity: rla_forward / rdn_forward through the C ABI against the
fp64 oracle on identical seeded inputs (element by element)."""
import math

import numpy as np
import pytest

import datagen
from tests.gpu_util import TOL, gpu_forward, oracle_forward, rel_err

pytestmark = pytest.mark.gpu


def check(variant, inp, dtype, device, clip=1.0, S0=None, R0=None, dense_B=None, label=""):
    o, Sf, Rf = gpu_forward(variant, inp, dtype, device, clip=clip, S0=S0, R0=R0, dense_B=dense_B)
    ro, rS, rR = oracle_forward(variant, inp, clip=clip, S0=S0, R0=R0)
    errs = dict(o=rel_err(o, ro), S=rel_err(Sf, rS), R=rel_err(Rf, rR))
    print("[%s %s %s] %s" % (variant, dtype, label, " ".join("%s=%.2e" % kv for kv in errs.items())))
    for key, e in errs.items():
        assert e <= TOL[dtype], (key, e)
    return errs


# --- small cases: several chunks, a ragged tail, both dtypes -----------------

@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("dtype,d,dv", [("f32", 64, 64), ("f32", 64, 128), ("bf16", 128, 128),
                                        ("bf16", 64, 64), ("bf16", 128, 64), ("bf16", 64, 128)])
def test_dense_ragged(device, variant, dtype, d, dv):
    wl = datagen.small(variant + "_fwd", dtype, [200, 200], H=3, d=d, dv=dv, varlen=False)
    inp = datagen.make_inputs(wl, seed=101)
    check(variant, inp, dtype, device, dense_B=2, label="B2 T200 d%d dv%d" % (d, dv))


@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("dtype,d", [("f32", 64), ("bf16", 128)])
def test_initial_states_and_clip_variants(device, variant, dtype, d):
    wl = datagen.small(variant + "_fwd", dtype, [130], H=2, d=d, varlen=False)
    inp = datagen.make_inputs(wl, seed=102)
    S0, R0 = datagen.random_states(7, 1, 2, d, d)
    check(variant, inp, dtype, device, S0=S0, R0=R0, dense_B=1, label="S0R0")
    check(variant, inp, dtype, device, clip=math.inf, dense_B=1, label="noclip")
    check(variant, inp, dtype, device, clip=0.0, dense_B=1, label="clip0")


@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("dtype,d", [("f32", 64), ("bf16", 128)])
def test_varlen_edges(device, variant, dtype, d):
    """Sequence lengths at and around the chunk size, an empty sequence, and a
    single token; states reset per sequence; final states per sequence."""
    lens = [1, 63, 0, 64, 65, 127, 200]
    wl = datagen.small(variant + "_fwd", dtype, lens, H=2, d=d)
    inp = datagen.make_inputs(wl, seed=103)
    S0, R0 = datagen.random_states(8, len(lens), 2, d, d)
    check(variant, inp, dtype, device, S0=S0, R0=R0, label="varlen")


@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_bf16_outputs(device, variant):
    """o stored in bf16: the kernel error bound plus the output rounding
    itself (at most 2^-8 |o| per element, i.e. 2^-8 max|o| / RMS(o))."""
    import torch
    from tests.gpu_util import dev, host
    import paper_2509_25223_amd as rla
    wl = datagen.small(variant + "_fwd", "bf16", [333], H=2, d=128, varlen=False)
    inp = datagen.make_inputs(wl, seed=104)
    q, k, v = (dev(inp[n], torch.bfloat16, device)[None] for n in ("q", "k", "v"))
    g = [dev(inp[n], torch.float32, device)[None] for n in ("alpha_s", "beta", "alpha_r", "gamma")]
    fn = rla.rdn_forward if variant == "rdn" else rla.rla_forward
    o, _, _ = fn(q, k, v, *g, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert o.dtype == torch.bfloat16
    ro, _, _ = oracle_forward(variant, inp)
    rms = np.sqrt(np.mean(ro ** 2))
    allow = TOL["bf16"] + 2.0 ** -8 * np.max(np.abs(ro)) / rms
    e = rel_err(host(o)[0], ro)
    print("[%s bf16-out] o=%.2e allowance=%.2e" % (variant, e, allow))
    assert e <= allow


def test_empty_problem(device):
    import torch
    import paper_2509_25223_amd as rla
    q = torch.zeros(2, 0, 2, 64, device=device, dtype=torch.bfloat16)
    g = torch.zeros(2, 0, 2, device=device)
    S0 = torch.randn(2, 2, 64, 64, device=device)
    o, Sf, Rf = rla.rdn_forward(q, q, q, g, g, g, g, S0=S0, R0=S0)
    torch.cuda.synchronize()
    assert o.shape == q.shape
    assert torch.equal(Sf, S0) and torch.equal(Rf, S0)
