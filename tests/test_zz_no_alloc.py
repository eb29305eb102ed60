"""The allocation-free RDN forward (rdn_forward_noalloc, for callers that
cannot allocate) against rdn_forward through the C ABI: the same kernels with
the workspace taken from the library's static per-device scratch array, so
the outputs must be bit-identical.  Two calls in a row, the second with a
smaller problem, so the second runs on an array still holding the first
call's contents; the first is also held to the bf16 bound against the
oracle."""
import numpy as np
import pytest

import datagen
import paper_2509_25223_amd as rla
from tests.gpu_util import TOL, dev, host, oracle_forward, rel_err

pytestmark = pytest.mark.gpu


def run_both(inp, varlen, B, H, d, device):
    import torch
    q, k, v = (dev(inp[n], torch.bfloat16, device) for n in ("q", "k", "v"))
    gates = [dev(inp[n], torch.float32, device) for n in ("alpha_s", "beta", "alpha_r", "gamma")]
    cu = None
    if varlen:
        cu = torch.from_numpy(np.asarray(inp["cu_seqlens"], np.int32)).to(device)
    else:
        T = q.shape[0] // B
        q, k, v = (x.view(B, T, H, d) for x in (q, k, v))
        gates = [g.view(B, T, H) for g in gates]
    N = len(inp["cu_seqlens"]) - 1
    S0, R0 = (dev(x, torch.float32, device) for x in datagen.random_states(61, N, H, d, d))
    ref = rla.rdn_forward(q, k, v, *gates, S0=S0, R0=R0, cu_seqlens=cu)
    # outputs allocated up front: the call itself allocates nothing
    o = torch.full(v.shape, float("nan"), dtype=torch.float32, device=device)
    Sf = torch.full((N, H, d, d), float("nan"), dtype=torch.float32, device=device)
    Rf = torch.full((N, H, d, d), float("nan"), dtype=torch.float32, device=device)
    got = rla.rdn_forward_noalloc(q, k, v, *gates, S0=S0, R0=R0, cu_seqlens=cu, out=o,
                                  S_final=Sf, R_final=Rf)
    torch.cuda.synchronize()
    return ref, got, host(S0), host(R0)


def test_noalloc_forward_matches_rdn_forward(device):
    import torch
    H, d = 4, 128
    # first call: three packed sequences (1830 tokens); second: one dense 300-token sequence
    cases = [([1000, 700, 130], True, 1, 501), ([300], False, 1, 502)]
    for n_call, (lens, varlen, B, seed) in enumerate(cases):
        wl = datagen.small("rdn_fwd", "bf16", lens, H=H, d=d, varlen=varlen)
        inp = datagen.make_inputs(wl, seed=seed)
        ref, got, S0, R0 = run_both(inp, varlen, B, H, d, device)
        for a, b, name in zip(ref, got, ("o", "S_final", "R_final")):
            assert torch.equal(a, b), (n_call, name)
        ro, rS, rR = oracle_forward("rdn", inp, S0=S0, R0=R0)
        errs = dict(o=rel_err(host(got[0]).reshape(ro.shape), ro), S=rel_err(host(got[1]), rS),
                    R=rel_err(host(got[2]), rR))
        print("[noalloc call %d, %d tokens] bit-identical to rdn_forward; %s" % (
            n_call + 1, sum(lens), " ".join("%s=%.2e" % kv for kv in errs.items())), flush=True)
        for key, e in errs.items():
            assert e <= TOL["bf16"], (n_call, key, e)


def test_noalloc_forward_rejects_oversized_problem(device):
    import torch
    q = torch.zeros(1, 19712, 16, 128, dtype=torch.bfloat16, device=device)
    g = torch.zeros(1, 19712, 16, dtype=torch.float32, device=device)
    with pytest.raises(rla.RLAError) as err:
        rla.rdn_forward_noalloc(q, q, q, g, g, g, g)
    assert err.value.status == rla.RLA_ERR_SCRATCH
