"""Pins of the fp64 oracle to facts the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a hand-worked
example, an exact reduction to a textbook recurrence, a closed form, an
invariant, brute-force finite differences, or an independent chunked
formulation.  All run on the CPU.
"""
import math
import os

import numpy as np
import pytest

import oracle
from oracle import chunked
from tests import textbook as tb

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rand_problem(seed, T=37, H=2, dk=8, dv=6, mu=2.0, states=False, unit=True):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((T, H, dk))
    k = rng.standard_normal((T, H, dk))
    if unit:
        q /= np.linalg.norm(q, axis=-1, keepdims=True)
        k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((T, H, dv))
    sig = lambda x: 1 / (1 + np.exp(-x))
    aS = sig(rng.standard_normal((T, H)) + mu)
    b = sig(rng.standard_normal((T, H)))
    aR = sig(rng.standard_normal((T, H)) + mu)
    g = sig(rng.standard_normal((T, H)))
    S0 = R0 = None
    if states:
        S0 = rng.standard_normal((1, H, dk, dv)) / math.sqrt(dk)
        R0 = rng.standard_normal((1, H, dk, dv)) / math.sqrt(dk)
    return dict(q=q, k=k, v=v, alpha_s=aS, beta=b, alpha_r=aR, gamma=g, S0=S0, R0=R0)


def fwd(variant, p, clip=1.0, **kw):
    args = dict(p)
    args.update(kw)
    return oracle.forward(variant, args["q"], args["k"], args["v"], args["alpha_s"], args["beta"],
                          args["alpha_r"], args["gamma"], clip=clip, S0=args["S0"], R0=args["R0"],
                          cu_seqlens=args.get("cu_seqlens"))


# ---------------------------------------------------------------------------
# Hand-worked example (tests/golden/hand_example_2tok.txt)
# ---------------------------------------------------------------------------

def _read_golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = line.split()
            vals[(parts[0], parts[1])] = np.array([float(x) for x in parts[2:]])
    return vals


@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_hand_worked_two_token_example(variant):
    gold = _read_golden("hand_example_2tok.txt")
    k = np.array([[1.0, 0.0], [0.6, 0.8]])[:, None, :]
    q = np.array([[1.0, 0.0], [0.0, 1.0]])[:, None, :]
    v = np.array([[2.0, 0.5], [0.0, 1.0]])[:, None, :]
    a = np.array([[0.5], [1.0]])
    o, S, R = oracle.forward(variant, q, k, v, a, a, a, a, clip=1.0)
    np.testing.assert_allclose(o[0, 0], gold[(variant, "o1")], atol=1e-14)
    np.testing.assert_allclose(o[1, 0], gold[(variant, "o2")], atol=1e-14)
    # stored transposed: element (i, j) = paper S[j][i]
    np.testing.assert_allclose(S[0, 0].T.ravel(), gold[(variant, "S2")], atol=1e-14)
    np.testing.assert_allclose(R[0, 0].T.ravel(), gold[(variant, "R2")], atol=1e-14)


# ---------------------------------------------------------------------------
# Exact reductions to textbook recurrences (Table 1; Sec. 3.1 special cases)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("clip_zero", [False, True])
def test_rdn_without_residual_branch_is_gated_delta_rule(clip_zero):
    """gamma = 0 (or c = 0) with R0 = 0 switches the residual branch off: R
    stays zero, S follows the gated delta rule, and o_t is that rule's base
    prediction a_t S_{t-1} q_t (Table 1, Gated DeltaNet row)."""
    p = rand_problem(1, states=True)
    p["R0"] = None
    if clip_zero:
        o, S, R = fwd("rdn", p, clip=0.0)
    else:
        p["gamma"] = np.zeros_like(p["gamma"])
        o, S, R = fwd("rdn", p)
    for h in range(p["q"].shape[1]):
        Ss = tb.gated_delta_states(p["k"][:, h], p["v"][:, h], p["alpha_s"][:, h], p["beta"][:, h],
                                   S0=p["S0"][0, h].T)
        np.testing.assert_allclose(S[0, h].T, Ss[-1], atol=1e-13)
        assert np.all(R[0, h] == 0.0)
        base = np.einsum("t,tjk,tk->tj", p["alpha_s"][:, h], Ss[:-1], p["q"][:, h])
        np.testing.assert_allclose(o[:, h], base, atol=1e-13)
        # and o differs from the gated-delta output S_t q_t by exactly the
        # single-token correction b_t (v_t - a_t S_{t-1} k_t)(k_t . q_t)
        gdn_out = np.einsum("tjk,tk->tj", Ss[1:], p["q"][:, h])
        corr = (p["beta"][:, h, None] * (p["v"][:, h] - p["alpha_s"][:, h, None] *
                np.einsum("tjk,tk->tj", Ss[:-1], p["k"][:, h])) *
                np.sum(p["k"][:, h] * p["q"][:, h], -1)[:, None])
        np.testing.assert_allclose(o[:, h] + corr, gdn_out, atol=1e-13)


def test_rdn_reduces_to_deltanet_readout():
    """aR = 0, no clip, gamma = sqrt(beta), aS = 1: R_t = gamma r_t k_t^T and
    o_t = S_{t-1}q_t + beta_t (v_t - S_{t-1}k_t) k_t.q_t = S_t q_t, the
    DeltaNet output (Table 1, DeltaNet row)."""
    p = rand_problem(2)
    p["alpha_s"] = np.ones_like(p["alpha_s"])
    p["alpha_r"] = np.zeros_like(p["alpha_r"])
    p["gamma"] = np.sqrt(p["beta"])
    o, S, R = fwd("rdn", p, clip=math.inf)
    for h in range(p["q"].shape[1]):
        Ss = tb.gated_delta_states(p["k"][:, h], p["v"][:, h], np.ones(len(p["k"])), p["beta"][:, h])
        np.testing.assert_allclose(o[:, h], np.einsum("tjk,tk->tj", Ss[1:], p["q"][:, h]), atol=1e-13)


def test_rla_reduces_to_one_step_delta_correction():
    """RLA with aR = 0, no clip, gamma = sqrt(beta): the correction becomes
    the one-step delta term beta_t (v_t - S_{t-1}k_t) k_t^T q_t (Sec. 3.1)."""
    p = rand_problem(3)
    p["alpha_r"] = np.zeros_like(p["alpha_r"])
    p["gamma"] = np.sqrt(p["beta"])
    o, S, R = fwd("rla", p, clip=math.inf)
    for h in range(p["q"].shape[1]):
        Ss = tb.scalar_gated_states(p["k"][:, h], p["v"][:, h], p["alpha_s"][:, h], p["beta"][:, h])
        prev = Ss[:-1]
        base = p["alpha_s"][:, h, None] * np.einsum("tjk,tk->tj", prev, p["q"][:, h])
        resid = p["v"][:, h] - np.einsum("tjk,tk->tj", prev, p["k"][:, h])
        corr = p["beta"][:, h, None] * resid * np.sum(p["k"][:, h] * p["q"][:, h], -1)[:, None]
        np.testing.assert_allclose(o[:, h], base + corr, atol=1e-13)


def test_rla_without_residual_branch_is_scalar_gated_la():
    """RLA with gamma = 0: S is scalar-gated linear attention's state (App. D
    baseline) and o_t = sGLA's o_t - beta_t v_t (k_t . q_t)."""
    p = rand_problem(4)
    p["gamma"] = np.zeros_like(p["gamma"])
    o, S, R = fwd("rla", p)
    for h in range(p["q"].shape[1]):
        Ss = tb.scalar_gated_states(p["k"][:, h], p["v"][:, h], p["alpha_s"][:, h], p["beta"][:, h])
        np.testing.assert_allclose(S[0, h].T, Ss[-1], atol=1e-13)
        sgla = np.einsum("tjk,tk->tj", Ss[1:], p["q"][:, h])
        corr = p["beta"][:, h, None] * p["v"][:, h] * np.sum(p["k"][:, h] * p["q"][:, h], -1)[:, None]
        np.testing.assert_allclose(o[:, h], sgla - corr, atol=1e-13)


@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_two_pass_composition(variant):
    """The paper computes the method as two passes of a base linear-attention
    rule (Sec. 4.1): the base pass on (k, v) yields the clipped residuals, and
    the same rule run on (k, r) with (aR, gamma) yields R.  Composing two
    textbook passes must reproduce the oracle exactly, with random S0, R0."""
    p = rand_problem(5, states=True)
    clip = 0.7
    o, S, R = fwd(variant, p, clip=clip)
    states = tb.gated_delta_states if variant == "rdn" else tb.scalar_gated_states
    for h in range(p["q"].shape[1]):
        k, q, v = p["k"][:, h], p["q"][:, h], p["v"][:, h]
        Ss = states(k, v, p["alpha_s"][:, h], p["beta"][:, h], S0=p["S0"][0, h].T)
        r = np.clip(v - np.einsum("tjk,tk->tj", Ss[:-1], k), -clip, clip)
        Rs = states(k, r, p["alpha_r"][:, h], p["gamma"][:, h], S0=p["R0"][0, h].T)
        out = (p["alpha_s"][:, h, None] * np.einsum("tjk,tk->tj", Ss[:-1], q) +
               p["gamma"][:, h, None] * np.einsum("tjk,tk->tj", Rs[1:], q))
        np.testing.assert_allclose(o[:, h], out, atol=1e-13)
        np.testing.assert_allclose(S[0, h].T, Ss[-1], atol=1e-13)
        np.testing.assert_allclose(R[0, h].T, Rs[-1], atol=1e-13)


# ---------------------------------------------------------------------------
# Closed forms and invariants
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_orthonormal_write_then_read(variant):
    """All gates 1, S0 = R0 = 0, orthonormal keys: every write lands in an
    orthogonal direction, so S_T k_j = v_j, and reading with q_t = k_t gives
    o_t = S_{t-1}k_t + R_t k_t = 0 + clip(v_t)."""
    rng = np.random.default_rng(6)
    d, T, c = 8, 8, 0.8
    Qm, _ = np.linalg.qr(rng.standard_normal((d, d)))
    k = Qm.T[:T][:, None, :]
    v = 1.5 * rng.standard_normal((T, 1, 5))
    ones = np.ones((T, 1))
    o, S, R = oracle.forward(variant, k, k, v, ones, ones, ones, ones, clip=c)
    np.testing.assert_allclose(o[:, 0], np.clip(v[:, 0], -c, c), atol=1e-13)
    np.testing.assert_allclose(S[0, 0].T @ k[:, 0].T, v[:, 0].T, atol=1e-13)
    # R stores the clipped residuals along the same keys
    np.testing.assert_allclose(R[0, 0].T @ k[:, 0].T, np.clip(v[:, 0], -c, c).T, atol=1e-13)


def test_repeated_key_overwrites():
    """RDN with beta = 1: writing the same key twice overwrites (S k = v2),
    and the second residual is clip(v2 - v1); reading with q = k at the
    second token returns v1 + clip(v2 - v1)."""
    k = np.array([0.6, 0.8])
    v1 = np.array([0.3, -2.0, 1.0])
    v2 = np.array([2.0, -1.5, 0.1])
    kk = np.stack([k, k])[:, None, :]
    vv = np.stack([v1, v2])[:, None, :]
    ones = np.ones((2, 1))
    o, S, R = oracle.forward("rdn", kk, kk, vv, ones, ones, ones, ones, clip=1.0)
    np.testing.assert_allclose(S[0, 0].T @ k, v2, atol=1e-14)
    np.testing.assert_allclose(o[1, 0], v1 + np.clip(v2 - v1, -1, 1), atol=1e-14)


def test_clip_is_negative_huber_gradient():
    """App. B: the clipped residual is the negative gradient of the Huber loss
    with threshold c at the prediction.  With the write/read set-up of the
    orthonormal test, o_t = r_t for a zero prediction, which must equal
    -dHuber/dv_hat at v_hat = 0, taken here by central differences of the
    Huber loss itself."""
    c = 0.9
    vals = np.array([-3.0, -0.95, -0.5, 0.0, 0.2, 0.85, 1.2, 4.0])
    T = len(vals)
    k = np.eye(T)[:, None, :]
    v = vals[:, None, None]
    ones = np.ones((T, 1))
    o, _, _ = oracle.forward("rla", k, k, v, ones, ones, ones, ones, clip=c)

    def huber(vhat, vv):
        e = abs(vv - vhat)
        return 0.5 * e * e if e <= c else c * (e - 0.5 * c)

    h = 1e-6
    neg_grad = np.array([-(huber(h, x) - huber(-h, x)) / (2 * h) for x in vals])
    np.testing.assert_allclose(o[:, 0, 0], neg_grad, atol=1e-8)


@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_linear_in_v_without_clip(variant):
    """With no clipping and zero initial states every stage is linear in v."""
    p = rand_problem(7)
    rng = np.random.default_rng(8)
    v2 = rng.standard_normal(p["v"].shape)
    o1, S1, R1 = fwd(variant, p, clip=math.inf)
    o2, S2, R2 = fwd(variant, p, clip=math.inf, v=v2)
    o3, S3, R3 = fwd(variant, p, clip=math.inf, v=p["v"] + 2.5 * v2)
    np.testing.assert_allclose(o3, o1 + 2.5 * o2, atol=1e-12)
    np.testing.assert_allclose(R3, R1 + 2.5 * R2, atol=1e-12)


@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_state_split_and_varlen(variant):
    """Running [0, t0) then [t0, T) with the final states passed on equals one
    call; a packed call with cu_seqlens equals separate calls."""
    p = rand_problem(9, T=50, states=True)
    o, S, R = fwd(variant, p)
    t0 = 23
    first = {key: (val[:t0] if key not in ("S0", "R0") else val) for key, val in p.items()}
    oa, Sa, Ra = fwd(variant, first)
    second = {key: (val[t0:] if key not in ("S0", "R0") else val) for key, val in p.items()}
    second["S0"], second["R0"] = Sa, Ra
    ob, Sb, Rb = fwd(variant, second)
    np.testing.assert_allclose(np.concatenate([oa, ob]), o, atol=1e-13)
    np.testing.assert_allclose(Sb, S, atol=1e-13)
    np.testing.assert_allclose(Rb, R, atol=1e-13)
    # packed: three sequences (one empty), each starting from its own state
    cu = np.array([0, 17, 17, 50])
    rng = np.random.default_rng(10)
    S0 = rng.standard_normal((3, 2, 8, 6))
    R0 = rng.standard_normal((3, 2, 8, 6))
    packed = dict(p, S0=S0, R0=R0, cu_seqlens=cu)
    op, Sp, Rp = fwd(variant, packed)
    for n in range(3):
        sl = slice(cu[n], cu[n + 1])
        sub = {key: (val[sl] if key not in ("S0", "R0") else val[n:n + 1]) for key, val in p.items()}
        sub["S0"], sub["R0"] = S0[n:n + 1], R0[n:n + 1]
        if cu[n + 1] == cu[n]:
            np.testing.assert_array_equal(Sp[n], S0[n])
            np.testing.assert_array_equal(Rp[n], R0[n])
            continue
        on, Sn, Rn = fwd(variant, sub)
        np.testing.assert_allclose(op[sl], on, atol=1e-13)
        np.testing.assert_allclose(Sp[n], Sn[0], atol=1e-13)
        np.testing.assert_allclose(Rp[n], Rn[0], atol=1e-13)


# ---------------------------------------------------------------------------
# Chunked formulation == token recurrence
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("chunk", [1, 3, 16, 64])
def test_chunked_equals_recurrent(variant, chunk):
    p = rand_problem(11, T=150, dk=16, dv=12, states=True)
    cu = np.array([0, 70, 150])
    rng = np.random.default_rng(12)
    S0 = rng.standard_normal((2, 2, 16, 12)) / 4
    R0 = rng.standard_normal((2, 2, 16, 12)) / 4
    args = (p["q"], p["k"], p["v"], p["alpha_s"], p["beta"], p["alpha_r"], p["gamma"])
    o, S, R = oracle.forward(variant, *args, clip=0.5, S0=S0, R0=R0, cu_seqlens=cu)
    oc, Sc, Rc = chunked.forward(variant, *args, clip=0.5, S0=S0, R0=R0, cu_seqlens=cu, chunk=chunk)
    np.testing.assert_allclose(oc, o, atol=1e-12)
    np.testing.assert_allclose(Sc, S, atol=1e-12)
    np.testing.assert_allclose(Rc, R, atol=1e-12)


# ---------------------------------------------------------------------------
# Backward == central finite differences of the forward
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("with_cu", [False, True])
def test_backward_matches_finite_differences(variant, with_cu):
    T, H, dk, dv = 14, 2, 5, 4
    p = rand_problem(13 + with_cu, T=T, H=H, dk=dk, dv=dv, states=False)
    rng = np.random.default_rng(20)
    cu = np.array([0, 6, T]) if with_cu else None
    N = 2 if with_cu else 1
    S0 = rng.standard_normal((N, H, dk, dv)) * 0.4
    R0 = rng.standard_normal((N, H, dk, dv)) * 0.4
    clip = 0.6
    gates = (p["alpha_s"], p["beta"], p["alpha_r"], p["gamma"])
    v, moved = oracle.nudge_margin(variant, p["q"], p["k"], p["v"], *gates, clip=clip, S0=S0, R0=R0,
                                   cu_seqlens=cu, margin=1e-3, grid="f64")
    inputs = dict(q=p["q"], k=p["k"], v=v, alpha_s=p["alpha_s"], beta=p["beta"],
                  alpha_r=p["alpha_r"], gamma=p["gamma"], S0=S0, R0=R0)
    dO = rng.standard_normal((T, H, dv))
    dSf = rng.standard_normal((N, H, dk, dv))
    dRf = rng.standard_normal((N, H, dk, dv))

    def loss(inp):
        o, S, R = oracle.forward(variant, inp["q"], inp["k"], inp["v"], inp["alpha_s"], inp["beta"],
                                 inp["alpha_r"], inp["gamma"], clip=clip, S0=inp["S0"], R0=inp["R0"],
                                 cu_seqlens=cu)
        return np.sum(o * dO) + np.sum(S * dSf) + np.sum(R * dRf)

    g = oracle.backward(variant, inputs["q"], inputs["k"], inputs["v"], inputs["alpha_s"],
                        inputs["beta"], inputs["alpha_r"], inputs["gamma"], dO, clip=clip, S0=S0,
                        R0=R0, dS_final=dSf, dR_final=dRf, cu_seqlens=cu)
    names = dict(q="dq", k="dk", v="dv", alpha_s="dalpha_s", beta="dbeta", alpha_r="dalpha_r",
                 gamma="dgamma", S0="dS0", R0="dR0")
    h = 1e-6
    for key, gkey in names.items():
        base = inputs[key]
        fd = np.zeros(base.size)
        for idx in range(base.size):
            plus = {kk: vv for kk, vv in inputs.items()}
            minus = dict(plus)
            a = base.copy().ravel(); a[idx] += h
            b = base.copy().ravel(); b[idx] -= h
            plus[key] = a.reshape(base.shape)
            minus[key] = b.reshape(base.shape)
            fd[idx] = (loss(plus) - loss(minus)) / (2 * h)
        an = g[gkey].ravel()
        scale = max(1.0, np.max(np.abs(fd)))
        err = np.max(np.abs(an - fd)) / scale
        assert err < 1e-6, (gkey, err)


def test_nudge_keeps_margin_and_grid():
    """The kink-margin helper leaves every pre-clip residual at least the
    margin away from +-c and keeps moved values on the bf16 grid."""
    import datagen
    p = rand_problem(30, T=64, H=2, dk=16, dv=16)
    v = datagen.round_to_bf16(p["v"]).astype(np.float64)
    gates = (p["alpha_s"], p["beta"], p["alpha_r"], p["gamma"])
    vn, moved = oracle.nudge_margin("rdn", p["q"], p["k"], v, *gates, clip=1.0, margin=1e-2, grid="bf16")
    assert moved > 0
    np.testing.assert_array_equal(datagen.round_to_bf16(vn).astype(np.float64), vn)
    # re-derive the residuals token by token with the textbook gated delta rule
    for h in range(2):
        Ss = tb.gated_delta_states(p["k"][:, h], vn[:, h], p["alpha_s"][:, h], p["beta"][:, h])
        x = vn[:, h] - np.einsum("tjk,tk->tj", Ss[:-1], p["k"][:, h])
        assert np.min(np.abs(np.abs(x) - 1.0)) >= 1e-2 - 1e-12
