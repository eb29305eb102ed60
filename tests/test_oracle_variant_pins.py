"""Pins of the oracle's variants to facts the paper and the mathematics fix.

The variants are the paper's alternatives to the boxed formulation of
Sec. 3.4: the log-cosh residual r = c tanh(x / c) (App. B), the ungated
output S_{t-1} q_t + R_t q_t (the output-combination ablation of Sec. 4.3)
and the residual of the decayed prediction x_t = v_t - a_t S_{t-1} k_t (the
prediction of Table 1's gated rows).  Every pin compares the oracle with
something other than itself: the derivative of the loss the residual comes
from, exact reductions to the boxed formulation or to textbook recurrences,
read-outs of independently computed states, the chunked formulation, and
central finite differences for the hand-derived backward.  CPU only.
"""
import math

import numpy as np
import pytest

import oracle
from oracle import chunked
from tests import textbook as tb

ALL = oracle.TANH | oracle.UNGATED | oracle.DECAYED


def rand_problem(seed, T=37, H=2, dk=8, dv=6, mu=2.0):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((T, H, dk))
    k = rng.standard_normal((T, H, dk))
    q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((T, H, dv))
    sig = lambda x: 1 / (1 + np.exp(-x))
    return dict(q=q, k=k, v=v, alpha_s=sig(rng.standard_normal((T, H)) + mu),
                beta=sig(rng.standard_normal((T, H))),
                alpha_r=sig(rng.standard_normal((T, H)) + mu),
                gamma=sig(rng.standard_normal((T, H))), S0=None, R0=None)


def fwd(variant, p, clip=1.0, flags=0, **kw):
    a = dict(p)
    a.update(kw)
    return oracle.forward(variant, a["q"], a["k"], a["v"], a["alpha_s"], a["beta"], a["alpha_r"],
                          a["gamma"], clip=clip, S0=a["S0"], R0=a["R0"],
                          cu_seqlens=a.get("cu_seqlens"), flags=flags)


# --- log-cosh residual --------------------------------------------------------

@pytest.mark.parametrize("c", [1.0, 0.7])
def test_tanh_is_negative_logcosh_gradient(c):
    """App. B: the log-cosh loss's negative gradient at the prediction is tanh
    of the residual (scaled form: loss c^2 log cosh(e / c), gradient
    c tanh(e / c); c = 1 is the paper's).  Orthonormal keys, q = k and unit
    gates make o_t = r_t for a zero prediction (RLA), compared with central
    differences of the loss itself."""
    vals = np.array([-3.0, -0.95, -0.5, 0.0, 0.2, 0.85, 1.2, 4.0])
    T = len(vals)
    k = np.eye(T)[:, None, :]
    v = vals[:, None, None]
    ones = np.ones((T, 1))
    o, _, _ = oracle.forward("rla", k, k, v, ones, ones, ones, ones, clip=c, flags=oracle.TANH)

    def logcosh(vhat, vv):
        return c * c * math.log(math.cosh((vv - vhat) / c))

    h = 1e-6
    neg_grad = np.array([-(logcosh(h, x) - logcosh(-h, x)) / (2 * h) for x in vals])
    np.testing.assert_allclose(o[:, 0, 0], neg_grad, atol=1e-8)


@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_tanh_limits(variant):
    """c = inf: r = x, the unclipped forward exactly; c = 0: r = 0, the same
    as clipping at 0; a very large c agrees with no clipping to O(x^3 / c^2)."""
    p = rand_problem(40)
    ref_inf = fwd(variant, p, clip=math.inf)
    got_inf = fwd(variant, p, clip=math.inf, flags=oracle.TANH)
    ref_zero = fwd(variant, p, clip=0.0)
    got_zero = fwd(variant, p, clip=0.0, flags=oracle.TANH)
    got_big = fwd(variant, p, clip=1e4, flags=oracle.TANH)
    for a, b in zip(ref_inf, got_inf):
        np.testing.assert_array_equal(a, b)
    for a, b in zip(ref_zero, got_zero):
        np.testing.assert_array_equal(a, b)
    for a, b in zip(ref_inf, got_big):
        np.testing.assert_allclose(a, b, atol=1e-6)


# --- ungated output ------------------------------------------------------------

@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_ungated_equals_gated_at_unit_weights(variant):
    """With aS = 1 and gamma = 1 the two output combinations coincide."""
    p = rand_problem(41)
    p["alpha_s"] = np.ones_like(p["alpha_s"])
    p["gamma"] = np.ones_like(p["gamma"])
    a = fwd(variant, p)
    b = fwd(variant, p, flags=oracle.UNGATED)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_ungated_output_reads_the_states(variant):
    """o_t = S_{t-1} q_t + R_t q_t with S_{t-1} and R_t taken from separate
    calls on the prefixes [0, t) and [0, t]; the states do not depend on the
    output combination."""
    p = rand_problem(42, T=12)
    o, S, R = fwd(variant, p, flags=oracle.UNGATED)
    _, Sg, Rg = fwd(variant, p)
    np.testing.assert_array_equal(S, Sg)
    np.testing.assert_array_equal(R, Rg)
    for t in range(1, 12):
        pre = {key: (val[:t] if key not in ("S0", "R0") else val) for key, val in p.items()}
        inc = {key: (val[:t + 1] if key not in ("S0", "R0") else val) for key, val in p.items()}
        _, S_prev, _ = fwd(variant, pre)
        _, _, R_t = fwd(variant, inc)
        q = p["q"][t]   # [H, dk]; states [1, H, dk, dv] (transposed)
        want = np.einsum("hi,hij->hj", q, S_prev[0]) + np.einsum("hi,hij->hj", q, R_t[0])
        np.testing.assert_allclose(o[t], want, atol=1e-13)


# --- decayed residual ----------------------------------------------------------

@pytest.mark.parametrize("variant", ["rdn", "rla"])
def test_decayed_equals_literal_at_unit_decay(variant):
    p = rand_problem(43)
    p["alpha_s"] = np.ones_like(p["alpha_s"])
    a = fwd(variant, p)
    b = fwd(variant, p, flags=oracle.DECAYED)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def test_decayed_rdn_reads_out_the_gated_delta_rule_for_any_decay():
    """With the decayed residual, aR = 0, no clip and gamma = sqrt(beta), the
    correction is beta_t (v_t - a_t S_{t-1} k_t)(k_t . q_t), so o_t = S_t q_t
    of the gated delta rule (Table 1, Gated DeltaNet row) for any decay a_t;
    the boxed (undecayed) residual gives this only for a_t = 1."""
    p = rand_problem(44)
    p["alpha_r"] = np.zeros_like(p["alpha_r"])
    p["gamma"] = np.sqrt(p["beta"])
    o, _, _ = fwd("rdn", p, clip=math.inf, flags=oracle.DECAYED)
    o_lit, _, _ = fwd("rdn", p, clip=math.inf)
    for h in range(p["q"].shape[1]):
        Ss = tb.gated_delta_states(p["k"][:, h], p["v"][:, h], p["alpha_s"][:, h], p["beta"][:, h])
        want = np.einsum("tjk,tk->tj", Ss[1:], p["q"][:, h])
        np.testing.assert_allclose(o[:, h], want, atol=1e-13)
        assert np.max(np.abs(o_lit[:, h] - want)) > 1e-3


def test_decayed_rla_one_step_correction():
    """RLA, decayed residual, aR = 0, no clip, gamma = sqrt(beta):
    o_t = a_t S_{t-1} q_t + beta_t (v_t - a_t S_{t-1} k_t)(k_t . q_t) with the
    scalar-gated states of the textbook recurrence."""
    p = rand_problem(45)
    p["alpha_r"] = np.zeros_like(p["alpha_r"])
    p["gamma"] = np.sqrt(p["beta"])
    o, _, _ = fwd("rla", p, clip=math.inf, flags=oracle.DECAYED)
    for h in range(p["q"].shape[1]):
        Ss = tb.scalar_gated_states(p["k"][:, h], p["v"][:, h], p["alpha_s"][:, h], p["beta"][:, h])
        a = p["alpha_s"][:, h, None]
        base = a * np.einsum("tjk,tk->tj", Ss[:-1], p["q"][:, h])
        resid = p["v"][:, h] - a * np.einsum("tjk,tk->tj", Ss[:-1], p["k"][:, h])
        corr = p["beta"][:, h, None] * resid * np.sum(p["k"][:, h] * p["q"][:, h], -1)[:, None]
        np.testing.assert_allclose(o[:, h], base + corr, atol=1e-13)


# --- chunked formulation of the variants == recurrence ---------------------------

@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("flags", [oracle.TANH, oracle.UNGATED, oracle.DECAYED, ALL])
def test_chunked_variants_equal_recurrent(variant, flags):
    p = rand_problem(46, T=150, dk=16, dv=12)
    cu = np.array([0, 70, 150])
    rng = np.random.default_rng(47)
    S0 = rng.standard_normal((2, 2, 16, 12)) / 4
    R0 = rng.standard_normal((2, 2, 16, 12)) / 4
    args = (p["q"], p["k"], p["v"], p["alpha_s"], p["beta"], p["alpha_r"], p["gamma"])
    kw = dict(tanh=bool(flags & oracle.TANH), ungated=bool(flags & oracle.UNGATED),
              decayed=bool(flags & oracle.DECAYED))
    o, S, R = oracle.forward(variant, *args, clip=0.5, S0=S0, R0=R0, cu_seqlens=cu, flags=flags)
    for chunk in (3, 64):
        oc, Sc, Rc = chunked.forward(variant, *args, clip=0.5, S0=S0, R0=R0, cu_seqlens=cu,
                                     chunk=chunk, **kw)
        np.testing.assert_allclose(oc, o, atol=1e-12)
        np.testing.assert_allclose(Sc, S, atol=1e-12)
        np.testing.assert_allclose(Rc, R, atol=1e-12)


# --- backward == central finite differences -----------------------------------

@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("flags", [oracle.TANH, oracle.UNGATED, oracle.DECAYED, ALL])
def test_variant_backward_matches_finite_differences(variant, flags):
    T, H, dk, dv = 14, 2, 5, 4
    p = rand_problem(48 + flags, T=T, H=H, dk=dk, dv=dv)
    rng = np.random.default_rng(49)
    cu = np.array([0, 6, T])
    N = 2
    S0 = rng.standard_normal((N, H, dk, dv)) * 0.4
    R0 = rng.standard_normal((N, H, dk, dv)) * 0.4
    clip = 0.6
    gates = (p["alpha_s"], p["beta"], p["alpha_r"], p["gamma"])
    v, _ = oracle.nudge_margin(variant, p["q"], p["k"], p["v"], *gates, clip=clip, S0=S0, R0=R0,
                               cu_seqlens=cu, margin=1e-3, grid="f64", flags=flags)
    inputs = dict(q=p["q"], k=p["k"], v=v, alpha_s=p["alpha_s"], beta=p["beta"],
                  alpha_r=p["alpha_r"], gamma=p["gamma"], S0=S0, R0=R0)
    dO = rng.standard_normal((T, H, dv))
    dSf = rng.standard_normal((N, H, dk, dv))
    dRf = rng.standard_normal((N, H, dk, dv))

    def loss(inp):
        o, S, R = oracle.forward(variant, inp["q"], inp["k"], inp["v"], inp["alpha_s"], inp["beta"],
                                 inp["alpha_r"], inp["gamma"], clip=clip, S0=inp["S0"], R0=inp["R0"],
                                 cu_seqlens=cu, flags=flags)
        return np.sum(o * dO) + np.sum(S * dSf) + np.sum(R * dRf)

    g = oracle.backward(variant, inputs["q"], inputs["k"], inputs["v"], inputs["alpha_s"],
                        inputs["beta"], inputs["alpha_r"], inputs["gamma"], dO, clip=clip, S0=S0,
                        R0=R0, dS_final=dSf, dR_final=dRf, cu_seqlens=cu, flags=flags)
    names = dict(q="dq", k="dk", v="dv", alpha_s="dalpha_s", beta="dbeta", alpha_r="dalpha_r",
                 gamma="dgamma", S0="dS0", R0="dR0")
    h = 1e-6
    for key, gkey in names.items():
        base = inputs[key]
        fd = np.zeros(base.size)
        for idx in range(base.size):
            plus = dict(inputs)
            minus = dict(inputs)
            a = base.copy().ravel(); a[idx] += h
            b = base.copy().ravel(); b[idx] -= h
            plus[key] = a.reshape(base.shape)
            minus[key] = b.reshape(base.shape)
            fd[idx] = (loss(plus) - loss(minus)) / (2 * h)
        an = g[gkey].ravel()
        scale = max(1.0, np.max(np.abs(fd)))
        err = np.max(np.abs(an - fd)) / scale
        assert err < 1e-6, (gkey, err)


def test_planted_variant_mistakes_fail_the_pins():
    """Sanity of the pins: the boxed forward (no flags) differs from every
    variant on generic inputs, so a flag the oracle ignored would fail the
    pins above that compare against independent quantities."""
    p = rand_problem(50)
    base = fwd("rdn", p)[0]
    for f in (oracle.TANH, oracle.UNGATED, oracle.DECAYED):
        assert np.max(np.abs(fwd("rdn", p, flags=f)[0] - base)) > 1e-3
