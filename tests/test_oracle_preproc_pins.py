"""Pins of the oracle's input pre-processing (SiLU + L2 normalisation of q, k;
Mamba-2 decay re-parameterisation; sigmoid write strengths) to closed forms
and to central finite differences of its own forward.  CPU only."""
import math

import numpy as np
import pytest

import oracle
from oracle import preproc


def test_qk_transform_closed_forms():
    """Equal inputs give equal unit entries; SiLU(0) = 0 drops a coordinate;
    a large negative input is switched off by SiLU; sigma(1) = 0.7310585786...
    fixes the SiLU slope at one point."""
    np.testing.assert_allclose(preproc.qk_transform(np.ones((1, 4))), np.full((1, 4), 0.5), atol=1e-15)
    np.testing.assert_allclose(preproc.qk_transform(np.array([[1.0, 0.0, 0.0]])), [[1.0, 0.0, 0.0]],
                               atol=1e-15)
    np.testing.assert_allclose(preproc.qk_transform(np.array([[2.0, -100.0]])), [[1.0, 0.0]], atol=1e-30)
    # [1, x]: SiLU(1) = sigma(1) = 0.7310585786300049; choose x with SiLU(x) = -SiLU(1)... use ratios
    y = preproc.qk_transform(np.array([[1.0, 3.0]]))
    s1, s3 = 0.7310585786300049, 3.0 * 0.9525741268224334   # 1 sigma(1), 3 sigma(3)
    np.testing.assert_allclose(y, [[s1 / math.hypot(s1, s3), s3 / math.hypot(s1, s3)]], atol=1e-15)
    # an all-zero row stays zero (the 1e-12 floor of x / max(||x||, eps))
    np.testing.assert_array_equal(preproc.qk_transform(np.zeros((1, 3))), np.zeros((1, 3)))


def test_decay_reparameterisation_closed_form():
    """With a = 1 and b = 0, exp(-softplus(z)) = 1 / (1 + e^z) = sigmoid(-z):
    the pre-processed forward equals the plain one given those decays."""
    rng = np.random.default_rng(60)
    T, H, d = 20, 2, 6
    q = rng.standard_normal((T, H, d))
    k = rng.standard_normal((T, H, d))
    v = rng.standard_normal((T, H, d))
    za, zr = rng.standard_normal((T, H)) - 2.0, rng.standard_normal((T, H)) - 2.0
    zb, zg = rng.standard_normal((T, H)), rng.standard_normal((T, H))
    ones, zeros = np.ones(H), np.zeros(H)
    o1, S1, R1 = preproc.forward("rdn", q, k, v, za, zb, zr, zg, ones, zeros)
    qn = preproc.qk_transform(q)
    kn = preproc.qk_transform(k)
    o2, S2, R2 = oracle.forward("rdn", qn, kn, v, 1.0 / (1.0 + np.exp(za)), 1.0 / (1.0 + np.exp(-zb)),
                                1.0 / (1.0 + np.exp(zr)), 1.0 / (1.0 + np.exp(-zg)))
    for a, b in ((o1, o2), (S1, S2), (R1, R2)):
        np.testing.assert_allclose(a, b, atol=1e-13)


@pytest.mark.parametrize("variant", ["rdn", "rla"])
@pytest.mark.parametrize("qk_norm,gate_preact", [(True, True), (True, False), (False, True)])
def test_preproc_backward_matches_finite_differences(variant, qk_norm, gate_preact):
    T, H, dk, dv = 12, 2, 5, 4
    rng = np.random.default_rng(61)
    cu = np.array([0, 5, T])
    inputs = dict(q=rng.standard_normal((T, H, dk)), k=rng.standard_normal((T, H, dk)),
                  v=rng.standard_normal((T, H, dv)),
                  z_as=rng.standard_normal((T, H)) - 1.0, z_b=rng.standard_normal((T, H)),
                  z_ar=rng.standard_normal((T, H)) - 1.0, z_g=rng.standard_normal((T, H)),
                  decay_a=np.abs(rng.standard_normal(H)) + 0.5, decay_b=rng.standard_normal(H))
    if not gate_preact:   # plain gate values in (0, 1)
        for key in ("z_as", "z_b", "z_ar", "z_g"):
            inputs[key] = 1.0 / (1.0 + np.exp(-inputs[key]))
    S0 = rng.standard_normal((2, H, dk, dv)) * 0.4
    R0 = rng.standard_normal((2, H, dk, dv)) * 0.4
    dO = rng.standard_normal((T, H, dv))
    clip = math.inf   # smooth (the clip's kink is pinned elsewhere)
    kw = dict(clip=clip, S0=S0, R0=R0, cu_seqlens=cu, qk_norm=qk_norm, gate_preact=gate_preact,
              flags=oracle.TANH)

    def loss(inp):
        o, S, R = preproc.forward(variant, inp["q"], inp["k"], inp["v"], inp["z_as"], inp["z_b"],
                                  inp["z_ar"], inp["z_g"], inp["decay_a"], inp["decay_b"], **kw)
        return np.sum(o * dO)

    g = preproc.backward(variant, inputs["q"], inputs["k"], inputs["v"], inputs["z_as"], inputs["z_b"],
                         inputs["z_ar"], inputs["z_g"], dO, inputs["decay_a"], inputs["decay_b"], **kw)
    names = dict(q="dq", k="dk", v="dv", z_as="dalpha_s", z_b="dbeta", z_ar="dalpha_r", z_g="dgamma")
    if gate_preact:
        names.update(decay_a="ddecay_a", decay_b="ddecay_b")
    h = 1e-6
    for key, gkey in names.items():
        base = inputs[key]
        fd = np.zeros(base.size)
        for idx in range(base.size):
            plus, minus = dict(inputs), dict(inputs)
            a = base.copy().ravel(); a[idx] += h
            b = base.copy().ravel(); b[idx] -= h
            plus[key] = a.reshape(base.shape)
            minus[key] = b.reshape(base.shape)
            fd[idx] = (loss(plus) - loss(minus)) / (2 * h)
        an = np.asarray(g[gkey]).ravel()
        err = np.max(np.abs(an - fd)) / max(1.0, np.max(np.abs(fd)))
        assert err < 1e-6, (gkey, err)
