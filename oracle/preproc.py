"""fp64 oracle of the operator's input pre-processing (test infrastructure only).

The paper's attention block (Sec. 3.4, closing paragraph, and the caption of
its architecture figure) feeds the recurrences with
  q_t, k_t  after a SiLU activation and L2 normalisation over the head
            dimension, y / max(||y||, 1e-12) (the torch F.normalize form);
  alpha_t = exp(-a softplus(z^alpha_t + b)), the Mamba-2 re-parameterisation
            with learnable scalars a > 0, b (here one pair per head, shared by
            the decays of S and R; pass the same pre-activations for both to
            tie the decays as the paper does);
  beta_t = sigmoid(z^beta_t),  gamma_t = sigmoid(z^gamma_t).
Every step is computed in fp64 exactly as defined, with no rounding of the
normalised rows: whatever precision an implementation keeps them in is part
of the error measured against this oracle.
``forward`` applies these steps to raw inputs and calls the recurrent oracle;
``backward`` calls the recurrent oracle's adjoint on the transformed inputs
and applies the chain rule of each step, so it returns gradients with respect
to the raw q, k, the pre-activations and the per-head (a, b).
Only the test suite and the benchmark's CPU leg use this module.
"""
from __future__ import annotations

import numpy as np

import oracle


def _silu(x):
    return x / (1.0 + np.exp(-x))


def _sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def _softplus(x):
    return np.logaddexp(0.0, x)


NORM_EPS = 1e-12


def qk_transform(x):
    """q_hat = SiLU(x) / max(||SiLU(x)||, 1e-12) over the last axis (fp64)."""
    y = _silu(np.asarray(x, np.float64))
    return y / np.maximum(np.linalg.norm(y, axis=-1, keepdims=True), NORM_EPS)


def qk_transform_grad(x, dxhat):
    """Gradient w.r.t. x of <dxhat, qk_transform(x)>: through the norm
    (dy = (dxhat - xhat (xhat . dxhat)) / ||y||; below the floor the scale is
    the constant 1 / 1e-12) and SiLU' = s (1 + x (1 - s))."""
    x = np.asarray(x, np.float64)
    s = _sigmoid(x)
    y = x * s
    n = np.linalg.norm(y, axis=-1, keepdims=True)
    floor = n < NORM_EPS
    nn = np.maximum(n, NORM_EPS)
    yh = y / nn
    dy = np.where(floor, dxhat / NORM_EPS,
                  (dxhat - yh * np.sum(yh * dxhat, axis=-1, keepdims=True)) / nn)
    return dy * s * (1.0 + x * (1.0 - s))


def head_axis_param(p, shape):
    """Broadcast a per-head parameter [H] against gate arrays [..., H]."""
    return np.asarray(p, np.float64).reshape((1,) * (len(shape) - 1) + (-1,))


def decay_from_preact(z, a, b):
    """alpha = exp(-a softplus(z + b)), a and b per head (last axis of z)."""
    z = np.asarray(z, np.float64)
    A, Bb = head_axis_param(a, z.shape), head_axis_param(b, z.shape)
    return np.exp(-A * _softplus(z + Bb))


def transform_inputs(q, k, z_as, z_b, z_ar, z_g, decay_a, decay_b, qk_norm=True, gate_preact=True):
    """The operator's inputs (q, k, alpha_s, beta, alpha_r, gamma) from raw ones."""
    if qk_norm:
        q, k = qk_transform(q), qk_transform(k)
    if gate_preact:
        return (q, k, decay_from_preact(z_as, decay_a, decay_b), _sigmoid(np.asarray(z_b, np.float64)),
                decay_from_preact(z_ar, decay_a, decay_b), _sigmoid(np.asarray(z_g, np.float64)))
    return q, k, z_as, z_b, z_ar, z_g


def forward(variant, q, k, v, z_as, z_b, z_ar, z_g, decay_a=None, decay_b=None, clip=1.0,
            S0=None, R0=None, cu_seqlens=None, flags=0, qk_norm=True, gate_preact=True):
    """Forward from raw inputs: (o, S_final, R_final)."""
    qq, kk, aS, bb, aR, gg = transform_inputs(q, k, z_as, z_b, z_ar, z_g, decay_a, decay_b,
                                             qk_norm, gate_preact)
    return oracle.forward(variant, qq, kk, v, aS, bb, aR, gg, clip=clip, S0=S0, R0=R0,
                          cu_seqlens=cu_seqlens, flags=flags)


def backward(variant, q, k, v, z_as, z_b, z_ar, z_g, dO, decay_a=None, decay_b=None, clip=1.0,
             S0=None, R0=None, dS_final=None, dR_final=None, cu_seqlens=None, flags=0,
             qk_norm=True, gate_preact=True):
    """Gradients w.r.t. the raw inputs: dq, dk (raw q, k), dv, dalpha_s, dbeta,
    dalpha_r, dgamma (pre-activations), dS0, dR0 and, with gate_preact,
    ddecay_a, ddecay_b [H] (summed over every token of both decays)."""
    qq, kk, aS, bb, aR, gg = transform_inputs(q, k, z_as, z_b, z_ar, z_g, decay_a, decay_b,
                                             qk_norm, gate_preact)
    g = oracle.backward(variant, qq, kk, v, aS, bb, aR, gg, dO, clip=clip, S0=S0, R0=R0,
                        dS_final=dS_final, dR_final=dR_final, cu_seqlens=cu_seqlens, flags=flags)
    out = dict(g)
    if qk_norm:
        out["dq"] = qk_transform_grad(q, g["dq"])
        out["dk"] = qk_transform_grad(k, g["dk"])
    if gate_preact:
        zs, zr = np.asarray(z_as, np.float64), np.asarray(z_ar, np.float64)
        A, Bb = head_axis_param(decay_a, zs.shape), head_axis_param(decay_b, zs.shape)
        # d alpha / d z = alpha * (-a sigmoid(z + b)); d alpha / d a = alpha * (-softplus(z + b));
        # d alpha / d b = d alpha / d z
        dls = g["dalpha_s"] * aS   # gradient of log alpha_s
        dlr = g["dalpha_r"] * aR
        out["dalpha_s"] = dls * (-A * _sigmoid(zs + Bb))
        out["dalpha_r"] = dlr * (-A * _sigmoid(zr + Bb))
        red = tuple(range(zs.ndim - 1))
        out["ddecay_a"] = (np.sum(dls * -_softplus(zs + Bb), axis=red) +
                           np.sum(dlr * -_softplus(zr + Bb), axis=red))
        out["ddecay_b"] = np.sum(out["dalpha_s"], axis=red) + np.sum(out["dalpha_r"], axis=red)
        out["dbeta"] = g["dbeta"] * bb * (1.0 - bb)
        out["dgamma"] = g["dgamma"] * gg * (1.0 - gg)
    return out
