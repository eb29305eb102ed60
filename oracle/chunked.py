"""Chunked fp64 formulation of the RLA / RDN forward (test infrastructure only).

The paper trains with chunk-wise parallel kernels (Sec. 2.1 cites the chunk
form of gated linear attention; Sec. 4.1 builds on such kernels) but does not
write the chunk form out.  This module states it, in fp64 numpy, so the tests
can pin it against the token recurrence of ``rla_oracle.c`` for several chunk
sizes.  The GPU kernels use the same algebra; they share no code with this.

Derivation (paper orientation S, R in R^{dv x dk}; one chunk of C tokens,
local index t = 1..C, start states S0, R0):
  g_t = sum_{j<=t} log aS_j, h_t = sum_{j<=t} log aR_j   (g_0 = h_0 = 0)
  Gram G = K K^T, scores P = Q K^T   (rows are tokens)
  The delta-rule update S_t = aS_t S_{t-1} + u_t k_t^T with
  u_t = b_t (v_t - aS_t S_{t-1} k_t) unrolls to
      S_t = e^{g_t} S0 + sum_{i<=t} e^{g_t - g_i} u_i k_i^T,
  so the u_t solve the unit lower-triangular system
      u_t + b_t sum_{i<t} e^{g_t-g_i} G_ti u_i = b_t (v_t - e^{g_t} S0 k_t),
  i.e. U = T diag(b) (V - diag(e^g) K S0^T) with T = (I + A)^{-1},
  A_ti = b_t e^{g_t-g_i} G_ti for i < t.
  Then, with exact exponents of differences only:
      p_t = S_{t-1} k_t   = e^{g_{t-1}} S0 k_t + sum_{i<t} e^{g_{t-1}-g_i} G_ti u_i
      b_t = aS_t S_{t-1} q_t = e^{g_t} S0 q_t  + sum_{i<t}  e^{g_t-g_i} P_ti u_i
      x_t = v_t - p_t,  r_t = clip(x_t)
  The R path is the same delta rule with (aR, gamma, r) in place of
  (aS, b, v); its readout is inclusive of the current token:
      c_t = R_t q_t = e^{h_t} R0 q_t + sum_{i<=t} e^{h_t-h_i} P_ti uR_i
      o_t = b_t + gamma_t c_t
  Chunk-end states: S_C = e^{g_C} S0 + sum_i e^{g_C-g_i} u_i k_i^T, same for R.
  RLA: T = I on both paths, u_t = b_t v_t and uR_t = gamma_t r_t.
Variants (keyword flags):
  tanh     r_t = c tanh(x_t / c) instead of the clip (log-cosh loss, App. B);
  ungated  o_t = S_{t-1} q_t + R_t q_t: the read-out of S uses the same
           decays as p_t, b'_t = e^{g_{t-1}} S0 q_t + sum_{i<t} e^{g_{t-1}-g_i} P_ti u_i,
           and o_t = b'_t + c_t;
  decayed  x_t = v_t - aS_t S_{t-1} k_t: the prediction uses the decays of b_t,
           p~_t = e^{g_t} S0 k_t + sum_{i<t} e^{g_t-g_i} G_ti u_i.
"""
from __future__ import annotations

import math

import numpy as np


def _clip(x, c):
    return x if (c is None or math.isinf(c)) else np.clip(x, -c, c)


def _tanh_resid(x, c):
    if c is None or math.isinf(c):
        return x
    if c == 0:
        return np.zeros_like(x)
    return c * np.tanh(x / c)


def _solve_unit_lower(A, rhs):
    """(I + A) X = rhs for strictly-lower A, by forward substitution."""
    C = A.shape[0]
    X = np.zeros_like(rhs)
    for t in range(C):
        X[t] = rhs[t] - A[t, :t] @ X[:t]
    return X


def chunk_step(variant, Q, K, V, aS, b, aR, g, clip, S0, R0, tanh=False, ungated=False,
               decayed=False):
    """One chunk.  Q, K: [C, dk]; V: [C, dv]; gates: [C]; S0, R0: [dv, dk]
    (paper orientation).  Returns (O [C, dv], S_C, R_C)."""
    C = Q.shape[0]
    gs = np.cumsum(np.log(aS))
    gr = np.cumsum(np.log(aR))
    gs_prev = np.concatenate([[0.0], gs[:-1]])
    G = K @ K.T
    P = Q @ K.T
    lower_strict = np.tril(np.ones((C, C)), -1)
    lower = np.tril(np.ones((C, C)), 0)
    dec_s = np.exp(np.minimum(gs[:, None] - gs[None, :], 0.0))          # e^{g_t - g_i}
    dec_s_prev = np.exp(np.minimum(gs_prev[:, None] - gs[None, :], 0.0))  # e^{g_{t-1} - g_i}
    dec_r = np.exp(np.minimum(gr[:, None] - gr[None, :], 0.0))
    KS = K @ S0.T            # rows (S0 k_t)^T
    QS = Q @ S0.T
    KR = K @ R0.T
    QR = Q @ R0.T
    if variant == "rdn":
        A = b[:, None] * dec_s * G * lower_strict
        U = _solve_unit_lower(A, b[:, None] * (V - np.exp(gs)[:, None] * KS))
    else:
        U = b[:, None] * V
    if decayed:
        p = np.exp(gs)[:, None] * KS + (dec_s * G * lower_strict) @ U
    else:
        p = np.exp(gs_prev)[:, None] * KS + (dec_s_prev * G * lower_strict) @ U
    if ungated:
        base = np.exp(gs_prev)[:, None] * QS + (dec_s_prev * P * lower_strict) @ U
    else:
        base = np.exp(gs)[:, None] * QS + (dec_s * P * lower_strict) @ U
    r = _tanh_resid(V - p, clip) if tanh else _clip(V - p, clip)
    if variant == "rdn":
        AR = g[:, None] * dec_r * G * lower_strict
        UR = _solve_unit_lower(AR, g[:, None] * (r - np.exp(gr)[:, None] * KR))
    else:
        UR = g[:, None] * r
    corr = np.exp(gr)[:, None] * QR + (dec_r * P * lower) @ UR
    O = base + (corr if ungated else g[:, None] * corr)
    S1 = math.exp(gs[-1]) * S0 + (np.exp(gs[-1] - gs)[:, None] * U).T @ K
    R1 = math.exp(gr[-1]) * R0 + (np.exp(gr[-1] - gr)[:, None] * UR).T @ K
    return O, S1, R1


def forward(variant, q, k, v, alpha_s, beta, alpha_r, gamma, clip=1.0, S0=None, R0=None,
            cu_seqlens=None, chunk=64, **flags):
    """Chunked forward with the same conventions as ``oracle.forward``:
    q, k [ntok, H, dk], v [ntok, H, dv], gates [ntok, H], states [N, H, dk, dv]
    (transposed storage).  Chunks restart at every sequence start; the last
    chunk of a sequence may be partial."""
    q, k, v = (np.asarray(a, dtype=np.float64) for a in (q, k, v))
    gates = [np.asarray(a, dtype=np.float64) for a in (alpha_s, beta, alpha_r, gamma)]
    ntok, H, dk = q.shape
    dv = v.shape[2]
    cu = np.array([0, ntok]) if cu_seqlens is None else np.asarray(cu_seqlens)
    N = len(cu) - 1
    o = np.zeros((ntok, H, dv))
    Sf = np.zeros((N, H, dk, dv))
    Rf = np.zeros((N, H, dk, dv))
    for n in range(N):
        for h in range(H):
            S = np.zeros((dv, dk)) if S0 is None else np.asarray(S0, np.float64)[n, h].T.copy()
            R = np.zeros((dv, dk)) if R0 is None else np.asarray(R0, np.float64)[n, h].T.copy()
            for c0 in range(int(cu[n]), int(cu[n + 1]), chunk):
                c1 = min(c0 + chunk, int(cu[n + 1]))
                sl = slice(c0, c1)
                O, S, R = chunk_step(variant, q[sl, h], k[sl, h], v[sl, h],
                                     *[gg[sl, h] for gg in gates], clip, S, R, **flags)
                o[sl, h] = O
            Sf[n, h] = S.T
            Rf[n, h] = R.T
    return o, Sf, Rf
