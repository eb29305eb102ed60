"""Textbook recurrences from the linear-attention literature, written
independently of the oracle, used to pin it through exact reductions.

States here use the paper's orientation (d_v x d_k) and plain numpy loops.
  gated delta rule (Gated DeltaNet, Table 1 row 5):
      S_t = a_t S_{t-1} (I - b_t k_t k_t^T) + b_t v_t k_t^T
  DeltaNet (Table 1 row 4; Sec. 2.2 delta rule): the above with a_t = 1
  scalar-gated linear attention (sGLA, App. D baseline):
      S_t = a_t S_{t-1} + b_t v_t k_t^T,  read-out o_t = S_t q_t
"""
import numpy as np


def gated_delta_states(k, v, a, b, S0=None):
    """All states S_0..S_T of the gated delta rule for one head.
    k [T, dk], v [T, dv], a, b [T] -> array [T+1, dv, dk]."""
    T, dk = k.shape
    dv = v.shape[1]
    S = np.zeros((dv, dk)) if S0 is None else np.array(S0, dtype=np.float64)
    out = [S.copy()]
    eye = np.eye(dk)
    for t in range(T):
        S = a[t] * S @ (eye - b[t] * np.outer(k[t], k[t])) + b[t] * np.outer(v[t], k[t])
        out.append(S.copy())
    return np.array(out)


def scalar_gated_states(k, v, a, b, S0=None):
    """All states S_0..S_T of scalar-gated linear attention for one head."""
    T, dk = k.shape
    dv = v.shape[1]
    S = np.zeros((dv, dk)) if S0 is None else np.array(S0, dtype=np.float64)
    out = [S.copy()]
    for t in range(T):
        S = a[t] * S + b[t] * np.outer(v[t], k[t])
        out.append(S.copy())
    return np.array(out)
