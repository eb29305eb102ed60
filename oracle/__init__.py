"""fp64 CPU oracle for the RLA / RDN sequence-mixing operators.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The GPU library never imports this
package and shares no code with it.

The arithmetic lives in ``rla_oracle.c`` (token-by-token recurrence of the
paper's Sec. 3.4 boxed formulations, plus the hand-derived adjoint).  This
module only marshals numpy arrays to it.  ``chunked`` holds a second, chunked
fp64 formulation used to pin the chunk algebra the GPU kernels rely on.

Array conventions (all numpy, any float dtype; computed in fp64):
  q, k : [ntok, H, dk] or [B, T, H, dk]      v : [ntok, H, dv] or [B, T, H, dv]
  alpha_s, beta, alpha_r, gamma : [ntok, H] or [B, T, H]
  S0, R0 : [N, H, dk, dv]  (transposed w.r.t. the paper's d_v x d_k states)
  cu_seqlens : [N+1] ints, or None for B equal-length sequences of length T.
  clip : float; math.inf means no clipping.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "rla_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

RLA = 0
RDN = 1
# variant bits (combine with `flags=`): the log-cosh residual r = c tanh(x / c)
# (App. B), the ungated output S_{t-1} q + R_t q (Sec. 4.3 ablation), the
# decayed residual x = v - aS S_{t-1} k (Table 1's gated prediction)
TANH = 2
UNGATED = 4
DECAYED = 8


def build(force: bool = True) -> str:
    """Compile rla_oracle.c into liboracle.so with gcc (fp64, OpenMP)."""
    if not force and os.path.exists(_LIB_PATH) and os.path.getmtime(_LIB_PATH) >= os.path.getmtime(_SRC):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fopenmp", "-fno-fast-math",
           "-ffp-contract=off", _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build(force=False)
            lib = ctypes.CDLL(_LIB_PATH)
            i64, dbl, pd, pi64 = ctypes.c_int64, ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p
            lib.orc_forward.argtypes = [ctypes.c_int, i64, pi64, i64, i64, i64, i64,
                                        pd, pd, pd, pd, pd, pd, pd, dbl, pd, pd, pd, pd, pd]
            lib.orc_forward.restype = ctypes.c_int
            lib.orc_backward.argtypes = [ctypes.c_int, i64, pi64, i64, i64, i64, i64,
                                         pd, pd, pd, pd, pd, pd, pd, dbl, pd, pd, pd, pd, pd,
                                         pd, pd, pd, pd, pd, pd, pd, pd, pd]
            lib.orc_backward.restype = ctypes.c_int
            lib.orc_nudge_margin.argtypes = [ctypes.c_int, i64, pi64, i64, i64, i64, i64,
                                             pd, pd, pd, pd, pd, pd, pd, dbl, pd, pd, dbl,
                                             ctypes.c_int]
            lib.orc_nudge_margin.restype = ctypes.c_int64
            lib.orc_threads.argtypes = []
            lib.orc_threads.restype = ctypes.c_int
            _lib = lib
    return _lib


def threads() -> int:
    """OpenMP threads the oracle runs with."""
    return int(_load().orc_threads())


def _variant(name, flags: int = 0) -> int:
    if flags & ~(TANH | UNGATED | DECAYED):
        raise ValueError("unknown variant flags")
    if name in ("rdn", RDN):
        return RDN | flags
    if name in ("rla", RLA):
        return RLA | flags
    raise ValueError("variant must be 'rla' or 'rdn'")


class _Prob:
    """Flattened view of one call's arrays (fp64, C-contiguous)."""

    def __init__(self, q, k, v, gates, cu_seqlens, S0, R0):
        q = np.asarray(q)
        self.batched = q.ndim == 4
        if self.batched:
            B, T = q.shape[0], q.shape[1]
            self.out_lead = (B, T)
            if cu_seqlens is not None:
                raise ValueError("cu_seqlens requires [ntok, H, d] inputs")
            cu = np.arange(B + 1, dtype=np.int64) * T
        else:
            self.out_lead = (q.shape[0],)
            cu = (np.array([0, q.shape[0]], dtype=np.int64) if cu_seqlens is None
                  else np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int64)))
        self.cu = cu
        self.N = len(cu) - 1
        f = lambda a: np.ascontiguousarray(np.asarray(a, dtype=np.float64))
        self.q = f(q).reshape(-1, q.shape[-2], q.shape[-1])
        self.k = f(k).reshape(self.q.shape[0], q.shape[-2], -1)
        self.v = f(v).reshape(self.q.shape[0], q.shape[-2], -1)
        self.ntok, self.H, self.dk = self.q.shape
        self.dv = self.v.shape[2]
        self.gates = [f(g).reshape(self.ntok, self.H) for g in gates]
        self.S0 = None if S0 is None else f(S0).reshape(self.N, self.H, self.dk, self.dv)
        self.R0 = None if R0 is None else f(R0).reshape(self.N, self.H, self.dk, self.dv)

    def reshape_tok(self, a):
        return a.reshape(self.out_lead + a.shape[1:])


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _clip_arg(clip: float) -> float:
    if clip is None or math.isinf(clip):
        return -1.0
    if clip < 0 or math.isnan(clip):
        raise ValueError("clip must be >= 0 or inf")
    return float(clip)


def forward(variant, q, k, v, alpha_s, beta, alpha_r, gamma, clip=1.0,
            S0=None, R0=None, cu_seqlens=None, flags=0):
    """Token-recurrent fp64 forward.  Returns (o, S_final, R_final).
    flags: any of TANH, UNGATED, DECAYED."""
    lib = _load()
    p = _Prob(q, k, v, (alpha_s, beta, alpha_r, gamma), cu_seqlens, S0, R0)
    o = np.zeros((p.ntok, p.H, p.dv))
    Sf = np.zeros((p.N, p.H, p.dk, p.dv))
    Rf = np.zeros((p.N, p.H, p.dk, p.dv))
    rc = lib.orc_forward(_variant(variant, flags), p.N, _ptr(p.cu), p.ntok, p.H, p.dk, p.dv,
                         _ptr(p.q), _ptr(p.k), _ptr(p.v), *[_ptr(g) for g in p.gates],
                         _clip_arg(clip), _ptr(p.S0), _ptr(p.R0), _ptr(o), _ptr(Sf), _ptr(Rf))
    if rc != 0:
        raise MemoryError("oracle forward failed")
    return p.reshape_tok(o), Sf, Rf


def backward(variant, q, k, v, alpha_s, beta, alpha_r, gamma, dO, clip=1.0,
             S0=None, R0=None, dS_final=None, dR_final=None, cu_seqlens=None, flags=0):
    """Adjoint of ``forward`` for L = <dO,o> + <dS_final,S_T> + <dR_final,R_T>.

    Returns a dict with dq, dk, dv, dalpha_s, dbeta, dalpha_r, dgamma, dS0, dR0.
    """
    lib = _load()
    p = _Prob(q, k, v, (alpha_s, beta, alpha_r, gamma), cu_seqlens, S0, R0)
    f = lambda a: None if a is None else np.ascontiguousarray(np.asarray(a, dtype=np.float64))
    dO_ = f(dO).reshape(p.ntok, p.H, p.dv)
    dSf = None if dS_final is None else f(dS_final).reshape(p.N, p.H, p.dk, p.dv)
    dRf = None if dR_final is None else f(dR_final).reshape(p.N, p.H, p.dk, p.dv)
    out = dict(dq=np.zeros((p.ntok, p.H, p.dk)), dk=np.zeros((p.ntok, p.H, p.dk)),
               dv=np.zeros((p.ntok, p.H, p.dv)), dalpha_s=np.zeros((p.ntok, p.H)),
               dbeta=np.zeros((p.ntok, p.H)), dalpha_r=np.zeros((p.ntok, p.H)),
               dgamma=np.zeros((p.ntok, p.H)), dS0=np.zeros((p.N, p.H, p.dk, p.dv)),
               dR0=np.zeros((p.N, p.H, p.dk, p.dv)))
    rc = lib.orc_backward(_variant(variant, flags), p.N, _ptr(p.cu), p.ntok, p.H, p.dk, p.dv,
                          _ptr(p.q), _ptr(p.k), _ptr(p.v), *[_ptr(g) for g in p.gates],
                          _clip_arg(clip), _ptr(p.S0), _ptr(p.R0), _ptr(dO_), _ptr(dSf),
                          _ptr(dRf), _ptr(out["dq"]), _ptr(out["dk"]), _ptr(out["dv"]),
                          _ptr(out["dalpha_s"]), _ptr(out["dbeta"]), _ptr(out["dalpha_r"]),
                          _ptr(out["dgamma"]), _ptr(out["dS0"]), _ptr(out["dR0"]))
    if rc != 0:
        raise MemoryError("oracle backward failed")
    for key in ("dq", "dk", "dv", "dalpha_s", "dbeta", "dalpha_r", "dgamma"):
        out[key] = p.reshape_tok(out[key])
    return out


def nudge_margin(variant, q, k, v, alpha_s, beta, alpha_r, gamma, clip=1.0, S0=None, R0=None,
                 cu_seqlens=None, margin=1e-2, grid="bf16", flags=0):
    """Returns (v_moved, count): v moved so that every pre-clip residual stays
    at least ``margin`` away from the clip kink |x| = c, with moved values kept
    on the input dtype's grid (grid in {'bf16', 'f32', 'f64'}).  Gradient
    parity compares clip masks taken in two precisions; the margin keeps those
    masks equal.  Only v changes, and v_t does not influence S_{t-1}."""
    lib = _load()
    p = _Prob(q, k, v, (alpha_s, beta, alpha_r, gamma), cu_seqlens, S0, R0)
    vv = p.v.copy()
    bits = {"bf16": 16, "f32": 0, "f64": 64}[grid]
    moved = lib.orc_nudge_margin(_variant(variant, flags), p.N, _ptr(p.cu), p.ntok, p.H, p.dk, p.dv,
                                 _ptr(p.q), _ptr(p.k), _ptr(vv), *[_ptr(g) for g in p.gates],
                                 _clip_arg(clip), _ptr(p.S0), _ptr(p.R0), float(margin), bits)
    if moved < 0:
        raise MemoryError("oracle nudge failed")
    return p.reshape_tok(vv), int(moved)
