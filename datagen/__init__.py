"""Seeded synthetic inputs for the RLA / RDN sequence-mixing operators.

Shared by the tests, the benchmark and the smoke check.  This module draws
random numbers and lays them out; it holds none of the operators' arithmetic.

Shapes and distributions follow the paper's language-model setting (App. C,
Table 6: 16 heads of dimension 128 per layer; the clip bound c = 1 of Sec. 4.1)
and the synthetic recipe used throughout this repository:
  q, k ~ N(0, 1), then L2-normalised over the head dimension (Sec. 3.3 applies
       L2 normalisation to queries and keys), then rounded to the input dtype;
  v ~ N(0, 1), rounded to the input dtype;
  decay gates alpha_s, alpha_r = sigmoid(N(mu, 1)) with mu = 2 (RDN) or 3 (RLA);
  write strengths beta, gamma = sigmoid(N(0, 1));
  upstream gradient dO ~ N(0, 1) (input dtype).
Gates are always fp32 values.

Every sequence has its own generator, seeded by (seed, sequence index), so any
subset of sequences can be regenerated on its own.  Within a sequence the draw
order is q, k, v, alpha_s, beta, alpha_r, gamma, dO, each a full [L, H, d] or
[L, H] tensor in C order.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    op: str                 # "rla_fwd", "rdn_fwd", "rdn_fwdbwd"
    dtype: str              # "f32" or "bf16" (q, k, v, o, dq, dk, dv)
    H: int
    dk: int
    dv: int
    seqlens: tuple          # per-sequence lengths
    varlen: bool            # packed with cu_seqlens (B = 1) vs dense [B, T, ...]
    decay_mu: float = 2.0
    clip: float = 1.0

    @property
    def B(self) -> int:
        return 1 if self.varlen else len(self.seqlens)

    @property
    def T(self) -> int:
        return sum(self.seqlens) if self.varlen else self.seqlens[0]

    @property
    def ntok(self) -> int:
        return sum(self.seqlens)

    @property
    def variant(self) -> str:
        return "rla" if self.op.startswith("rla") else "rdn"

    def cu_seqlens(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.seqlens)]).astype(np.int64)

    def describe(self) -> dict:
        d = {"workload": self.name, "op": self.op, "dtype": self.dtype, "H": self.H,
             "d_k": self.dk, "d_v": self.dv, "tokens": self.ntok, "clip": self.clip}
        if self.varlen:
            d.update(num_seqs=len(self.seqlens), min_len=min(self.seqlens), max_len=max(self.seqlens))
        else:
            d.update(B=self.B, T=self.T)
        return d


def varlen_lengths(seed: int, total: int, lo: int, hi: int) -> tuple:
    """Lengths drawn uniformly from [lo, hi] until they reach `total` tokens;
    the last one is cut so the sum is exactly `total`."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 1 << 30])))
    out: List[int] = []
    acc = 0
    while acc < total:
        L = int(rng.integers(lo, hi + 1))
        L = min(L, total - acc)
        out.append(L)
        acc += L
    return tuple(out)


def dense(name, op, dtype, B, T, H, d, decay_mu=2.0, clip=1.0) -> Workload:
    return Workload(name, op, dtype, H, d, d, (T,) * B, False, decay_mu, clip)


#: The workloads: a small fp32 case, three forward workloads at language-model
#: shapes (dense RLA, dense RDN, packed variable-length RDN) and the
#: forward+backward training-step workload.
_ALL = [
    dense("rdn_fwd_f32_B1_H2_T256_d64", "rdn_fwd", "f32", 1, 256, 2, 64),
    dense("rla_fwd_bf16_B4_H16_T2048_d128", "rla_fwd", "bf16", 4, 2048, 16, 128, decay_mu=3.0),
    dense("rdn_fwd_bf16_B8_H16_T4096_d128", "rdn_fwd", "bf16", 8, 4096, 16, 128),
    Workload("rdn_fwd_varlen_bf16_262144tok_H16_d128", "rdn_fwd", "bf16", 16, 128, 128,
             varlen_lengths(4, 262144, 512, 32768), True),
    dense("rdn_fwdbwd_bf16_B4_H16_T4096_d128", "rdn_fwdbwd", "bf16", 4, 4096, 16, 128),
]
WORKLOADS: Dict[str, Workload] = {wl.name: wl for wl in _ALL}
#: seed of each workload's inputs
SEEDS: Dict[str, int] = {wl.name: i + 1 for i, wl in enumerate(_ALL)}
#: the training-step workload (forward + backward) used by the benchmark
TRAINING = "rdn_fwdbwd_bf16_B4_H16_T4096_d128"


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even onto the bf16 grid, returned as float32."""
    a = np.ascontiguousarray(x, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def _sigmoid(x: np.ndarray) -> np.ndarray:
    return (1.0 / (1.0 + np.exp(-x.astype(np.float64)))).astype(np.float32)


def _l2norm(x: np.ndarray) -> np.ndarray:
    n = np.sqrt(np.sum(x.astype(np.float64) ** 2, axis=-1, keepdims=True))
    return (x / np.maximum(n, 1e-30)).astype(np.float32)


def make_sequence(wl: Workload, seed: int, n: int, grads: bool = False) -> Dict[str, np.ndarray]:
    """Inputs of sequence n: arrays [L, H, d] / [L, H], float32 values on the
    grid of the workload's dtype."""
    L = wl.seqlens[n]
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, n])))
    H, dk, dv = wl.H, wl.dk, wl.dv
    rnd = (lambda a: round_to_bf16(a)) if wl.dtype == "bf16" else (lambda a: a.astype(np.float32))
    out = {}
    out["q"] = rnd(_l2norm(rng.standard_normal((L, H, dk), dtype=np.float32)))
    out["k"] = rnd(_l2norm(rng.standard_normal((L, H, dk), dtype=np.float32)))
    out["v"] = rnd(rng.standard_normal((L, H, dv), dtype=np.float32))
    out["alpha_s"] = _sigmoid(rng.standard_normal((L, H), dtype=np.float32) + wl.decay_mu)
    out["beta"] = _sigmoid(rng.standard_normal((L, H), dtype=np.float32))
    out["alpha_r"] = _sigmoid(rng.standard_normal((L, H), dtype=np.float32) + wl.decay_mu)
    out["gamma"] = _sigmoid(rng.standard_normal((L, H), dtype=np.float32))
    if grads:
        out["dO"] = rnd(rng.standard_normal((L, H, dv), dtype=np.float32))
    return out


def make_inputs(wl: Workload, seed: int, seqs: Optional[Sequence[int]] = None,
                grads: Optional[bool] = None) -> Dict[str, np.ndarray]:
    """Inputs for the sequences `seqs` (all by default), packed along tokens:
    arrays [ntok, H, d] / [ntok, H] plus 'cu_seqlens' [len(seqs)+1] (int64)."""
    if grads is None:
        grads = wl.op.endswith("fwdbwd")
    seqs = list(range(len(wl.seqlens))) if seqs is None else list(seqs)
    parts = [make_sequence(wl, seed, n, grads) for n in seqs]
    out = {key: np.concatenate([p[key] for p in parts], axis=0) for key in parts[0]}
    out["cu_seqlens"] = np.concatenate([[0], np.cumsum([wl.seqlens[n] for n in seqs])]).astype(np.int64)
    return out


def random_states(seed: int, N: int, H: int, dk: int, dv: int, scale: Optional[float] = None):
    """Initial states S0, R0 ~ N(0, 1/dk), fp32, [N, H, dk, dv]."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 1 << 31])))
    s = (1.0 / np.sqrt(dk)) if scale is None else scale
    S0 = (rng.standard_normal((N, H, dk, dv)) * s).astype(np.float32)
    R0 = (rng.standard_normal((N, H, dk, dv)) * s).astype(np.float32)
    return S0, R0


def small(op: str, dtype: str, seqlens: Sequence[int], H: int, d: int, decay_mu: float = 2.0,
          clip: float = 1.0, varlen: bool = True, dv: Optional[int] = None) -> Workload:
    """A reduced workload with the same distributions (for tests)."""
    return Workload("small", op, dtype, H, d, d if dv is None else dv, tuple(seqlens), varlen,
                    decay_mu, clip)
