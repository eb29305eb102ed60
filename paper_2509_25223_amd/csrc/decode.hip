// Recurrent (decoding) step of RLA / RDN: the token recurrence of Sec. 3.4
// run directly, 256-thread workgroups over (sequence, head, value block),
// advancing S and R by T tokens (T is small in decoding; the chunked path
// serves long T).
//
// The states (d_k x d_v fp32, stored transposed like the ABI: element (i, j)
// is the paper's S[j][i]) are read once into registers, updated token by
// token and written once, so a step moves 2 x 2 x d_k x d_v x 4 bytes per
// (sequence, head) plus the token vectors: it is bound by HBM bandwidth.
//
// Value columns evolve independently (every column sum runs over the key
// index), so each (sequence, head) is split over DV / BV workgroups of BV
// columns.  The states are touched once per step, so they are loaded and
// stored non-temporally (measured 8% faster than cached accesses).
// Thread layout: thread (rg, cg) owns columns 4cg..4cg+3 of the block on rows
// i = ii * RG + rg (ii < RPT), as float4 registers, so the lanes of a wave
// load adjacent row segments (coalesced 16-byte accesses).
//
// Per token, with k = k_t, q = q_t and four column sums over the key index
//   Sk = S^T k, Sq = S^T q, Rk = R^T k, Rq = R^T q     (S, R: the old states)
//   x = v - Sk,  r = clip(x)                            (Sec. 3.1, 3.3)
//   RDN: a = v - aS Sk,  b = r - aR Rk                  RLA: a = v,  b = r
//   S <- aS S + beta k a^T,   R <- aR R + gamma k b^T
//   o = aS Sq + gamma (aR Rq + gamma (k.q) b)           (= aS S_{t-1} q + gamma R_t q)
// which is the boxed update S_t = aS S_{t-1}(I - beta k k^T) + beta v k^T
// (RDN) or aS S_{t-1} + beta v k^T (RLA), and likewise for R with (aR, gamma,
// r), written in the transposed storage.  Variants: x = v - aS Sk (decayed
// residual), r = c tanh(x / c) (log-cosh residual), o = Sq + R_t q (ungated).
// Pre-processing: q, k rows through SiLU and x / max(||x||, 1e-12); gates from
// pre-activations (aS, aR = exp(-a_h softplus(z + b_h)), beta, gamma = sigmoid).
#include "kernels.hpp"

namespace rla {

namespace {

// value columns per workgroup (32, 64 and 128 measured within 1% of each
// other at 256 sequences x 16 heads; 64 was the fastest)
constexpr int kDecodeBV = 64;

template <typename IN, typename OT, int DK, int BV, bool RDN>
__global__ __launch_bounds__(kThreads) void decode_kernel(OpParams p) {
  constexpr int CG = BV / 4;           // float4 column groups
  constexpr int RG = kThreads / CG;    // row groups
  constexpr int RPT = DK / RG;         // rows per thread
  constexpr int GPW = 64 / CG;         // row groups per wave
  static_assert(RPT * RG == DK && GPW * CG == 64, "decode thread layout");
  __shared__ float sq[2][DK], sk[2][DK], sv[2][BV], sg[2][4];
  __shared__ float red[kWaves][4][BV];   // per-wave partial Sk, Sq, Rk, Rq
  __shared__ float coef[2][BV];          // a, b
  __shared__ float skq;

  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int cg = tid % CG, rg = tid / CG;
  const int H = p.H, DV = p.DV, T = (int)p.st.dense_T;
  const int nvb = DV / BV;
  const int pair = blockIdx.x / nvb, j0 = (blockIdx.x % nvb) * BV;
  const int n = pair / H, h = pair % H;
  const int64_t soff = (int64_t)pair * DK * DV + j0 + 4 * cg;
  const float clip = p.clip;

  floatx4 S[RPT], R[RPT];
#pragma unroll
  for (int ii = 0; ii < RPT; ++ii) {
    const int64_t o = soff + (int64_t)(ii * RG + rg) * DV;
    S[ii] = p.S0 ? __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(p.S0 + o)) : zero4();
    R[ii] = p.R0 ? __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(p.R0 + o)) : zero4();
  }

  const IN* qg = reinterpret_cast<const IN*>(p.q);
  const IN* kg = reinterpret_cast<const IN*>(p.k);
  const IN* vg = reinterpret_cast<const IN*>(p.v);
  OT* og = reinterpret_cast<OT*>(p.o);

  for (int t = 0; t < T; ++t) {
    const int b = t & 1;
    const int64_t tok = (int64_t)n * T + t;
    // ---- stage the token's vectors and gates (double-buffered) ----
    if (tid < DK) {
      sq[b][tid] = to_f<IN>(qg[(tok * H + h) * DK + tid]);
      sk[b][tid] = to_f<IN>(kg[(tok * H + h) * DK + tid]);
    }
    if (tid < BV) sv[b][tid] = to_f<IN>(vg[(tok * H + h) * DV + j0 + tid]);
    if (tid < 4) {
      const float* gp = tid == 0 ? p.alpha_s : tid == 1 ? p.beta : tid == 2 ? p.alpha_r : p.gamma;
      float gv = gp[tok * H + h];
      if (p.vflags & kVarGatePreact)
        gv = (tid & 1) ? sigmoid_f(gv) : __expf(-p.decay_param[h] * softplus_f(gv + p.decay_param[H + h]));
      sg[b][tid] = gv;
    }
    __syncthreads();
    if (p.vflags & kVarQkNorm) {   // wave 0: q, wave 1: k
      if (w < 2) {
        float* x = w == 0 ? sq[b] : sk[b];
        float y[DK / 64], ss = 0.f;
#pragma unroll
        for (int e = 0; e < DK / 64; ++e) {
          const float v = x[lane + 64 * e];
          y[e] = v / (1.f + __expf(-v));
          ss = __builtin_fmaf(y[e], y[e], ss);
        }
#pragma unroll
        for (int m = 1; m < 64; m <<= 1) ss += __shfl_xor(ss, m);
        const float inv = 1.f / fmaxf(sqrtf(ss), 1e-12f);
#pragma unroll
        for (int e = 0; e < DK / 64; ++e) x[lane + 64 * e] = y[e] * inv;
      }
      __syncthreads();
    }

    // ---- column sums over this thread's rows, then over the wave's row groups ----
    floatx4 pSk = zero4(), pSq = zero4(), pRk = zero4(), pRq = zero4();
#pragma unroll
    for (int ii = 0; ii < RPT; ++ii) {
      const int i = ii * RG + rg;
      const float ki = sk[b][i], qi = sq[b][i];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        pSk[c] = __builtin_fmaf(ki, S[ii][c], pSk[c]);
        pSq[c] = __builtin_fmaf(qi, S[ii][c], pSq[c]);
        pRk[c] = __builtin_fmaf(ki, R[ii][c], pRk[c]);
        pRq[c] = __builtin_fmaf(qi, R[ii][c], pRq[c]);
      }
    }
#pragma unroll
    for (int m = CG; m < 64; m <<= 1)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        pSk[c] += __shfl_xor(pSk[c], m);
        pSq[c] += __shfl_xor(pSq[c], m);
        pRk[c] += __shfl_xor(pRk[c], m);
        pRq[c] += __shfl_xor(pRq[c], m);
      }
    if (lane < CG) {
      *reinterpret_cast<floatx4*>(&red[w][0][4 * cg]) = pSk;
      *reinterpret_cast<floatx4*>(&red[w][1][4 * cg]) = pSq;
      *reinterpret_cast<floatx4*>(&red[w][2][4 * cg]) = pRk;
      *reinterpret_cast<floatx4*>(&red[w][3][4 * cg]) = pRq;
    }
    if (w == kWaves - 1) {   // k . q over the key index
      float kq = 0.f;
#pragma unroll
      for (int i = lane; i < DK; i += 64) kq = __builtin_fmaf(sk[b][i], sq[b][i], kq);
#pragma unroll
      for (int m = 1; m < 64; m <<= 1) kq += __shfl_xor(kq, m);
      if (lane == 0) skq = kq;
    }
    __syncthreads();

    // ---- per value column: residual, clip, update coefficients, output ----
    if (tid < BV) {
      const int j = tid;
      float Sk = 0.f, Sq = 0.f, Rk = 0.f, Rq = 0.f;
#pragma unroll
      for (int ww = 0; ww < kWaves; ++ww) {
        Sk += red[ww][0][j];
        Sq += red[ww][1][j];
        Rk += red[ww][2][j];
        Rq += red[ww][3][j];
      }
      const float aS = sg[b][0], aR = sg[b][2], gm = sg[b][3];
      const float vj = sv[b][j];
      const float x = (p.vflags & kVarDecayed) ? __builtin_fmaf(-aS, Sk, vj) : vj - Sk;
      const float r = (p.vflags & kVarTanh) ? resid_tanh(x, clip)
                                            : (clip < 0.f ? x : fminf(fmaxf(x, -clip), clip));
      const float ca = RDN ? __builtin_fmaf(-aS, Sk, vj) : vj;
      const float cb = RDN ? __builtin_fmaf(-aR, Rk, r) : r;
      coef[0][j] = ca;
      coef[1][j] = cb;
      const float rq = __builtin_fmaf(gm * skq, cb, aR * Rq);   // R_t q
      const bool ung = (p.vflags & kVarUngated) != 0;
      const float oj = __builtin_fmaf(ung ? 1.f : gm, rq, ung ? Sq : aS * Sq);
      const int64_t oo = (tok * H + h) * DV + j0 + j;
      if constexpr (sizeof(OT) == 4) og[oo] = oj;
      else og[oo] = f2bf(oj);
    }
    __syncthreads();

    // ---- state updates ----
    {
      const float aS = sg[b][0], bt = sg[b][1], aR = sg[b][2], gm = sg[b][3];
      const floatx4 ca = *reinterpret_cast<const floatx4*>(&coef[0][4 * cg]);
      const floatx4 cb = *reinterpret_cast<const floatx4*>(&coef[1][4 * cg]);
#pragma unroll
      for (int ii = 0; ii < RPT; ++ii) {
        const float ki = sk[b][ii * RG + rg];
        const float bk = bt * ki, gk = gm * ki;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          S[ii][c] = __builtin_fmaf(bk, ca[c], aS * S[ii][c]);
          R[ii][c] = __builtin_fmaf(gk, cb[c], aR * R[ii][c]);
        }
      }
    }
  }

#pragma unroll
  for (int ii = 0; ii < RPT; ++ii) {
    const int64_t o = soff + (int64_t)(ii * RG + rg) * DV;
    __builtin_nontemporal_store(S[ii], reinterpret_cast<floatx4*>(p.S_fin + o));
    __builtin_nontemporal_store(R[ii], reinterpret_cast<floatx4*>(p.R_fin + o));
  }
}

template <typename IN, typename OT, int DK>
hipError_t launch_decode_t(const OpParams& p, hipStream_t stream) {
  constexpr int BV = kDecodeBV;   // d_v in {64, 128} is a multiple of BV
  const int64_t grid = (int64_t)p.st.nseq * p.H * (p.DV / BV);
  if (grid == 0) return hipSuccess;
  if (p.rdn)
    hipLaunchKernelGGL((decode_kernel<IN, OT, DK, BV, true>), dim3((unsigned)grid), dim3(kThreads), 0, stream, p);
  else
    hipLaunchKernelGGL((decode_kernel<IN, OT, DK, BV, false>), dim3((unsigned)grid), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

template <typename IN, typename OT>
hipError_t launch_decode_in(const OpParams& p, hipStream_t stream) {
  if (p.DK == 128) return launch_decode_t<IN, OT, 128>(p, stream);
  return launch_decode_t<IN, OT, 64>(p, stream);
}

}  // namespace

hipError_t launch_decode(const OpParams& p, bool bf16, hipStream_t stream) {
  if (bf16) {
    if (p.out_bf16) return launch_decode_in<u16, u16>(p, stream);
    return launch_decode_in<u16, float>(p, stream);
  }
  return launch_decode_in<float, float>(p, stream);
}

}  // namespace rla
