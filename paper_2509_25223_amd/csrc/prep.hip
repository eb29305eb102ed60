// Chunk-parallel, state-independent work of one (chunk, head): one 256-thread
// workgroup per pair.
//
// For chunk tokens t, s = 0..63 (paper Sec. 3.4 recurrences, written in the
// chunk form; padding rows beyond the chunk's length carry k = q = 0,
// beta = gamma = 0 and decay 1, which makes them exact no-ops):
//   g_t = sum_{j<=t} log aS_j,  h_t = sum_{j<=t} log aR_j
//   Gram G = K K^T and scores P = Q K^T on bf16 (or fp32) MFMA; fp16 MFMA
//   for the fp16 rows of the in-operator q, k normalisation
//   MG[t][s] = e^{g_{t-1}-g_s} G[t][s]  (s < t)   -> S_{t-1} k_t read-out
//   MP[t][s] = e^{g_t - g_s}   P[t][s]  (s < t)   -> aS_t S_{t-1} q_t read-out
//   MR[t][s] = e^{h_t - h_s}   P[t][s]  (s <= t)  -> R_t q_t read-out
//   (decayed residual: MG with e^{g_t - g_s}, the aS_t S_{t-1} k_t read-out;
//    ungated output: MP with e^{g_{t-1} - g_s}, the S_{t-1} q_t read-out)
//   RDN only: the delta rule S_t = aS_t S_{t-1}(I - b_t k_t k_t^T) + b_t v_t k_t^T
//   makes the chunk's corrections U solve (I + A^S) U = rhs with
//   A^S[t][s] = b_t e^{g_t-g_s} G[t][s] (s < t); likewise A^R with (gamma, h).
//   T^S = (I + A^S)^{-1} and T^R = (I + A^R)^{-1} are formed here in fp32 by
//   blocked forward substitution (16 x 16 diagonal blocks, then block rows).
// All exponents are of differences g_t - g_s <= 0 (never e^{g} e^{-g}).
#include <type_traits>

#include "kernels.hpp"

namespace rla {

namespace {

constexpr int kLdA = kChunk + 4;   // fp32 64 x 64 scratch row stride

template <typename T, int DK>
struct PrepLayout {
  static constexpr int kLdK = DK + (sizeof(T) == 2 ? 8 : 4);   // Kc / Qc row stride
  static constexpr int kLdA = rla::kLdA;
  // region 0: Kc, Qc (T) -- later reused by As, Ar (fp32), which the
  // inversion overwrites with T^S, T^R
  static constexpr int kBytesKQ = 2 * kChunk * kLdK * (int)sizeof(T);
  static constexpr int kBytesA = 2 * kChunk * kLdA * 4;
  static constexpr int kBytes0 = kBytesKQ > kBytesA ? kBytesKQ : kBytesA;
  static constexpr int kBytesW = 4 * 256 * 4;                   // per-wave block products
  static constexpr int kBytesGates = 5 * kChunk * 4;
  static constexpr int kBytes = kBytes0 + kBytesW + kBytesGates;
  static_assert(kBytes <= 40 * 1024, "prep LDS: four workgroups per CU");
};

// Offset (in floats, row stride kLdA) of 16 x 16 block (bi, bj), bi >= bj, of
// an inverse T kept in the storage of its own A: diagonal blocks in place,
// off-diagonal ones in the (unused) mirror position above the diagonal,
// block (bi, bj) at (bj, bi), each block untransposed.
__device__ __forceinline__ int tblk(int bi, int bj) {
  return bi == bj ? 16 * bi * kLdA + 16 * bj : 16 * bj * kLdA + 16 * bi;
}

// Inverse T = (I + A)^{-1} of a unit lower-triangular 64 x 64 matrix (A
// strictly lower, fp32, row stride kLdA) for two matrices at once (A0, A1),
// in 16 x 16 blocks, each T written into the storage of its A (tblk): the
// diagonal blocks T_ii = (I + A_ii)^{-1} by forward substitution (one lane
// per column, every read of A_ii before the wave's writes), then each block
// column j by
//   T_ij = -T_ii * sum_{m=j}^{i-1} A_im T_mj        (i = j+1 .. 3)
// on fp32 MFMA, which reads only the off-diagonal blocks of A below the
// diagonal (never overwritten) and blocks of T.  Wave w takes matrix w >> 1
// and block column 0 (w even) or block columns 1 and 2 (w odd); a column
// only reads its own blocks and the diagonal ones, so one barrier separates
// the two phases.  P: 4 x 256 floats of per-wave scratch.
__device__ void invert_unit_lower_pair(float* A0, float* A1, float* P) {
  constexpr int ld = kLdA;
  typedef Mfma<float> F;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  // ---- diagonal blocks: lanes 0..31 of wave w solve blocks 2w and 2w+1 ----
  if (lane < 32) {
    const int b = 2 * w + (lane >> 4), mat = b >> 2, blk = b & 3, c = lane & 15;
    float* A = (mat ? A1 : A0) + (16 * blk) * ld + 16 * blk;
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float acc = (i == c) ? 1.f : 0.f;
#pragma unroll
      for (int k = 0; k < i; ++k) acc = __builtin_fmaf(-A[i * ld + k], x[k], acc);
      x[i] = (i < c) ? 0.f : acc;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) A[i * ld + c] = x[i];
  }
  __syncthreads();
  // ---- off-diagonal blocks, one block column chain per wave ----
  float* A = (w >> 1) ? A1 : A0;   // A below the diagonal, T per tblk
  float* Pw = P + w * 256;         // [16][16], k-major rows
  const int n = lane & 15, kg = lane >> 4;
  auto solve_block = [&](int i, int j) {   // T_ij from T_jj .. T_{i-1,j}
    floatx4 s = zero4();
    for (int m = j; m < i; ++m) {   // s += A_im T_mj
      const float* Y = A + tblk(m, j);
#pragma unroll
      for (int k0 = 0; k0 < 16; k0 += F::kStep)
        s = F::mma(A[(16 * i + n) * ld + 16 * m + k0 + kg], Y[(k0 + kg) * ld + n], s);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) Pw[(4 * kg + r) * 16 + n] = s[r];
    floatx4 t = zero4();
    const float* Tii = A + tblk(i, i);
#pragma unroll
    for (int k0 = 0; k0 < 16; k0 += F::kStep)   // T_ii * P (wave-local LDS order)
      t = F::mma(Tii[n * ld + k0 + kg], Pw[(k0 + kg) * 16 + n], t);
    float* Tij = A + tblk(i, j);
#pragma unroll
    for (int r = 0; r < 4; ++r) Tij[(4 * kg + r) * ld + n] = -t[r];
  };
  if ((w & 1) == 0) {
    solve_block(1, 0);
    solve_block(2, 0);
    solve_block(3, 0);
  } else {
    solve_block(2, 1);
    solve_block(3, 2);
    solve_block(3, 1);
  }
}

// T: input element type (bf16 bits or fp32).  The matrices are written as
// XT: fp16 for bf16 inputs (their entries are bounded by the decays, beta,
// gamma <= 1 and unit-scale keys; fp16 keeps 11 mantissa bits), fp32 otherwise.
template <typename T, int DK, bool RDN>
__global__ __launch_bounds__(kThreads) void prep_kernel(OpParams p) {
  typedef PrepLayout<T, DK> L;
  typedef typename std::conditional<sizeof(T) == 2, f16, float>::type XT;
  extern __shared__ __align__(16) unsigned char smem[];
  T* Kc = reinterpret_cast<T*>(smem);
  T* Qc = Kc + kChunk * L::kLdK;
  float* As = reinterpret_cast<float*>(smem);   // reuses region 0 after G, P
  float* Ar = As + kChunk * L::kLdA;             // (then T^S, T^R: tblk)
  float* W = reinterpret_cast<float*>(smem + L::kBytes0);
  float* gs = W + 4 * 256;
  float* gr = gs + kChunk;
  float* bt = gr + kChunk;
  float* gm = bt + kChunk;
  float* gsp = gm + kChunk;   // g_{t-1}

  // heads vary fastest over consecutive workgroups, which then read one
  // contiguous stretch of the token rows (every head of the chunk)
  const int h = blockIdx.x, c = blockIdx.y, tid = threadIdx.x;
  ChunkInfo ci;
  if (!chunk_info(p.st, c, ci)) return;
  const int H = p.H;

  // ---- every global load of the workgroup is issued before any is used:
  //      the gates (waves 0, 1), then the K, Q rows (zero padding beyond the
  //      chunk), so their latencies overlap ----
  const bool pre = (p.vflags & kVarGatePreact) != 0;
  float graw_a = 0.f, graw_b = 0.f;   // decay; beta (wave 0) or gamma (wave 1)
  if (tid < 128) {
    const int t = tid & 63;
    if (t < ci.len) {
      const int64_t gi = (ci.tok + t) * H + h;
      graw_a = (tid < 64 ? p.alpha_s : p.alpha_r)[gi];
      graw_b = (tid < 64 ? p.beta : p.gamma)[gi];
    }
  }
  {
    constexpr int kVec = 16 / sizeof(T);           // elements per 16-byte load
    constexpr int kPerRow = DK / kVec;
    constexpr int kIter = kChunk * kPerRow / kThreads;
    static_assert(kIter * kThreads == kChunk * kPerRow, "whole rows per step");
    const T* qg = reinterpret_cast<const T*>(p.q);
    const T* kg = reinterpret_cast<const T*>(p.k);
    uint4 kv[kIter], qv[kIter];
#pragma unroll
    for (int u = 0; u < kIter; ++u) {
      const int e = tid + u * kThreads, t = e / kPerRow, col = (e % kPerRow) * kVec;
      kv[u] = make_uint4(0, 0, 0, 0);
      qv[u] = make_uint4(0, 0, 0, 0);
      if (t < ci.len) {
        const int64_t off = ((ci.tok + t) * H + h) * (int64_t)DK + col;
        kv[u] = *reinterpret_cast<const uint4*>(kg + off);
        qv[u] = *reinterpret_cast<const uint4*>(qg + off);
      }
    }
#pragma unroll
    for (int u = 0; u < kIter; ++u) {
      const int e = tid + u * kThreads, t = e / kPerRow, col = (e % kPerRow) * kVec;
      *reinterpret_cast<uint4*>(Kc + t * L::kLdK + col) = kv[u];
      *reinterpret_cast<uint4*>(Qc + t * L::kLdK + col) = qv[u];
    }
  }
  // ---- gates: wave 0 scans log aS, wave 1 scans log aR ----
  // (pre-activations: log a = -a_h softplus(z + b_h), beta = sigmoid(z),
  //  gamma = sigmoid(z))
  if (tid < 128) {
    const int t = tid & 63;
    const bool valid = t < ci.len;
    float la = 0.f;
    if (valid) la = pre ? -p.decay_param[h] * softplus_f(graw_a + p.decay_param[H + h]) : log_decay(graw_a);
    const float cum = wave_inclusive_scan(la);
    const float wb = valid ? (pre ? sigmoid_f(graw_b) : graw_b) : 0.f;
    if (tid < 64) {
      gs[t] = cum;
      bt[t] = wb;
      gsp[t] = cum - la;
    } else {
      gr[t] = cum;
      gm[t] = wb;
    }
  }
  __syncthreads();
  float* gate_out = p.gate_ws + ((int64_t)c * H + h) * kGateBlock;
  if (tid < 64) {
    gate_out[tid] = gs[tid];
    gate_out[64 + tid] = gr[tid];
    gate_out[128 + tid] = bt[tid];
    gate_out[192 + tid] = gm[tid];
  }

  // ---- G = K K^T and P = Q K^T: wave w owns rows 16w..16w+15 (fp16 MFMA
  //      when q, k are the pre-processing's fp16 rows) ----
  const int w = tid >> 6;
  floatx4 G[4], P[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) {
    G[ct] = zero4();
    P[ct] = zero4();
    if (sizeof(T) == 2 && p.qk_f16) {
      const f16* Kh = reinterpret_cast<const f16*>(Kc);
      const f16* Qh = reinterpret_cast<const f16*>(Qc);
      mma_tile<f16, DK, true, true>(G[ct], Kh + 16 * w * L::kLdK, L::kLdK, Kh + 16 * ct * L::kLdK, L::kLdK);
      mma_tile<f16, DK, true, true>(P[ct], Qh + 16 * w * L::kLdK, L::kLdK, Kh + 16 * ct * L::kLdK, L::kLdK);
    } else {
      mma_tile<T, DK, true, true>(G[ct], Kc + 16 * w * L::kLdK, L::kLdK, Kc + 16 * ct * L::kLdK, L::kLdK);
      mma_tile<T, DK, true, true>(P[ct], Qc + 16 * w * L::kLdK, L::kLdK, Kc + 16 * ct * L::kLdK, L::kLdK);
    }
  }
  __syncthreads();   // Kc/Qc dead: region 0 becomes As/Ar

  XT* mats = reinterpret_cast<XT*>(p.mat_ws) + ((int64_t)c * H + h) * kNumMats * kMatElems;
  if (tid < kNumMats)   // each matrix's zero pad (the scans' DMA source above the diagonal)
    *reinterpret_cast<uint4*>(mats + tid * kMatElems + kMatPacked) = make_uint4(0, 0, 0, 0);
  floatx4 mg[4], mp[4], mr[4];   // this wave's 16-row strips of MG, MP, MR
  // the gate values of this lane's rows and columns, read once up front (a
  // read needed only under a condition would become a branch with its own
  // wait); masked entries are multiplied by 0
  float gs_t[4], gsp_t[4], gr_t[4], bt_t[4], gm_t[4], gs_s[4], gr_s[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int t = 16 * w + acc_row(r);
    gs_t[r] = gs[t];
    gsp_t[r] = gsp[t];
    gr_t[r] = gr[t];
    bt_t[r] = bt[t];
    gm_t[r] = gm[t];
  }
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) {
    const int s = 16 * ct + acc_col();
    gs_s[ct] = gs[s];
    gr_s[ct] = gr[s];
  }
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) {
    const int s = 16 * ct + acc_col();
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = 16 * w + acc_row(r);
      const float g = G[ct][r], pq = P[ct][r];
      const float es = __expf(fminf(gs_t[r] - gs_s[ct], 0.f));
      const float esp = __expf(fminf(gsp_t[r] - gs_s[ct], 0.f));
      const float er = __expf(fminf(gr_t[r] - gr_s[ct], 0.f));
      const bool lower = s < t;
      const float lm = lower ? 1.f : 0.f;
      const float eg = (p.vflags & kVarDecayed) ? es : esp;
      const float ep = (p.vflags & kVarUngated) ? esp : es;
      mg[ct][r] = lower ? eg * g : 0.f;
      mp[ct][r] = lower ? ep * pq : 0.f;
      mr[ct][r] = s <= t ? er * pq : 0.f;
      if constexpr (RDN) {
        As[t * L::kLdA + s] = lm * (bt_t[r] * es * g);
        Ar[t * L::kLdA + s] = lm * (gm_t[r] * er * g);
      }
    }
  }
  // the blocks on and below the diagonal, packed (tri_off): wave w holds
  // block row w
  if constexpr (sizeof(XT) == 2) {
    // fp16 rows leave in 16-byte stores: each 16 x 32 half strip goes through
    // this wave's block-product scratch (1 KiB, unused until the inversion),
    // written column-major (one 8-byte store of 4 rows per tile and lane) and
    // read back with transpose reads that give lane (g, i) row 16 w + i at
    // columns 8 g .. 8 g + 7 of the half strip
    typedef PadRows<XT, 16, 0> TS;   // [32 columns][16 rows]
    XT* stg = reinterpret_cast<XT*>(W + w * 256);
    const int g = (tid & 63) >> 4, i = tid & 15;
#pragma unroll
    for (int m = 0; m < 3; ++m) {
      const floatx4* x = m == 0 ? mg : m == 1 ? mp : mr;
      XT* base = mats + (m == 0 ? kMatMG : m == 1 ? kMatMP : kMatMR) * kMatElems;
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        if (2 * half > w) continue;   // both blocks of the strip pair above the diagonal
        asm volatile("" ::: "memory");   // the previous half strip's reads come first
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          f16x4 v4;
#pragma unroll
          for (int r = 0; r < 4; ++r) v4[r] = (f16)x[2 * half + k][r];
          *reinterpret_cast<f16x4*>(TS::ptr(stg, 16 * k + acc_col(), acc_row(0))) = v4;
        }
        asm volatile("" ::: "memory");   // the stores above come before the reads
        const uint4 v = tile_token_rows16_sync<TS>(stg, 0);
        const int s0 = 32 * half + 8 * g;
        if ((s0 >> 4) <= w) *reinterpret_cast<uint4*>(base + tri_off(16 * w + i, s0)) = v;
      }
    }
    asm volatile("" ::: "memory");
  } else {
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      if (ct > w) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = 16 * w + acc_row(r), s = 16 * ct + acc_col();
        mats[kMatMG * kMatElems + tri_off(t, s)] = mg[ct][r];
        mats[kMatMP * kMatElems + tri_off(t, s)] = mp[ct][r];
        mats[kMatMR * kMatElems + tri_off(t, s)] = mr[ct][r];
      }
    }
  }
  if constexpr (RDN) {
    __syncthreads();
    invert_unit_lower_pair(As, Ar, W);
    __syncthreads();
    // 8 consecutive elements per thread and step (16-byte fp16 stores), the
    // blocks on and below the diagonal packed (tri_off)
    for (int e = 8 * tid; e < kChunk * kChunk; e += 8 * kThreads) {
      const int t = e / kChunk, s = e % kChunk;
      const bool upper = (s >> 4) > (t >> 4);   // blocks above the diagonal are zero
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        // two 16-byte reads (blocks of T above the diagonal are zero: the
        // bits read there are cleared with a mask, not read under a
        // condition)
        const float* src = (m ? Ar : As) + tblk(t >> 4, s >> 4) + (t & 15) * L::kLdA + (s & 15);
        const uint4 b0 = keep_if(*reinterpret_cast<const uint4*>(src), !upper);
        const uint4 b1 = keep_if(*reinterpret_cast<const uint4*>(src + 4), !upper);
        const floatx4 f0 = __builtin_bit_cast(floatx4, b0), f1 = __builtin_bit_cast(floatx4, b1);
        XT vals[8];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          vals[k] = from_f<XT>(f0[k]);
          vals[4 + k] = from_f<XT>(f1[k]);
        }
        XT* dst = mats + (m ? kMatTR : kMatTS) * kMatElems + tri_off(t, s);
        if (upper) continue;
        if constexpr (sizeof(XT) == 2) {
          *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(vals);
        } else {
#pragma unroll
          for (int k = 0; k < 8; ++k) dst[k] = vals[k];
        }
      }
    }
  }
}

template <typename T, int DK, bool RDN>
hipError_t launch_prep_t(const OpParams& p, hipStream_t stream) {
  typedef PrepLayout<T, DK> L;
  auto kern = prep_kernel<T, DK, RDN>;
  hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, L::kBytes);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(kern, dim3(p.H, p.max_chunks), dim3(kThreads), L::kBytes, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_prep(const OpParams& p, bool bf16, hipStream_t stream) {
  if (p.max_chunks == 0) return hipSuccess;
  if (bf16) {
    if (p.DK == 128) return p.rdn ? launch_prep_t<u16, 128, true>(p, stream) : launch_prep_t<u16, 128, false>(p, stream);
    return p.rdn ? launch_prep_t<u16, 64, true>(p, stream) : launch_prep_t<u16, 64, false>(p, stream);
  }
  return p.rdn ? launch_prep_t<float, 64, true>(p, stream) : launch_prep_t<float, 64, false>(p, stream);
}

}  // namespace rla
