// Forward state-passing scan of RLA / RDN: one 256-thread workgroup per
// (sequence, head, value block of BV columns).  Value columns evolve
// independently (the clip is elementwise and every state update acts on rows
// of the paper's d_v x d_k states), so value blocks need no communication.
//
// The workgroup walks the sequence chunk by chunk.  S and R (d_k x BV fp32,
// stored transposed like the ABI) stay in MFMA accumulators for the whole
// sequence.  Per chunk, with the prep kernel's gate sums and matrices:
//   KS = K S0, QS = Q S0, KR = K R0, QR = Q R0                 (MFMA)
//   RDN: U = T^S diag(b) (V - e^{g} KS)     RLA: U = diag(b) V
//   p   = e^{g_{t-1}} KS + MG U         = S_{t-1} k_t         (Sec. 3.4)
//   r   = clip(V - p)                   fused, never written to HBM
//   b_t = e^{g} QS + MP U               = aS_t S_{t-1} q_t
//   RDN: UR = T^R diag(gamma) (r - e^{h} KR)   RLA: UR = diag(gamma) r
//   c_t = e^{h} QR + MR UR              = R_t q_t
//   o   = b + diag(gamma) c
//   S  <- e^{g_C} S + K^T diag(e^{g_C - g}) U,  R likewise with (h, UR)
//
// Operand precision (bf16 inputs; fp32 inputs use fp32 MFMA throughout):
//   K, Q x state: bf16 K/Q fragments (exact inputs, loaded from HBM straight
//     into registers) times the state split as bf16 hi + bf16 lo (~16-bit
//     mantissa, fp32 range): two MFMAs per step.
//   everything else: fp16 operands (intermediates bounded by the data, clip
//     and gates), fp32 accumulation.
// With `CKPT` the chunk-start states and the clip mask |x| <= c are stored
// for the backward pass.
#include <type_traits>

#include "kernels.hpp"

namespace rla {

namespace {

template <typename IN, int DK, int BV, bool RDN>
struct FwdLayout {
  static constexpr bool kBF = sizeof(IN) == 2;
  typedef typename std::conditional<kBF, f16, float>::type XT;
  static constexpr int kPad = kBF ? 8 : 4;
  static constexpr int kLdX = kChunk + kPad;    // K^T rows, matrices, per-token blocks
  static constexpr int kLdS = DK + kPad;        // state copies [BV][DK]
  static constexpr int kNumM = RDN ? 5 : 3;
  static constexpr int kNumCopies = kBF ? 4 : 2;
  static constexpr int kKT = 0;
  static constexpr int kCopies = kKT + DK * kLdX * (int)sizeof(XT);
  static constexpr int kCopyBytes = BV * kLdS * (int)sizeof(IN);
  static constexpr int kMats = kCopies + kNumCopies * kCopyBytes;
  static constexpr int kBufs = kMats + kNumM * kChunk * kLdX * (int)sizeof(XT);
  static constexpr int kBufBytes = BV * kLdX * (int)sizeof(XT);
  static constexpr int kVc = kBufs + 5 * kBufBytes;
  static constexpr int kGates = kVc + kChunk * BV * (int)sizeof(IN);
  static constexpr int kBytes = kGates + 10 * kChunk * 4;
  static_assert(kBytes <= 160 * 1024, "forward scan LDS");
};

// Writes this lane's 4 accumulator rows of a state tile into the transposed
// state copy: hi (and, for bf16, the residual lo).
template <typename IN>
__device__ __forceinline__ void store_state_copy(IN* hi, IN* lo, int ld, floatx4 v) {
  const int off = acc_col() * ld + acc_row(0);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if constexpr (sizeof(IN) == 2) {
      const u16 h = f2bf(v[r]);
      hi[off + r] = h;
      lo[off + r] = bf16_lo(v[r], h);
    } else {
      hi[off + r] = v[r];
    }
  }
}

template <typename IN, int DK, int BV, bool RDN, bool WRITE_O, bool CKPT, typename OT>
__global__ __launch_bounds__(kThreads) void fwd_scan_kernel(OpParams p) {
  typedef FwdLayout<IN, DK, BV, RDN> L;
  typedef typename L::XT XT;
  typedef Mfma<IN> MI;
  constexpr bool BF = L::kBF;
  constexpr int JT = BV / 16;        // value tiles per block
  constexpr int IT = DK / 64;        // state row tiles per wave
  constexpr int KS_STEPS = DK / MI::kStep;
  extern __shared__ __align__(16) unsigned char smem[];
  XT* KT = reinterpret_cast<XT*>(smem + L::kKT);
  IN* Shi = reinterpret_cast<IN*>(smem + L::kCopies);
  IN* Rhi = reinterpret_cast<IN*>(smem + L::kCopies + 1 * L::kCopyBytes);
  IN* Slo = reinterpret_cast<IN*>(smem + L::kCopies + 2 * L::kCopyBytes);   // bf16 only
  IN* Rlo = reinterpret_cast<IN*>(smem + L::kCopies + 3 * L::kCopyBytes);   // bf16 only
  XT* mats = reinterpret_cast<XT*>(smem + L::kMats);
  XT* Yt = reinterpret_cast<XT*>(smem + L::kBufs);               // Y, later YR
  XT* Ut = reinterpret_cast<XT*>(smem + L::kBufs + 1 * L::kBufBytes);
  XT* URt = reinterpret_cast<XT*>(smem + L::kBufs + 2 * L::kBufBytes);
  XT* DUt = reinterpret_cast<XT*>(smem + L::kBufs + 3 * L::kBufBytes);
  XT* DURt = reinterpret_cast<XT*>(smem + L::kBufs + 4 * L::kBufBytes);
  IN* Vc = reinterpret_cast<IN*>(smem + L::kVc);
  float* gbt = reinterpret_cast<float*>(smem + L::kGates);   // beta
  float* ggm = gbt + kChunk;        // gamma
  float* egs = ggm + kChunk;        // e^{g_t}
  float* egsp = egs + kChunk;       // e^{g_{t-1}}
  float* egr = egsp + kChunk;       // e^{h_t}
  float* dls = egr + kChunk;        // e^{g_C - g_t}
  float* dlr = dls + kChunk;        // e^{h_C - h_t}
  float* edge = dlr + kChunk;       // [0] = e^{g_C}, [1] = e^{h_C}

  // matrix slots in LDS: RDN {TS, MG, MP, TR, MR}, RLA {MG, MP, MR}
  XT* mTS = mats;
  XT* mMG = mats + (RDN ? 1 : 0) * kChunk * L::kLdX;
  XT* mMP = mats + (RDN ? 2 : 1) * kChunk * L::kLdX;
  XT* mTR = mats + 3 * kChunk * L::kLdX;
  XT* mMR = mats + (RDN ? 4 : 2) * kChunk * L::kLdX;

  const int H = p.H, DV = p.DV, tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  // XCD-aware block mapping: the value blocks of one (sequence, head) pair get
  // block ids that are congruent mod 8, so they share one XCD's L2.
  const int nvb = DV / BV;
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int pair = (slot / nvb) * 8 + xcd, vb = slot % nvb;
  if (pair >= p.st.nseq * H) return;
  const int n = seq_order(p.st, pair / H), h = pair % H;
  const SeqInfo si = seq_info(p.st, n);
  const int nch = (si.len + kChunk - 1) / kChunk;
  const int j0 = vb * BV;
  const float clip = p.clip;
  const int64_t state_off = ((int64_t)n * H + h) * DK * DV;

  // ---- initial states into accumulators (wave w: rows [w*DK/4, (w+1)*DK/4)) ----
  floatx4 Sacc[IT][JT], Racc[IT][JT];
#pragma unroll
  for (int it = 0; it < IT; ++it)
#pragma unroll
    for (int jt = 0; jt < JT; ++jt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = w * (DK / 4) + it * 16 + acc_row(r), j = j0 + jt * 16 + acc_col();
        Sacc[it][jt][r] = p.S0 ? p.S0[state_off + (int64_t)i * DV + j] : 0.f;
        Racc[it][jt][r] = p.R0 ? p.R0[state_off + (int64_t)i * DV + j] : 0.f;
      }
  auto write_state_copies = [&]() {
#pragma unroll
    for (int it = 0; it < IT; ++it)
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        const int o = (jt * 16) * L::kLdS + w * (DK / 4) + it * 16;
        store_state_copy<IN>(Shi + o, Slo + o, L::kLdS, Sacc[it][jt]);
        store_state_copy<IN>(Rhi + o, Rlo + o, L::kLdS, Racc[it][jt]);
      }
  };
  write_state_copies();

  const IN* qg = reinterpret_cast<const IN*>(p.q);
  const IN* kg = reinterpret_cast<const IN*>(p.k);
  const IN* vg = reinterpret_cast<const IN*>(p.v);
  OT* og = reinterpret_cast<OT*>(p.o);
  const XT* matg = reinterpret_cast<const XT*>(p.mat_ws);

  for (int c = 0; c < nch; ++c) {
    const int gc = si.chunk0 + c;
    const int64_t tok = si.start + (int64_t)c * kChunk;
    const int len = min(kChunk, si.len - c * kChunk);

    if constexpr (CKPT) {
      const int64_t off = ((int64_t)gc * H + h) * DK * DV;
#pragma unroll
      for (int it = 0; it < IT; ++it)
#pragma unroll
        for (int jt = 0; jt < JT; ++jt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int i = w * (DK / 4) + it * 16 + acc_row(r), j = j0 + jt * 16 + acc_col();
            p.ck_S[off + (int64_t)i * DV + j] = Sacc[it][jt][r];
            p.ck_R[off + (int64_t)i * DV + j] = Racc[it][jt][r];
          }
    }

    // ---- stage the chunk: K, Q fragments of this wave's rows into registers,
    //      K^T (XT) into LDS, V block, matrices, gates ----
    typename MI::frag Kf[KS_STEPS], Qf[KS_STEPS];
    {
      const int t = 16 * w + (lane & 15);
      const int64_t roff = ((tok + t) * H + h) * (int64_t)DK;
      load_rowfrags<IN, DK>(Kf, t < len ? kg + roff : nullptr);
      load_rowfrags<IN, DK>(Qf, t < len ? qg + roff : nullptr);
#pragma unroll
      for (int s = 0; s < KS_STEPS; ++s) {
        if constexpr (BF) {
          const u16x8 kv = __builtin_bit_cast(u16x8, Kf[s]);
#pragma unroll
          for (int e = 0; e < 8; ++e)
            KT[(s * 32 + (lane >> 4) * 8 + e) * L::kLdX + t] = from_f<XT>(bf2f(kv[e]));
        } else {
          KT[(s * 4 + (lane >> 4)) * L::kLdX + t] = Kf[s];
        }
      }
      constexpr int kVecV = 16 / sizeof(IN), kVPerRow = BV / kVecV;
      for (int e = tid; e < kChunk * kVPerRow; e += kThreads) {
        const int tt = e / kVPerRow, jj = (e % kVPerRow) * kVecV;
        uint4 vv = make_uint4(0, 0, 0, 0);
        if (tt < len) vv = *reinterpret_cast<const uint4*>(vg + ((tok + tt) * H + h) * (int64_t)DV + j0 + jj);
        *reinterpret_cast<uint4*>(Vc + tt * BV + jj) = vv;
      }
      constexpr int kVecM = 16 / sizeof(XT);
      constexpr int kMatVecs = kMatElems / kVecM;
      const XT* mg = matg + ((int64_t)gc * H + h) * kNumMats * kMatElems;
      constexpr int kSrc[5] = {kMatTS, kMatMG, kMatMP, kMatTR, kMatMR};
      constexpr int kSrcRla[3] = {kMatMG, kMatMP, kMatMR};
#pragma unroll
      for (int m = 0; m < L::kNumM; ++m) {
        const int src = RDN ? kSrc[m] : kSrcRla[m];
        for (int e = tid; e < kMatVecs; e += kThreads) {
          const int tt = e / (kChunk / kVecM), ss = (e % (kChunk / kVecM)) * kVecM;
          *reinterpret_cast<uint4*>(mats + (m * kChunk + tt) * L::kLdX + ss) =
              *reinterpret_cast<const uint4*>(mg + src * kMatElems + tt * kChunk + ss);
        }
      }
      if (tid < kChunk) {
        const float* gb = p.gate_ws + ((int64_t)gc * H + h) * kGateBlock;
        const int tt = tid;
        const float gs = gb[tt], gsl = gb[kChunk - 1], gsp = tt > 0 ? gb[tt - 1] : 0.f;
        const float gr = gb[64 + tt], grl = gb[64 + kChunk - 1];
        gbt[tt] = gb[128 + tt];
        ggm[tt] = gb[192 + tt];
        egs[tt] = __expf(gs);
        egsp[tt] = __expf(gsp);
        egr[tt] = __expf(gr);
        dls[tt] = __expf(gsl - gs);
        dlr[tt] = __expf(grl - gr);
        if (tt == 0) {
          edge[0] = __expf(gsl);
          edge[1] = __expf(grl);
        }
      }
    }
    __syncthreads();

    // ---- KS, QS, KR, QR for rows 16w..16w+15 ----
    floatx4 KS[JT], QS[JT], KR[JT], QR[JT];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      KS[jt] = zero4(); QS[jt] = zero4(); KR[jt] = zero4(); QR[jt] = zero4();
      const int o = jt * 16 * L::kLdS;
      mma_rega<IN, DK, true>(KS[jt], Kf, Shi + o, L::kLdS);
      mma_rega<IN, DK, true>(QS[jt], Qf, Shi + o, L::kLdS);
      mma_rega<IN, DK, true>(KR[jt], Kf, Rhi + o, L::kLdS);
      mma_rega<IN, DK, true>(QR[jt], Qf, Rhi + o, L::kLdS);
      if constexpr (BF) {
        mma_rega<IN, DK, true>(KS[jt], Kf, Slo + o, L::kLdS);
        mma_rega<IN, DK, true>(QS[jt], Qf, Slo + o, L::kLdS);
        mma_rega<IN, DK, true>(KR[jt], Kf, Rlo + o, L::kLdS);
        mma_rega<IN, DK, true>(QR[jt], Qf, Rlo + o, L::kLdS);
      }
    }
    float vloc[JT][4];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      floatx4 y;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = 16 * w + acc_row(r);
        vloc[jt][r] = to_f<IN>(Vc[t * BV + jt * 16 + acc_col()]);
        y[r] = RDN ? gbt[t] * (vloc[jt][r] - egs[t] * KS[jt][r]) : gbt[t] * vloc[jt][r];
      }
      if constexpr (RDN) {
        store_acc_t<XT>(Yt + jt * 16 * L::kLdX + 16 * w, L::kLdX, y);
      } else {
        floatx4 du;
#pragma unroll
        for (int r = 0; r < 4; ++r) du[r] = dls[16 * w + acc_row(r)] * y[r];
        store_acc_t<XT>(Ut + jt * 16 * L::kLdX + 16 * w, L::kLdX, y);
        store_acc_t<XT>(DUt + jt * 16 * L::kLdX + 16 * w, L::kLdX, du);
      }
    }
    __syncthreads();

    if constexpr (RDN) {   // U = T^S Y
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        floatx4 u = zero4();
        mma_tile<XT, kChunk, true, true>(u, mTS + 16 * w * L::kLdX, L::kLdX, Yt + jt * 16 * L::kLdX, L::kLdX);
        floatx4 du;
#pragma unroll
        for (int r = 0; r < 4; ++r) du[r] = dls[16 * w + acc_row(r)] * u[r];
        store_acc_t<XT>(Ut + jt * 16 * L::kLdX + 16 * w, L::kLdX, u);
        store_acc_t<XT>(DUt + jt * 16 * L::kLdX + 16 * w, L::kLdX, du);
      }
      __syncthreads();
    }

    // ---- residual, clip, base read-out ----
    floatx4 base[JT];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      floatx4 mgu = zero4(), mpu = zero4();
      mma_tile<XT, kChunk, true, true>(mgu, mMG + 16 * w * L::kLdX, L::kLdX, Ut + jt * 16 * L::kLdX, L::kLdX);
      mma_tile<XT, kChunk, true, true>(mpu, mMP + 16 * w * L::kLdX, L::kLdX, Ut + jt * 16 * L::kLdX, L::kLdX);
      floatx4 y;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = 16 * w + acc_row(r);
        const float x = vloc[jt][r] - egsp[t] * KS[jt][r] - mgu[r];
        const float rr = clip < 0.f ? x : fminf(fmaxf(x, -clip), clip);
        if constexpr (CKPT) {
          if (t < len)
            p.ck_mask[((tok + t) * H + h) * (int64_t)DV + j0 + jt * 16 + acc_col()] =
                (clip < 0.f || fabsf(x) <= clip) ? 1 : 0;
        }
        base[jt][r] = egs[t] * QS[jt][r] + mpu[r];
        y[r] = RDN ? ggm[t] * (rr - egr[t] * KR[jt][r]) : ggm[t] * rr;
      }
      if constexpr (RDN) {
        store_acc_t<XT>(Yt + jt * 16 * L::kLdX + 16 * w, L::kLdX, y);
      } else {
        floatx4 du;
#pragma unroll
        for (int r = 0; r < 4; ++r) du[r] = dlr[16 * w + acc_row(r)] * y[r];
        store_acc_t<XT>(URt + jt * 16 * L::kLdX + 16 * w, L::kLdX, y);
        store_acc_t<XT>(DURt + jt * 16 * L::kLdX + 16 * w, L::kLdX, du);
      }
    }
    __syncthreads();

    if constexpr (RDN) {   // UR = T^R YR
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        floatx4 u = zero4();
        mma_tile<XT, kChunk, true, true>(u, mTR + 16 * w * L::kLdX, L::kLdX, Yt + jt * 16 * L::kLdX, L::kLdX);
        floatx4 du;
#pragma unroll
        for (int r = 0; r < 4; ++r) du[r] = dlr[16 * w + acc_row(r)] * u[r];
        store_acc_t<XT>(URt + jt * 16 * L::kLdX + 16 * w, L::kLdX, u);
        store_acc_t<XT>(DURt + jt * 16 * L::kLdX + 16 * w, L::kLdX, du);
      }
      __syncthreads();
    }

    // ---- correction read-out and output ----
    if constexpr (WRITE_O) {
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        floatx4 mru = zero4();
        mma_tile<XT, kChunk, true, true>(mru, mMR + 16 * w * L::kLdX, L::kLdX, URt + jt * 16 * L::kLdX, L::kLdX);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = 16 * w + acc_row(r);
          const float cc = egr[t] * QR[jt][r] + mru[r];
          if (t < len)
            og[((tok + t) * H + h) * (int64_t)DV + j0 + jt * 16 + acc_col()] =
                from_f<OT>(base[jt][r] + ggm[t] * cc);
        }
      }
    }

    // ---- state update: S <- e^{g_C} S + K^T DU, R <- e^{h_C} R + K^T DUR ----
    const float eS = edge[0], eR = edge[1];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const XT* Ai = KT + (w * (DK / 4) + it * 16) * L::kLdX;
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        Sacc[it][jt] *= eS;
        Racc[it][jt] *= eR;
        mma_tile<XT, kChunk, true, true>(Sacc[it][jt], Ai, L::kLdX, DUt + jt * 16 * L::kLdX, L::kLdX);
        mma_tile<XT, kChunk, true, true>(Racc[it][jt], Ai, L::kLdX, DURt + jt * 16 * L::kLdX, L::kLdX);
      }
    }
    __syncthreads();   // all reads of the state copies, K^T and the blocks are done
    write_state_copies();
  }

  if (p.S_fin || p.R_fin) {
#pragma unroll
    for (int it = 0; it < IT; ++it)
#pragma unroll
      for (int jt = 0; jt < JT; ++jt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = w * (DK / 4) + it * 16 + acc_row(r), j = j0 + jt * 16 + acc_col();
          if (p.S_fin) p.S_fin[state_off + (int64_t)i * DV + j] = Sacc[it][jt][r];
          if (p.R_fin) p.R_fin[state_off + (int64_t)i * DV + j] = Racc[it][jt][r];
        }
  }
}

template <typename IN, int DK, int BV, bool RDN, bool WRITE_O, bool CKPT, typename OT>
hipError_t launch_fwd_t(const OpParams& p, hipStream_t stream) {
  typedef FwdLayout<IN, DK, BV, RDN> L;
  auto kern = fwd_scan_kernel<IN, DK, BV, RDN, WRITE_O, CKPT, OT>;
  hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, L::kBytes);
  if (err != hipSuccess) return err;
  const int nvb = p.DV / BV;
  const int npairs = p.st.nseq * p.H;
  const int grid = ((npairs + 7) / 8) * 8 * nvb;
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(kThreads), L::kBytes, stream, p);
  return hipGetLastError();
}

template <typename IN, int DK, int BV, typename OT>
hipError_t launch_fwd_dk(const OpParams& p, bool write_o, bool ckpt, hipStream_t s) {
  if (p.rdn) {
    if (ckpt) return write_o ? launch_fwd_t<IN, DK, BV, true, true, true, OT>(p, s) : launch_fwd_t<IN, DK, BV, true, false, true, OT>(p, s);
    return launch_fwd_t<IN, DK, BV, true, true, false, OT>(p, s);
  }
  if (ckpt) return write_o ? launch_fwd_t<IN, DK, BV, false, true, true, OT>(p, s) : launch_fwd_t<IN, DK, BV, false, false, true, OT>(p, s);
  return launch_fwd_t<IN, DK, BV, false, true, false, OT>(p, s);
}

}  // namespace

hipError_t launch_fwd_scan(const OpParams& p, bool bf16, bool write_o, bool ckpt,
                           hipStream_t stream) {
  if (bf16) {
    if (p.out_bf16) {
      if (p.DK == 128) return launch_fwd_dk<u16, 128, 32, u16>(p, write_o, ckpt, stream);
      return launch_fwd_dk<u16, 64, 32, u16>(p, write_o, ckpt, stream);
    }
    if (p.DK == 128) return launch_fwd_dk<u16, 128, 32, float>(p, write_o, ckpt, stream);
    return launch_fwd_dk<u16, 64, 32, float>(p, write_o, ckpt, stream);
  }
  return launch_fwd_dk<float, 64, 16, float>(p, write_o, ckpt, stream);
}

}  // namespace rla
