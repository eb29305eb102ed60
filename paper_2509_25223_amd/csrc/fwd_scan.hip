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
// Variants: decayed residual p = e^{g} KS + MG U (= aS_t S_{t-1} k_t, MG with
// e^{g_t - g_s}); ungated output b = e^{g_{t-1}} QS + MP U (= S_{t-1} q_t, MP
// with e^{g_{t-1} - g_s}) and o = b + c; log-cosh residual r = c tanh(x / c).
//
// Operand precision (bf16 inputs; fp32 inputs use fp32 MFMA throughout):
//   K, Q x state: bf16 K/Q fragments (exact inputs, loaded from HBM straight
//     into registers) times the state split as bf16 hi + bf16 lo (~16-bit
//     mantissa, fp32 range): two MFMAs per step.  When q, k are the fp16 rows
//     of the in-operator normalisation (qk_f16, variant instance), each row
//     is split as bf16 hi + bf16 lo too (exact: 11 = 8 + 3 bits) and a third
//     MFMA adds lo x state-hi.
//   everything else: fp16 operands (intermediates bounded by the data, clip
//     and gates), fp32 accumulation.
// With `CKPT` the chunk-start states, the clip mask |x| <= c and the blocks
// U, UR and r (token-major, mm type) are stored for the backward pass.
#include <type_traits>

#include "kernels.hpp"

namespace rla {

namespace {

template <typename IN, int DK, int BV, bool RDN>
struct FwdLayout {
  static constexpr bool kBF = sizeof(IN) == 2;
  typedef typename std::conditional<kBF, f16, float>::type XT;
  typedef Tile<XT, kChunk> TT;   // token tiles: per-token blocks [BV][64]
  // K for the state update's K^T operand: bf16 inputs keep K row-major [64][DK]
  // (16-byte stores at the commit, transpose reads at the update); fp32
  // inputs store K^T [DK][64]
  typedef typename std::conditional<kBF, TrTile<XT, DK>, TT>::type TK;
  typedef Tile<IN, DK> TSC;      // state copies [BV][DK]
  // matrix slots (swizzled 64 x 64 tiles filled by LDS-DMA); with bf16 inputs
  // T^R and MR are double-buffered so the next chunk's copies land early
  static constexpr bool kDB = kBF;
  static constexpr int kNumSlots = RDN ? (kDB ? 7 : 5) : (kDB ? 4 : 3);
  static constexpr int kNumCopies = kBF ? 4 : 2;
  static constexpr int kKT = 0;
  static constexpr int kCopies = kKT + (kBF ? kChunk * TK::kRowB : DK * TT::kRowB);
  static constexpr int kCopyBytes = BV * TSC::kRowB;
  static constexpr int kMats = kCopies + kNumCopies * kCopyBytes;
  static constexpr int kBufs = kMats + kNumSlots * Swz<XT>::kBytes;
  static constexpr int kBufBytes = BV * TT::kRowB;
  static constexpr int kVc = kBufs + 5 * kBufBytes;
  static constexpr int kVBytes = kChunk * BV * (int)sizeof(IN);
  static constexpr int kGraw = kVc + kVBytes;
  static constexpr int kGates = kGraw + kGateBlock * 4;
  // output staging, so that o, the clip mask and r leave in 16-byte stores:
  // r value-major (token tile), mask token-major [64][BV] bytes, o
  // token-major [64][BV + 4] fp32
  static constexpr int kRst = kGates + 10 * kChunk * 4;
  static constexpr int kMst = kRst + kBufBytes;
  static constexpr int kLdO = BV + 4;
  static constexpr int kOst = kMst + kChunk * BV;
  static constexpr int kBytes = kOst + kChunk * kLdO * 4;
  static_assert(kVBytes == 4 * 1024, "V block = one DMA instruction per wave");
  static_assert(kBytes <= 160 * 1024, "forward scan LDS");
  // slot of each matrix (RDN: TS MG MP TR[2] MR[2]; RLA: MG MP MR[2])
  __device__ static constexpr int slot(int mat, int buf) {
    if (RDN) {
      if (mat == kMatTS) return 0;
      if (mat == kMatMG) return 1;
      if (mat == kMatMP) return 2;
      if (mat == kMatTR) return kDB ? 3 + buf : 3;
      return kDB ? 5 + buf : 4;   // MR
    }
    if (mat == kMatMG) return 0;
    if (mat == kMatMP) return 1;
    return kDB ? 2 + buf : 2;     // MR
  }
};

// Writes this lane's 4 accumulator rows of a state tile into the transposed
// state copies (tile rows r0 + column, columns c0 + row): hi (and, for bf16,
// the residual lo).
template <class TL, typename IN>
__device__ __forceinline__ void store_state_copy(IN* hi, IN* lo, int r0, int c0, floatx4 v) {
  // r0, c0 multiples of 16
  const int o = TL::off_split(r0, acc_col(), acc_row(0) * (int)sizeof(IN), c0 * (int)sizeof(IN));
  if constexpr (sizeof(IN) == 2) {   // 8-byte stores of 4 consecutive rows
    uint2 h2, l2;
    bf16_split2(v[0], v[1], h2.x, l2.x);
    bf16_split2(v[2], v[3], h2.y, l2.y);
    *reinterpret_cast<uint2*>(reinterpret_cast<char*>(hi) + o) = h2;
    *reinterpret_cast<uint2*>(reinterpret_cast<char*>(lo) + o) = l2;
  } else {
    *reinterpret_cast<floatx4*>(reinterpret_cast<char*>(hi) + o) = v;
  }
}

// VAR: an instance that reads the variant flags and qk_f16 (the default
// instance compiles them away, so the boxed operator keeps its register budget)
template <typename IN, int DK, int BV, bool RDN, bool WRITE_O, bool CKPT, typename OT, bool VAR>
__global__ __launch_bounds__(kThreads) void fwd_scan_kernel(OpParams p) {
  typedef FwdLayout<IN, DK, BV, RDN> L;
  typedef typename L::XT XT;
  typedef Mfma<IN> MI;
  typedef typename L::TT TT;
  typedef typename L::TK TK;
  constexpr bool BF = L::kBF;
  constexpr int JT = BV / 16;        // value tiles per block
  constexpr int IT = DK / 64;        // state row tiles per wave
  constexpr int KS_STEPS = DK / MI::kStep;
  // store instructions per wave of the two checkpointed states (save_state_f16:
  // one row store and one scale store per 16-row tile; fp32: one per row)
  constexpr int kCkptStores = 2 * (BF ? 2 * IT : 4 * IT * JT);
  extern __shared__ __align__(16) unsigned char smem[];
  XT* KT = reinterpret_cast<XT*>(smem + L::kKT);
  IN* Shi = reinterpret_cast<IN*>(smem + L::kCopies);
  IN* Rhi = reinterpret_cast<IN*>(smem + L::kCopies + 1 * L::kCopyBytes);
  IN* Slo = reinterpret_cast<IN*>(smem + L::kCopies + 2 * L::kCopyBytes);   // bf16 only
  IN* Rlo = reinterpret_cast<IN*>(smem + L::kCopies + 3 * L::kCopyBytes);   // bf16 only
  auto mat = [&](int m, int buf) {
    return reinterpret_cast<XT*>(smem + L::kMats + L::slot(m, buf) * Swz<XT>::kBytes);
  };
  XT* Yt = reinterpret_cast<XT*>(smem + L::kBufs);               // Y, later YR
  XT* Ut = reinterpret_cast<XT*>(smem + L::kBufs + 1 * L::kBufBytes);
  XT* URt = reinterpret_cast<XT*>(smem + L::kBufs + 2 * L::kBufBytes);
  XT* DUt = reinterpret_cast<XT*>(smem + L::kBufs + 3 * L::kBufBytes);
  XT* DURt = reinterpret_cast<XT*>(smem + L::kBufs + 4 * L::kBufBytes);
  IN* Vc = reinterpret_cast<IN*>(smem + L::kVc);
  float* graw = reinterpret_cast<float*>(smem + L::kGraw);   // prep's gate block
  float* gbt = reinterpret_cast<float*>(smem + L::kGates);   // beta
  float* ggm = gbt + kChunk;        // gamma
  float* egs = ggm + kChunk;        // e^{g_t}
  float* egsp = egs + kChunk;       // e^{g_{t-1}}
  float* egr = egsp + kChunk;       // e^{h_t}
  float* dls = egr + kChunk;        // e^{g_C - g_t}
  float* dlr = dls + kChunk;        // e^{h_C - h_t}
  float* edge = dlr + kChunk;       // [0] = e^{g_C}, [1] = e^{h_C}
  // output weight of c: gamma (ungated: 1); the default instance reads gamma
  float* gout = VAR ? edge + kChunk : ggm;
  // per-token factors of S0 in the residual's and the base read-out's terms
  const int vf = VAR ? p.vflags : 0;
  const bool qk16 = VAR && BF && p.qk_f16;   // q, k rows are fp16
  const float* ekp = (vf & kVarDecayed) ? egs : egsp;
  const float* eqb = (vf & kVarUngated) ? egsp : egs;
  const bool tanh_resid = (vf & kVarTanh) != 0;
  XT* Rst = reinterpret_cast<XT*>(smem + L::kRst);            // r (saving mode)
  uint8_t* Mst = reinterpret_cast<uint8_t*>(smem + L::kMst);  // clip mask (saving mode)
  float* Ost = reinterpret_cast<float*>(smem + L::kOst);      // o

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
        store_state_copy<typename L::TSC>(Shi, Slo, jt * 16, w * (DK / 4) + it * 16, Sacc[it][jt]);
        store_state_copy<typename L::TSC>(Rhi, Rlo, jt * 16, w * (DK / 4) + it * 16, Racc[it][jt]);
      }
  };
  write_state_copies();

  const IN* qg = reinterpret_cast<const IN*>(p.q);
  const IN* kg = reinterpret_cast<const IN*>(p.k);
  const IN* vg = reinterpret_cast<const IN*>(p.v);
  OT* og = reinterpret_cast<OT*>(p.o);
  const XT* matg = reinterpret_cast<const XT*>(p.mat_ws);
  XT* fblk = reinterpret_cast<XT*>(p.fwd_blk);   // CKPT: U, UR, r blocks

  // ---- staging of chunk c+1 while chunk c computes ----
  //   K, Q fragments: register prefetch (issued after P1, when chunk c's are dead)
  //   V block, gate block, T^R, MR: LDS-DMA after P1 (V, gates dead; T^R/MR
  //     double-buffered); T^S, MG, MP: LDS-DMA after P3 (their last use)
  // Completion: every wave waits for its vector memory operations and the
  // whole workgroup passes a barrier at the end of chunk c.
  typename MI::frag Kn[KS_STEPS], Qn[KS_STEPS];
  auto chunk_len = [&](int c) { return min(kChunk, si.len - c * kChunk); };
  auto mat_src = [&](int c, int m) {
    return matg + ((int64_t)(si.chunk0 + c) * H + h) * kNumMats * kMatElems + m * kMatElems;
  };
  const MatDma<XT> mdo;   // this lane's matrix DMA offsets
  auto issue_regs = [&](int c) {
    const int64_t tok = si.start + (int64_t)c * kChunk;
    const int t = 16 * w + (lane & 15);
    const int64_t roff = ((tok + t) * H + h) * (int64_t)DK;
    const bool ok = t < chunk_len(c);
    load_rowfrags<IN, DK>(Kn, ok ? kg + roff : nullptr);
    load_rowfrags<IN, DK>(Qn, ok ? qg + roff : nullptr);
  };
  auto issue_early = [&](int c) {   // V, gates, T^R, MR
    const int64_t tok = si.start + (int64_t)c * kChunk;
    const int len = chunk_len(c);
    {   // V block: wave w moves rows 16w..16w+15 (64 bytes each)
      constexpr int kChunksPerRow = BV * (int)sizeof(IN) / 16;
      const int P = w * 64 + lane, t = P / kChunksPerRow, cc = P % kChunksPerRow;
      const int ts = t < len ? t : len - 1;   // padding rows: any valid row (multiplied by 0)
      const IN* src = vg + ((tok + ts) * H + h) * (int64_t)DV + j0 + cc * (16 / (int)sizeof(IN));
      dma16(src, reinterpret_cast<char*>(Vc) + w * 1024);
    }
    if (w == 0)
      dma_linear_wave(p.gate_ws + ((int64_t)(si.chunk0 + c) * H + h) * kGateBlock, graw,
                      kGateBlock * 4);
    if constexpr (L::kDB) {
      if constexpr (RDN) dma_mat64<XT>(mat_src(c, kMatTR), mat(kMatTR, c & 1), mdo);
      dma_mat64<XT>(mat_src(c, kMatMR), mat(kMatMR, c & 1), mdo);
    }
  };
  auto issue_late = [&](int c) {    // T^S, MG, MP
    if constexpr (RDN) dma_mat64<XT>(mat_src(c, kMatTS), mat(kMatTS, 0), mdo);
    dma_mat64<XT>(mat_src(c, kMatMG), mat(kMatMG, 0), mdo);
    dma_mat64<XT>(mat_src(c, kMatMP), mat(kMatMP, 0), mdo);
  };
  auto issue_tail = [&](int c) {    // T^R, MR when single-buffered
    if constexpr (!L::kDB) {
      if constexpr (RDN) dma_mat64<XT>(mat_src(c, kMatTR), mat(kMatTR, 0), mdo);
      dma_mat64<XT>(mat_src(c, kMatMR), mat(kMatMR, 0), mdo);
    }
  };
  if (nch > 0) {
    issue_regs(0);
    issue_early(0);
    issue_late(0);
    issue_tail(0);
    wait_vmem();
  }
  barrier_lds();

  for (int c = 0; c < nch; ++c) {
    const int gc = si.chunk0 + c;
    const int64_t tok = si.start + (int64_t)c * kChunk;
    const int len = chunk_len(c);
    const int buf = c & 1;

    // ---- commit: K, Q fragments from the prefetch registers, K^T (XT) and
    //      the gate-derived vectors into LDS ----
    typename MI::frag Kf[KS_STEPS], Qf[KS_STEPS];
    typename MI::frag Klo[VAR ? KS_STEPS : 1], Qlo[VAR ? KS_STEPS : 1];   // fp16 rows: bf16 residuals
    {
      const int t = 16 * w + (lane & 15);
#pragma unroll
      for (int s2 = 0; s2 < KS_STEPS; ++s2) {
        Kf[s2] = Kn[s2];
        Qf[s2] = Qn[s2];
        if constexpr (BF) {   // row t, 8 columns: one 16-byte store
          const u16x8 kv = __builtin_bit_cast(u16x8, Kf[s2]);
          f16x8 kh;
          if constexpr (VAR) {
            if (qk16) {   // fp16 rows: K^T as is; hi + lo bf16 fragments for the state products
              kh = __builtin_bit_cast(f16x8, kv);
              const f16x8 qh = __builtin_bit_cast(f16x8, Qf[s2]);
              u16x8 khi, klo, qhi, qlo;
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                const float kx = (float)kh[e], qx = (float)qh[e];
                khi[e] = f2bf(kx);
                klo[e] = f2bf(kx - bf2f(khi[e]));
                qhi[e] = f2bf(qx);
                qlo[e] = f2bf(qx - bf2f(qhi[e]));
              }
              Kf[s2] = __builtin_bit_cast(typename MI::frag, khi);
              Klo[s2] = __builtin_bit_cast(typename MI::frag, klo);
              Qf[s2] = __builtin_bit_cast(typename MI::frag, qhi);
              Qlo[s2] = __builtin_bit_cast(typename MI::frag, qlo);
            } else {
#pragma unroll
              for (int e = 0; e < 8; ++e) kh[e] = (f16)bf2f(kv[e]);
            }
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) kh[e] = (f16)bf2f(kv[e]);
          }
          *reinterpret_cast<f16x8*>(TK::ptr(KT, t, s2 * 32 + (lane >> 4) * 8)) = kh;
        } else {
          *TT::ptr(KT, s2 * 4 + (lane >> 4), t) = Kf[s2];
        }
      }
      // gate vectors (lane = token), shared out over the four waves by a
      // wave-uniform index; the chunk-edge factors are stored by every lane
      // of their wave to one address
      const int tt = lane, wu = __builtin_amdgcn_readfirstlane(w);
      if (wu == 0) {
        egs[tt] = __expf(graw[tt]);
        egsp[tt] = tt > 0 ? __expf(graw[max(tt - 1, 0)]) : 1.f;
      } else if (wu == 1) {
        const float gr = graw[64 + tt], grl = graw[64 + kChunk - 1];
        egr[tt] = __expf(gr);
        dlr[tt] = __expf(grl - gr);
        edge[1] = __expf(grl);
      } else if (wu == 2) {
        const float gs = graw[tt], gsl = graw[kChunk - 1];
        dls[tt] = __expf(gsl - gs);
        edge[0] = __expf(gsl);
      } else {
        gbt[tt] = graw[128 + tt];
        ggm[tt] = graw[192 + tt];
        if constexpr (VAR) gout[tt] = (vf & kVarUngated) ? 1.f : graw[192 + tt];
      }
    }
    barrier_lds();

    // ---- P1: KS, QS, KR, QR for rows 16w..16w+15 ----
    floatx4 KS[JT], QS[JT], KR[JT], QR[JT];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      KS[jt] = zero4(); QS[jt] = zero4(); KR[jt] = zero4(); QR[jt] = zero4();
      typedef typename L::TSC TSC;
      mma_rega_tile<IN, DK, TSC>(KS[jt], Kf, Shi, jt * 16);
      mma_rega_tile<IN, DK, TSC>(QS[jt], Qf, Shi, jt * 16);
      mma_rega_tile<IN, DK, TSC>(KR[jt], Kf, Rhi, jt * 16);
      mma_rega_tile<IN, DK, TSC>(QR[jt], Qf, Rhi, jt * 16);
      if constexpr (BF) {
        mma_rega_tile<IN, DK, TSC>(KS[jt], Kf, Slo, jt * 16);
        mma_rega_tile<IN, DK, TSC>(QS[jt], Qf, Slo, jt * 16);
        mma_rega_tile<IN, DK, TSC>(KR[jt], Kf, Rlo, jt * 16);
        mma_rega_tile<IN, DK, TSC>(QR[jt], Qf, Rlo, jt * 16);
        if constexpr (VAR) {
          if (qk16) {
            mma_rega_tile<IN, DK, TSC>(KS[jt], Klo, Shi, jt * 16);
            mma_rega_tile<IN, DK, TSC>(QS[jt], Qlo, Shi, jt * 16);
            mma_rega_tile<IN, DK, TSC>(KR[jt], Klo, Rhi, jt * 16);
            mma_rega_tile<IN, DK, TSC>(QR[jt], Qlo, Rhi, jt * 16);
          }
        }
      }
    }
    float vloc[JT][4];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      floatx4 y;
      if constexpr (BF) {   // V at this lane's accumulator positions: one transpose read
        const u16x4 v4 = acc_tile_tr<PadRows<IN, BV, 0>>(Vc, 16 * w, jt * 16);
#pragma unroll
        for (int r = 0; r < 4; ++r) vloc[jt][r] = bf2f(v4[r]);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = 16 * w + acc_row(r);
        if constexpr (!BF) vloc[jt][r] = to_f<IN>(Vc[t * BV + jt * 16 + acc_col()]);
        y[r] = RDN ? gbt[t] * __builtin_fmaf(-egs[t], KS[jt][r], vloc[jt][r]) : gbt[t] * vloc[jt][r];
      }
      if constexpr (RDN) {
        store_acc_tile<TT>(Yt, jt * 16, 16 * w, y);
      } else {
        floatx4 du;
#pragma unroll
        for (int r = 0; r < 4; ++r) du[r] = dls[16 * w + acc_row(r)] * y[r];
        store_acc_tile<TT>(Ut, jt * 16, 16 * w, y);
        store_acc_tile<TT>(DUt, jt * 16, 16 * w, du);
      }
    }
    // matrix fragments are loaded ahead of the barriers that precede their
    // products (each matrix landed in an earlier chunk)
    MatFrags<XT> aTS, aMG, aMP;
    if constexpr (RDN) aTS = swz_rows_frags<XT>(mat(kMatTS, 0), 16 * w);
    else {
      aMG = swz_rows_frags<XT>(mat(kMatMG, 0), 16 * w);
      aMP = swz_rows_frags<XT>(mat(kMatMP, 0), 16 * w);
    }
    barrier_lds();
    if (c + 1 < nch) {
      issue_regs(c + 1);
      issue_early(c + 1);
    }

    if constexpr (RDN) {   // ---- P2: U = T^S Y ----
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        floatx4 u = zero4();
        mma_frags<XT>(u, aTS, Yt, jt * 16);
        floatx4 du;
#pragma unroll
        for (int r = 0; r < 4; ++r) du[r] = dls[16 * w + acc_row(r)] * u[r];
        store_acc_tile<TT>(Ut, jt * 16, 16 * w, u);
        store_acc_tile<TT>(DUt, jt * 16, 16 * w, du);
      }
      aMG = swz_rows_frags<XT>(mat(kMatMG, 0), 16 * w);
      aMP = swz_rows_frags<XT>(mat(kMatMP, 0), 16 * w);
      barrier_lds();
    }

    // ---- P3: residual, clip, base read-out ----
    // (explicit fmas: every instantiation, saving or not, rounds alike)
    floatx4 base[JT];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      floatx4 mgu = zero4(), mpu = zero4();
      mma_frags<XT>(mgu, aMG, Ut, jt * 16);
      mma_frags<XT>(mpu, aMP, Ut, jt * 16);
      floatx4 y, rv;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = 16 * w + acc_row(r);
        const float x = __builtin_fmaf(-ekp[t], KS[jt][r], vloc[jt][r]) - mgu[r];
        const float rr = tanh_resid ? resid_tanh(x, clip)
                                    : (clip < 0.f ? x : fminf(fmaxf(x, -clip), clip));
        rv[r] = rr;
        if constexpr (CKPT) Mst[t * BV + jt * 16 + acc_col()] = (clip < 0.f || fabsf(x) <= clip) ? 1 : 0;
        base[jt][r] = __builtin_fmaf(eqb[t], QS[jt][r], mpu[r]);
        y[r] = RDN ? ggm[t] * __builtin_fmaf(-egr[t], KR[jt][r], rr) : ggm[t] * rr;
      }
      if constexpr (RDN) {
        store_acc_tile<TT>(Yt, jt * 16, 16 * w, y);
      } else {
        floatx4 du;
#pragma unroll
        for (int r = 0; r < 4; ++r) du[r] = dlr[16 * w + acc_row(r)] * y[r];
        store_acc_tile<TT>(URt, jt * 16, 16 * w, y);
        store_acc_tile<TT>(DURt, jt * 16, 16 * w, du);
      }
      if constexpr (CKPT) store_acc_tile<TT>(Rst, jt * 16, 16 * w, rv);
    }
    MatFrags<XT> aTR, aMR;
    if constexpr (L::kDB) {   // double-buffered: landed in the previous chunk
      if constexpr (RDN) aTR = swz_rows_frags<XT>(mat(kMatTR, buf), 16 * w);
      else aMR = swz_rows_frags<XT>(mat(kMatMR, buf), 16 * w);
    }
    if constexpr (!L::kDB) wait_vmem();   // single-buffered T^R / MR of this chunk
    barrier_lds();
    if (c + 1 < nch) issue_late(c + 1);
    // chunk-start states for the gradient kernel, straight from the
    // accumulators (bf16 inputs: fp16 scaled per (16 rows, 32 columns)),
    // stored after the chunk's last prefetch.  With bf16 inputs the state
    // update's transpose reads wait for them along with the prefetched data;
    // fp32 inputs leave them in flight past the chunk's end.
    if constexpr (CKPT) {
      const int64_t off = ((int64_t)gc * H + h) * DK * DV + j0;
      if constexpr (BF) {   // blocked [DV / 32][DK][32]: each wave store is 1 KiB contiguous
        const int64_t ob = ((int64_t)gc * H + h) * DK * DV + (int64_t)j0 * DK;
        const int64_t so = ((int64_t)gc * H + h) * (DK / 16) * (DV / 32) + j0 / 32;
        save_state_f16<IT>(Sacc, reinterpret_cast<f16*>(p.ck_S) + ob, 32, p.ck_S_sc + so, DV / 32, w * (DK / 4));
        save_state_f16<IT>(Racc, reinterpret_cast<f16*>(p.ck_R) + ob, 32, p.ck_R_sc + so, DV / 32, w * (DK / 4));
      } else {
        save_state_f32<IT, JT>(Sacc, reinterpret_cast<float*>(p.ck_S) + off, DV, w * (DK / 4));
        save_state_f32<IT, JT>(Racc, reinterpret_cast<float*>(p.ck_R) + off, DV, w * (DK / 4));
      }
    }
    if constexpr (!L::kDB) {
      if constexpr (RDN) aTR = swz_rows_frags<XT>(mat(kMatTR, buf), 16 * w);
      else aMR = swz_rows_frags<XT>(mat(kMatMR, buf), 16 * w);
    }

    if constexpr (RDN) {   // ---- P4: UR = T^R YR ----
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        floatx4 u = zero4();
        mma_frags<XT>(u, aTR, Yt, jt * 16);
        floatx4 du;
#pragma unroll
        for (int r = 0; r < 4; ++r) du[r] = dlr[16 * w + acc_row(r)] * u[r];
        store_acc_tile<TT>(URt, jt * 16, 16 * w, u);
        store_acc_tile<TT>(DURt, jt * 16, 16 * w, du);
      }
      aMR = swz_rows_frags<XT>(mat(kMatMR, buf), 16 * w);
      barrier_lds();
    }

    // ---- P5: correction read-out; o staged, stored after the end barrier ----
    if constexpr (WRITE_O) {
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        floatx4 mru = zero4();
        mma_frags<XT>(mru, aMR, URt, jt * 16);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = 16 * w + acc_row(r);
          Ost[t * L::kLdO + jt * 16 + acc_col()] =
              __builtin_fmaf(gout[t], __builtin_fmaf(egr[t], QR[jt][r], mru[r]), base[jt][r]);
        }
      }
    }

    // ---- state update: S <- e^{g_C} S + K^T DU, R <- e^{h_C} R + K^T DUR ----
    // (bf16 inputs: the K^T fragments from transpose reads issued as inline
    // assembly, which leaves the next chunk's DMA and the checkpoint stores
    // in flight; the builtin would drain them first)
    const float eS = edge[0], eR = edge[1];
    if constexpr (BF) {
      typedef Mfma<XT> MX;
      constexpr int NF = IT * (kChunk / MX::kStep);
      int fr0[NF], fk0[NF];
#pragma unroll
      for (int n = 0; n < NF; ++n) {
        fr0[n] = w * (DK / 4) + (n / (kChunk / MX::kStep)) * 16;
        fk0[n] = (n % (kChunk / MX::kStep)) * MX::kStep;
      }
      typename MX::frag kt[NF];
      frags_tr_sync<TK, XT, NF>(KT, fr0, fk0, kt);
#pragma unroll
      for (int it = 0; it < IT; ++it)
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) {
          Sacc[it][jt] *= eS;
          Racc[it][jt] *= eR;
#pragma unroll
          for (int ks = 0; ks < kChunk / MX::kStep; ++ks) {
            const int n = it * (kChunk / MX::kStep) + ks;
            Sacc[it][jt] = MX::mma(kt[n], TT::template frag<MX>(DUt, jt * 16, ks * MX::kStep), Sacc[it][jt]);
            Racc[it][jt] = MX::mma(kt[n], TT::template frag<MX>(DURt, jt * 16, ks * MX::kStep), Racc[it][jt]);
          }
        }
    } else {
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const int i0 = w * (DK / 4) + it * 16;
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) {
          Sacc[it][jt] *= eS;
          Racc[it][jt] *= eR;
          mma_tiles<XT, kChunk, TK, TT>(Sacc[it][jt], KT, i0, DUt, jt * 16);
          mma_tiles<XT, kChunk, TK, TT>(Racc[it][jt], KT, i0, DURt, jt * 16);
        }
      }
    }
    // the next chunk's DMA data must have landed before anyone reads it; the
    // checkpoint stores, issued after the chunk's last DMA, may still be in
    // flight
    wait_vmem_but<CKPT ? kCkptStores : 0>();
    barrier_lds();
    if (c + 1 < nch) issue_tail(c + 1);   // single-buffered T^R / MR: waited at P3
    // ---- this chunk's staged outputs, in 16-byte stores (the buffers are
    //      next written after the coming chunk's first barrier) ----
    if constexpr (WRITE_O) {
      constexpr int kVE = 16 / (int)sizeof(OT);
      constexpr int kVPR = BV / kVE;
      static_assert((kChunk * kVPR) % kThreads == 0, "whole o vectors per thread");
#pragma unroll
      for (int u = 0; u < kChunk * kVPR / kThreads; ++u) {
        const int e = tid + u * kThreads, t = e / kVPR, v = e % kVPR;
        if (t < len) {
          OT* dst = og + ((tok + t) * H + h) * (int64_t)DV + j0 + v * kVE;
          const float* src = Ost + t * L::kLdO + v * kVE;
          if constexpr (sizeof(OT) == 4) {
            *reinterpret_cast<float4*>(dst) = *reinterpret_cast<const float4*>(src);
          } else {
            u16x8 ov;
#pragma unroll
            for (int k = 0; k < 8; ++k) ov[k] = f2bf(src[k]);
            *reinterpret_cast<u16x8*>(dst) = ov;
          }
        }
      }
    }
    if constexpr (CKPT) {
      {   // clip mask rows
        constexpr int kVPR = BV / 16;
        const int t = tid / kVPR, v = tid % kVPR;
        if (tid < kChunk * kVPR && t < len)
          *reinterpret_cast<uint4*>(p.ck_mask + ((tok + t) * H + h) * (int64_t)DV + j0 + v * 16) =
              *reinterpret_cast<const uint4*>(Mst + t * BV + v * 16);
      }
      // U, UR, r rows (value-major in LDS): rows past the end are zero
      constexpr int kVE = 16 / (int)sizeof(XT);
      constexpr int kVPR = BV / kVE;
      static_assert(kChunk * kVPR == kThreads, "one block vector per thread");
      const int t = lane, v = w;   // lanes read consecutive tokens: no bank conflicts
#pragma unroll
      for (int b = 0; b < 3; ++b) {
        const XT* srcb = b == 0 ? Ut : b == 1 ? URt : Rst;
        uint4 x;
        if constexpr (BF) {   // two transpose reads per 16-byte row piece
          x = keep_if(tile_token_vec8<TT>(srcb, v * kVE), t < len);
        } else {
          XT vals[kVE];
#pragma unroll
          for (int k = 0; k < kVE; ++k) vals[k] = t < len ? TT::at(srcb, v * kVE + k, t) : from_f<XT>(0.f);
          x = *reinterpret_cast<const uint4*>(vals);
        }
        *reinterpret_cast<uint4*>(fblk + blk_off(gc, h, H, b, DV) + (int64_t)t * DV + j0 + v * kVE) = x;
      }
    }
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

// ---------------------------------------------------------------------------
// Wave-specialised forward scan: bf16 inputs, d_k = 128, 32 value columns,
// the boxed operator (no variant flags).  Eight waves per workgroup in two
// groups of four that pass the same barriers in the same order:
//   chain waves (0-3): hold S and R (rows 32 w' .. 32 w' + 31) in their
//     accumulators and do every product of the chunk (the algebra of
//     fwd_scan_kernel), loading only their own K and Q rows and storing
//     nothing to HBM: o goes to LDS;
//   side waves (4-7): all other HBM traffic — the chunk-start checkpoints
//     (formed from the LDS state copies), the U, U^R, r blocks, the clip
//     mask and o, and the staging of the next chunk (LDS-DMA of V and the
//     matrices, the gate values) — so it overlaps the chain instead of
//     stalling it.
// Per chunk (phase: chain waves | side waves):
//   1: K^T commit; KS, KR, QS, QR;               | the previous chunk's o rows;
//      Y = diag(b)(V - e^g KS)                     DMA of the next chunk's V, MG,
//                                                   MP, T^R, MR; its gate values;
//                                                   S checkpoint
//   2: U = T^S Y; next K, Q rows                  | DMA of the next T^S
//   3: p, r = clip(V - p), mask, Y^R;             | R checkpoint; U rows
//      base = e^g QS + MP U
//   4: U^R = T^R Y^R                              | r rows, mask
//   5: S, R update; o = base + diag(gamma) c      | wait for the DMA; next gate
//      into free LDS; state copies                  vectors; U^R rows
// V, MG, MP, T^R and MR are double-buffered; T^S (read into registers
// before the first barrier) is refilled from phase 2.  The precision scheme
// and the arithmetic are those of fwd_scan_kernel, except that the split-
// state products sum the hi and lo terms per k-step and the checkpoints are
// formed from the bf16 hi + lo state copies (the fp32 state to ~16 bits)
// instead of the accumulators.
// ---------------------------------------------------------------------------
template <typename IN, int DK, int BV, bool RDN>
struct FwdWsLayout {
  typedef f16 XT;
  typedef Tile<XT, kChunk> TT;
  typedef TrTile<XT, DK> TK;
  typedef Tile<IN, DK> TSC;
  static constexpr int kNumSlots = RDN ? 9 : 6;
  static constexpr int kKT = 0;
  static constexpr int kCopies = kKT + kChunk * TK::kRowB;
  static constexpr int kCopyBytes = BV * TSC::kRowB;
  static constexpr int kMats = kCopies + 4 * kCopyBytes;
  static constexpr int kBufs = kMats + kNumSlots * kPkBytes;   // matrices as their ten lower blocks
  static constexpr int kBufBytes = BV * TT::kRowB;
  static constexpr int kVBytes = kChunk * BV * (int)sizeof(IN);
  static constexpr int kVc = kBufs + 5 * kBufBytes;   // two V blocks (chunk parity)
  static constexpr int kGateVec = 8 * kChunk;         // floats per chunk's gate vectors
  static constexpr int kGates = kVc + 2 * kVBytes;    // two sets (chunk parity)
  static constexpr int kRst = kGates + 2 * kGateVec * 4;
  static constexpr int kMst = kRst + kBufBytes;
  static constexpr int kGraw = kMst + kChunk * BV;      // the gate block (one side wave's DMA)
  static constexpr int kZero = kGraw + kGateBlock * 4;   // 16 zero bytes (blocks above the diagonal)
  // fp32 outputs: o of a chunk, column-major [BV][kOstLd] (the pad keeps the
  // side's 4-byte gathers of one token's 4 columns in distinct banks)
  static constexpr int kOstLd = kChunk + 4;
  static constexpr int kOst = kZero + 16;
  static constexpr int kBytes = kOst + BV * kOstLd * 4;
  static_assert(sizeof(IN) == 2 && DK == 128 && BV == 32, "bf16, d_k 128, 32 columns");
  static_assert(kVBytes == 4 * 1024, "V block = one DMA instruction per side wave");
  static_assert(kBytes <= 160 * 1024, "forward scan LDS");
  // RDN: T^S, then MG, MP, T^R, MR each double-buffered; RLA: MG, MP, MR
  __device__ static constexpr int slot(int mat, int buf) {
    if (RDN) {
      if (mat == kMatTS) return 0;
      if (mat == kMatMG) return 1 + buf;
      if (mat == kMatMP) return 3 + buf;
      if (mat == kMatTR) return 5 + buf;
      return 7 + buf;
    }
    if (mat == kMatMG) return buf;
    if (mat == kMatMP) return 2 + buf;
    return 4 + buf;
  }
};

template <typename IN, int DK, int BV, bool RDN, bool WRITE_O, bool CKPT, typename OT>
__global__ __launch_bounds__(2 * kThreads) void fwd_scan_ws_kernel(OpParams p) {
  typedef FwdWsLayout<IN, DK, BV, RDN> L;
  typedef typename L::XT XT;
  typedef Mfma<IN> MI;
  typedef typename L::TT TT;
  typedef typename L::TK TK;
  typedef typename L::TSC TSC;
  constexpr int JT = BV / 16;          // value tiles per block
  constexpr int IT = DK / 64;          // state row tiles per wave
  constexpr int KS_STEPS = DK / MI::kStep;
  extern __shared__ __align__(16) unsigned char smem[];
  XT* KT = reinterpret_cast<XT*>(smem + L::kKT);
  IN* Shi = reinterpret_cast<IN*>(smem + L::kCopies);
  IN* Rhi = reinterpret_cast<IN*>(smem + L::kCopies + 1 * L::kCopyBytes);
  IN* Slo = reinterpret_cast<IN*>(smem + L::kCopies + 2 * L::kCopyBytes);
  IN* Rlo = reinterpret_cast<IN*>(smem + L::kCopies + 3 * L::kCopyBytes);
  auto mat = [&](int m, int buf) {
    return reinterpret_cast<XT*>(smem + L::kMats + L::slot(m, buf) * kPkBytes);
  };
  const XT* zero16 = reinterpret_cast<const XT*>(smem + L::kZero);
  XT* Yt = reinterpret_cast<XT*>(smem + L::kBufs);               // Y, later YR
  XT* Ut = reinterpret_cast<XT*>(smem + L::kBufs + 1 * L::kBufBytes);
  XT* URt = reinterpret_cast<XT*>(smem + L::kBufs + 2 * L::kBufBytes);
  XT* DUt = reinterpret_cast<XT*>(smem + L::kBufs + 3 * L::kBufBytes);
  XT* DURt = reinterpret_cast<XT*>(smem + L::kBufs + 4 * L::kBufBytes);
  auto vblk = [&](int c) { return reinterpret_cast<IN*>(smem + L::kVc + (c & 1) * L::kVBytes); };
  float* gates = reinterpret_cast<float*>(smem + L::kGates);
  XT* Rst = reinterpret_cast<XT*>(smem + L::kRst);            // r (saving mode)
  uint8_t* Mst = reinterpret_cast<uint8_t*>(smem + L::kMst);  // clip mask (saving mode)
  float* graw = reinterpret_cast<float*>(smem + L::kGraw);     // prep's gate block

  const int H = p.H, DV = p.DV, tid = threadIdx.x, lane = tid & 63;
  const int wu = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool chain = wu < kWaves;      // wave-uniform role
  const int ww = wu & (kWaves - 1);    // index within the role's four waves
  // XCD-aware block mapping (as fwd_scan_kernel)
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

  const IN* qg = reinterpret_cast<const IN*>(p.q);
  const IN* kg = reinterpret_cast<const IN*>(p.k);
  const IN* vg = reinterpret_cast<const IN*>(p.v);
  OT* og = reinterpret_cast<OT*>(p.o);
  const XT* matg = reinterpret_cast<const XT*>(p.mat_ws);
  XT* fblk = reinterpret_cast<XT*>(p.fwd_blk);   // CKPT: U, UR, r blocks
  auto chunk_len = [&](int c) { return min(kChunk, si.len - c * kChunk); };
  auto mat_src = [&](int c, int m) {
    return matg + ((int64_t)(si.chunk0 + c) * H + h) * kNumMats * kMatElems + m * kMatElems;
  };
  // gate vectors of chunk c: beta, gamma, e^{g_t}, e^{g_{t-1}}, e^{h_t},
  // e^{g_C - g_t}, e^{h_C - h_t}, then [e^{g_C}, e^{h_C}]
  auto gvec = [&](int c, int k) { return gates + (c & 1) * L::kGateVec + k * kChunk; };

  // One loop body, instantiated once per role (std::true_type: chain
  // waves): both roles pass the same barriers in the same order by
  // construction, and each instance gets its own registers.
  auto run = [&](auto role) {
  constexpr bool CH = decltype(role)::value;
  floatx4 Sacc[IT][JT], Racc[IT][JT];  // chain: the states
  typename MI::frag Kn[KS_STEPS], Qn[KS_STEPS];   // chain: next chunk's K, Q rows 16 ww + (lane & 15)
  if constexpr (CH) {
#pragma unroll
    for (int it = 0; it < IT; ++it)
#pragma unroll
      for (int jt = 0; jt < JT; ++jt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = ww * (DK / 4) + it * 16 + acc_row(r), j = j0 + jt * 16 + acc_col();
          Sacc[it][jt][r] = p.S0 ? p.S0[state_off + (int64_t)i * DV + j] : 0.f;
          Racc[it][jt][r] = p.R0 ? p.R0[state_off + (int64_t)i * DV + j] : 0.f;
        }
  }
  auto write_state_copies = [&]() {
#pragma unroll
    for (int it = 0; it < IT; ++it)
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        store_state_copy<TSC>(Shi, Slo, jt * 16, ww * (DK / 4) + it * 16, Sacc[it][jt]);
        store_state_copy<TSC>(Rhi, Rlo, jt * 16, ww * (DK / 4) + it * 16, Racc[it][jt]);
      }
  };
  // Global addresses are a chunk's uniform base plus a 32-bit lane offset
  // that does not change from chunk to chunk, so the memory instructions take
  // a scalar base and the lane part is formed once.
  auto issue_rows = [&](typename MI::frag (&dst)[KS_STEPS], const IN* src, int c) {
    const int64_t tok = si.start + (int64_t)c * kChunk;
    const int t = 16 * ww + (lane & 15);
    const bool ok = t < chunk_len(c);
    const IN* base = src + (tok * H + h) * (int64_t)DK;
    const uint32_t o = (uint32_t)(t * H * DK + (lane >> 4) * 8);
#pragma unroll
    for (int s2 = 0; s2 < KS_STEPS; ++s2) {
      u16x8 v = {0, 0, 0, 0, 0, 0, 0, 0};
      if (ok) v = *reinterpret_cast<const u16x8*>(base + o + s2 * 32);
      dst[s2] = __builtin_bit_cast(typename MI::frag, v);
    }
  };
  // side wave 0 moves chunk c's gate block (g, h, beta, gamma) into LDS with
  // one DMA instruction and, after its wait, forms every gate vector
  auto issue_gates = [&](int c) {
    if (ww == 0) dma_linear_wave(p.gate_ws + ((int64_t)(si.chunk0 + c) * H + h) * kGateBlock, graw, kGateBlock * 4);
  };
  auto write_gates = [&](int c) {
    if (ww != 0) return;
    const int t = lane;
    const float g = graw[t], gp = graw[max(t - 1, 0)], gl = graw[kChunk - 1];
    const float hr = graw[64 + t], hl = graw[64 + kChunk - 1];
    gvec(c, 0)[t] = graw[128 + t];
    gvec(c, 1)[t] = graw[192 + t];
    gvec(c, 2)[t] = __expf(g);
    gvec(c, 3)[t] = t > 0 ? __expf(gp) : 1.f;
    gvec(c, 4)[t] = __expf(hr);
    gvec(c, 5)[t] = __expf(gl - g);
    gvec(c, 6)[t] = __expf(hl - hr);
    gvec(c, 7)[0] = __expf(gl);   // every lane stores the same value
    gvec(c, 7)[1] = __expf(hl);
  };
  // side waves: the five DMA instructions of the g-th matrix of a group are
  // dealt round-robin over the four side waves (the group's instruction k
  // to wave k mod 4)
  auto dma_mat = [&](int c, int m, int slot_buf, int g) {
    dma_mat_packed<false>(mat_src(c, m), mat(m, slot_buf), ((ww - 5 * g) % 4 + 4) % 4, kWaves);
  };
  auto issue_early = [&](int c) {   // V, MG, MP, T^R, MR of chunk c (double-buffered)
    const int64_t tok = si.start + (int64_t)c * kChunk;
    const int len = chunk_len(c);
    constexpr int kChunksPerRow = BV * (int)sizeof(IN) / 16;
    const int P = ww * 64 + lane, t = P / kChunksPerRow, cc = P % kChunksPerRow;
    const int ts = t < len ? t : len - 1;   // padding rows: any valid row (multiplied by 0)
    dma16(vg + (tok * H + h) * (int64_t)DV + j0 + (uint32_t)(ts * H * DV + cc * (16 / (int)sizeof(IN))),
          reinterpret_cast<char*>(vblk(c)) + ww * 1024);
    int g = 0;
    dma_mat(c, kMatMG, c & 1, g++);
    dma_mat(c, kMatMP, c & 1, g++);
    if constexpr (RDN) dma_mat(c, kMatTR, c & 1, g++);
    dma_mat(c, kMatMR, c & 1, g++);
  };
  auto issue_ts = [&](int c) {   // T^S (single-buffered)
    if constexpr (RDN) dma_mat(c, kMatTS, 0, 0);
  };
  // side waves: tokens 16 ww .. 16 ww + 15 of a token-major block, one
  // 64-byte segment per token (lane (g, i): token 16 ww + i, values 8 g ..
  // 8 g + 7); rows past the end are zero
  auto store_block = [&](int c, int b, const XT* src) {
    static_assert(BV == 32 && sizeof(XT) == 2, "four lanes per 32-value token row");
    const int64_t gc = si.chunk0 + c;
    const int t = 16 * ww + (lane & 15);
    const uint4 x = keep_if(tile_token_rows16_sync<TT>(src, 16 * ww), t < chunk_len(c));
    *reinterpret_cast<uint4*>(fblk + blk_off(gc, h, H, b, DV) + j0 + (uint32_t)(t * DV + 8 * (lane >> 4))) = x;
  };
  // side waves: chunk-start state X (st: 0 = S, 1 = R) from its copies
  // (hi + lo), rows 32 ww .. 32 ww + 31, fp16 blocked [DV / 32][DK][32] with
  // one power-of-two scale per 16-row tile.  Transpose reads of the copies
  // give lane (g, i) state row t0 + i at columns 8 g .. 8 g + 7, so one
  // 16-row tile is one 1 KiB store; the wave's two tile scales leave in one
  // store (lane l writes tile l's)
  auto store_ckpt = [&](int c, int st) {
    const int64_t gc = si.chunk0 + c;
    const IN* hi = st ? Rhi : Shi;
    const IN* lo = st ? Rlo : Slo;
    f16* dst = reinterpret_cast<f16*>(st ? p.ck_R : p.ck_S) + ((int64_t)gc * H + h) * DK * DV + (int64_t)j0 * DK;
    float sc[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int t0 = ww * (DK / 4) + 16 * it;
      const uint4 xh = tile_token_rows16_sync<TSC>(hi, t0), xl = tile_token_rows16_sync<TSC>(lo, t0);
      const uint32_t wh[4] = {xh.x, xh.y, xh.z, xh.w}, wl[4] = {xl.x, xl.y, xl.z, xl.w};
      floatx4 a, b;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float v0 = __uint_as_float(wh[e] << 16) + __uint_as_float(wl[e] << 16);
        const float v1 = __uint_as_float(wh[e] & 0xFFFF0000u) + __uint_as_float(wl[e] & 0xFFFF0000u);
        if (e < 2) { a[2 * e] = v0; a[2 * e + 1] = v1; } else { b[2 * e - 4] = v0; b[2 * e - 3] = v1; }
      }
      const int ex = pow2_scale_exp(wave_absmax_bits(lane_absmax_bits(a, b)));
      const float f = exp2_int(-ex);
      const uint4 v = {cvt_pk_f16(a[0] * f, a[1] * f), cvt_pk_f16(a[2] * f, a[3] * f),
                       cvt_pk_f16(b[0] * f, b[1] * f), cvt_pk_f16(b[2] * f, b[3] * f)};
      *reinterpret_cast<uint4*>(dst + (uint32_t)((t0 + (lane & 15)) * 32 + 8 * (lane >> 4))) = v;
      sc[it] = exp2_int(ex);
    }
    static_assert(IT == 2, "two tiles per wave");
    const int64_t so = ((int64_t)gc * H + h) * (DK / 16) * (DV / 32) + j0 / 32;
    if (lane < IT)   // one lane per tile scale
      (st ? p.ck_R_sc : p.ck_S_sc)[so + (int64_t)(ww * IT + lane) * (DV / 32)] = lane ? sc[1] : sc[0];
  };

  // KS, KR, QS, QR for this wave's 16 token rows (K, Q as A fragments)
  // from the state copies: each B fragment read once serves the K and the Q
  // product; eight independent MFMA chains (value tile x state x K/Q), each
  // adding the hi and the lo product of every k-step
  auto split_products = [&](const typename MI::frag (&kf)[KS_STEPS], const typename MI::frag (&qf)[KS_STEPS],
                            floatx4 (&ks)[JT], floatx4 (&kr)[JT], floatx4 (&qs)[JT], floatx4 (&qr)[JT]) {
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) ks[jt] = kr[jt] = qs[jt] = qr[jt] = zero4();
#pragma unroll
    for (int s2 = 0; s2 < KS_STEPS; ++s2)
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        const int k0 = s2 * MI::kStep;
        const typename MI::frag sh = TSC::template frag<MI>(Shi, jt * 16, k0);
        const typename MI::frag rh = TSC::template frag<MI>(Rhi, jt * 16, k0);
        const typename MI::frag sl = TSC::template frag<MI>(Slo, jt * 16, k0);
        const typename MI::frag rl = TSC::template frag<MI>(Rlo, jt * 16, k0);
        ks[jt] = MI::mma(kf[s2], sh, ks[jt]);
        qs[jt] = MI::mma(qf[s2], sh, qs[jt]);
        kr[jt] = MI::mma(kf[s2], rh, kr[jt]);
        qr[jt] = MI::mma(qf[s2], rh, qr[jt]);
        ks[jt] = MI::mma(kf[s2], sl, ks[jt]);
        qs[jt] = MI::mma(qf[s2], sl, qs[jt]);
        kr[jt] = MI::mma(kf[s2], rl, kr[jt]);
        qr[jt] = MI::mma(qf[s2], rl, qr[jt]);
      }
  };

  // o leaves through LDS regions that are free from phase 5 until the side
  // waves read them in the next chunk's phase 1: value tile 0 in chunk c's
  // V block, tile 1 in the r block; wave ww's 16 rows as 1 KiB at ww KiB,
  // row-major [16][16] in OT.  The side wave reads its slice of the V block
  // before its own DMA refills that slice.
  auto ostage = [&](int c, int jt) {
    return reinterpret_cast<char*>(jt ? reinterpret_cast<char*>(Rst) : reinterpret_cast<char*>(vblk(c))) + ww * 1024;
  };
  // fp32 o from the column-major stage: four 4-byte reads give a lane 4
  // columns of one token
  float* ost = reinterpret_cast<float*>(smem + L::kOst);
  auto store_o = [&](int c) {   // side waves: chunk c's o rows 16 ww .. 16 ww + 15
    constexpr int kVE = 16 / (int)sizeof(OT);   // elements per 16 bytes
    const int64_t tok = si.start + (int64_t)c * kChunk;
    const int len = chunk_len(c);
    const int t = 16 * ww + lane / (16 / kVE), col = (lane % (16 / kVE)) * kVE;
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      const uint4 v = sizeof(OT) == 4 ? lds_read4x1_sync(ost + (jt * 16 + col) * L::kOstLd + t, L::kOstLd * 4)
                                      : lds_read16_sync(ostage(c, jt) + (lane % (16 * 16 / kVE)) * 16);
      if (lane < 16 * 16 / kVE && t < len)
        *reinterpret_cast<uint4*>(og + (tok * H + h) * (int64_t)DV + j0 + jt * 16 + (uint32_t)(t * H * DV + col)) = v;
    }
  };

  // ---- prologue: chunk 0's staging and the initial state copies ----
  if (threadIdx.x == 0) *reinterpret_cast<uint4*>(smem + L::kZero) = uint4{0, 0, 0, 0};
  if (nch > 0) {
    if constexpr (CH) {
      issue_rows(Kn, kg, 0);
      issue_rows(Qn, qg, 0);
    } else {
      issue_gates(0);
      issue_early(0);
      issue_ts(0);
      wait_vmem();
      write_gates(0);
    }
  }
  if constexpr (CH) write_state_copies();
  barrier_lds();

  floatx4 KS[JT], KR[JT], QS[JT], QR[JT], base[JT];
  float vloc[JT][4];
  MatFrags<XT> aTS, aMG, aMP, aTR, aMR;
  for (int c = 0; c < nch; ++c) {
    const int len = chunk_len(c);
    const int buf = c & 1;
    const bool more = c + 1 < nch;
    const float* gbt = gvec(c, 0);
    const float* ggm = gvec(c, 1);
    const float* egs = gvec(c, 2);
    const float* egsp = gvec(c, 3);
    const float* egr = gvec(c, 4);
    const float* dls = gvec(c, 5);
    const float* dlr = gvec(c, 6);
    const float* edge = gvec(c, 7);
    const int64_t tok = si.start + (int64_t)c * kChunk;

    // ======== phase 1 ========
    if constexpr (CH) {
      typename MI::frag Kf[KS_STEPS], Qf[KS_STEPS];
      const int t = 16 * ww + (lane & 15);
#pragma unroll
      for (int s2 = 0; s2 < KS_STEPS; ++s2) {   // K^T commit: row t, 8 columns per store
        Kf[s2] = Kn[s2];
        Qf[s2] = Qn[s2];
        const u16x8 kv = __builtin_bit_cast(u16x8, Kf[s2]);
        f16x8 kh;
#pragma unroll
        for (int e = 0; e < 8; ++e) kh[e] = (f16)bf2f(kv[e]);
        *reinterpret_cast<f16x8*>(TK::ptr(KT, t, s2 * 32 + (lane >> 4) * 8)) = kh;
      }
      split_products(Kf, Qf, KS, KR, QS, QR);
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        const u16x4 v4 = acc_tile_tr<PadRows<IN, BV, 0>>(vblk(c), 16 * ww, jt * 16);
        floatx4 y;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int tr = 16 * ww + acc_row(r);
          vloc[jt][r] = bf2f(v4[r]);
          y[r] = RDN ? gbt[tr] * __builtin_fmaf(-egs[tr], KS[jt][r], vloc[jt][r]) : gbt[tr] * vloc[jt][r];
        }
        if constexpr (RDN) {
          store_acc_tile<TT>(Yt, jt * 16, 16 * ww, y);
        } else {
          floatx4 du;
#pragma unroll
          for (int r = 0; r < 4; ++r) du[r] = dls[16 * ww + acc_row(r)] * y[r];
          store_acc_tile<TT>(Ut, jt * 16, 16 * ww, y);
          store_acc_tile<TT>(DUt, jt * 16, 16 * ww, du);
        }
      }
      if constexpr (RDN) aTS = packed_rows_frags(mat(kMatTS, 0), ww, zero16);
      else aMG = packed_rows_frags(mat(kMatMG, buf), ww, zero16);
    } else {
      if constexpr (WRITE_O) {
        if (c > 0) store_o(c - 1);   // before the DMA below refills chunk c - 1's V block
      }
      if (more) {
        issue_early(c + 1);
        issue_gates(c + 1);
      }
      if constexpr (CKPT) store_ckpt(c, 0);   // chunk-start S
    }
    barrier_lds();

    // ======== phase 2 ========
    if constexpr (CH) {
      if constexpr (RDN) {   // U = T^S Y
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) {
          floatx4 u = zero4();
          mma_frags<XT>(u, aTS, Yt, jt * 16);
          floatx4 du;
#pragma unroll
          for (int r = 0; r < 4; ++r) du[r] = dls[16 * ww + acc_row(r)] * u[r];
          store_acc_tile<TT>(Ut, jt * 16, 16 * ww, u);
          store_acc_tile<TT>(DUt, jt * 16, 16 * ww, du);
        }
        aMG = packed_rows_frags(mat(kMatMG, buf), ww, zero16);
      }
      if constexpr (WRITE_O) aMP = packed_rows_frags(mat(kMatMP, buf), ww, zero16);
      if (more) {   // the next K, Q rows, while the side waves issue little
        issue_rows(Kn, kg, c + 1);
        issue_rows(Qn, qg, c + 1);
      }
    } else {
      if (more) issue_ts(c + 1);   // T^S was read into registers before the first barrier
    }
    barrier_lds();

    // ======== phase 3 ========
    if constexpr (CH) {   // residual, clip, Y^R (explicit fmas as fwd_scan_kernel)
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        floatx4 mgu = zero4();
        mma_frags<XT>(mgu, aMG, Ut, jt * 16);
        floatx4 y, rv;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = 16 * ww + acc_row(r);
          const float x = __builtin_fmaf(-egsp[t], KS[jt][r], vloc[jt][r]) - mgu[r];
          const float rr = clip < 0.f ? x : fminf(fmaxf(x, -clip), clip);
          rv[r] = rr;
          if constexpr (CKPT) Mst[t * BV + jt * 16 + acc_col()] = (clip < 0.f || fabsf(x) <= clip) ? 1 : 0;
          y[r] = RDN ? ggm[t] * __builtin_fmaf(-egr[t], KR[jt][r], rr) : ggm[t] * rr;
        }
        if constexpr (RDN) {
          store_acc_tile<TT>(Yt, jt * 16, 16 * ww, y);
        } else {
          floatx4 du;
#pragma unroll
          for (int r = 0; r < 4; ++r) du[r] = dlr[16 * ww + acc_row(r)] * y[r];
          store_acc_tile<TT>(URt, jt * 16, 16 * ww, y);
          store_acc_tile<TT>(DURt, jt * 16, 16 * ww, du);
        }
        if constexpr (CKPT) store_acc_tile<TT>(Rst, jt * 16, 16 * ww, rv);
      }
      if constexpr (WRITE_O) {   // base = e^g QS + MP U
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) {
          floatx4 mpu = zero4();
          mma_frags<XT>(mpu, aMP, Ut, jt * 16);
#pragma unroll
          for (int r = 0; r < 4; ++r) base[jt][r] = __builtin_fmaf(egs[16 * ww + acc_row(r)], QS[jt][r], mpu[r]);
        }
      }
      if constexpr (RDN) aTR = packed_rows_frags(mat(kMatTR, buf), ww, zero16);
    } else {
      if constexpr (CKPT) store_ckpt(c, 1);   // chunk-start R
      if constexpr (CKPT) store_block(c, 0, Ut);
    }
    barrier_lds();

    // ======== phase 4 ========
    if constexpr (CH) {
      if constexpr (RDN) {   // U^R = T^R Y^R
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) {
          floatx4 u = zero4();
          mma_frags<XT>(u, aTR, Yt, jt * 16);
          floatx4 du;
#pragma unroll
          for (int r = 0; r < 4; ++r) du[r] = dlr[16 * ww + acc_row(r)] * u[r];
          store_acc_tile<TT>(URt, jt * 16, 16 * ww, u);
          store_acc_tile<TT>(DURt, jt * 16, 16 * ww, du);
        }
      }
      if constexpr (WRITE_O) aMR = packed_rows_frags(mat(kMatMR, buf), ww, zero16);
    } else {
      if constexpr (CKPT) {
        store_block(c, 2, Rst);
        {   // clip mask rows (side waves 0 and 1, one 16-byte piece per lane);
            // past the end, a lane rewrites the last row's own bytes, so the
            // store needs no lane condition
          constexpr int kVPR = BV / 16;
          const int e = (ww & 1) * 64 + lane, t = min(e / kVPR, len - 1), v = e % kVPR;
          if (ww < 2)
            *reinterpret_cast<uint4*>(p.ck_mask + (tok * H + h) * (int64_t)DV + j0 + (uint32_t)(t * H * DV + v * 16)) =
                lds_read16_sync(Mst + t * BV + v * 16);
        }
      }
    }
    barrier_lds();

    // ======== phase 5 ========
    if constexpr (CH) {   // S <- e^{g_C} S + K^T DU, R <- e^{h_C} R + K^T DUR
      const float eS = edge[0], eR = edge[1];
      typedef Mfma<XT> MX;
      constexpr int NF = IT * (kChunk / MX::kStep);
      int fr0[NF], fk0[NF];
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        fr0[f] = ww * (DK / 4) + (f / (kChunk / MX::kStep)) * 16;
        fk0[f] = (f % (kChunk / MX::kStep)) * MX::kStep;
      }
      typename MX::frag kt[NF];
      frags_tr_sync<TK, XT, NF>(KT, fr0, fk0, kt);
#pragma unroll
      for (int it = 0; it < IT; ++it)
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) {
          Sacc[it][jt] *= eS;
          Racc[it][jt] *= eR;
#pragma unroll
          for (int ks = 0; ks < kChunk / MX::kStep; ++ks) {
            const int f = it * (kChunk / MX::kStep) + ks;
            Sacc[it][jt] = MX::mma(kt[f], TT::template frag<MX>(DUt, jt * 16, ks * MX::kStep), Sacc[it][jt]);
            Racc[it][jt] = MX::mma(kt[f], TT::template frag<MX>(DURt, jt * 16, ks * MX::kStep), Racc[it][jt]);
          }
        }
      if constexpr (WRITE_O) {   // o = base + diag(gamma) (e^h QR + MR UR), this wave's rows
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) {
          floatx4 mru = zero4(), ov;
          mma_frags<XT>(mru, aMR, URt, jt * 16);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int t = 16 * ww + acc_row(r);
            ov[r] = __builtin_fmaf(ggm[t], __builtin_fmaf(egr[t], QR[jt][r], mru[r]), base[jt][r]);
          }
          if constexpr (sizeof(OT) == 4) {   // this lane's 4 tokens of its column, one store
            *reinterpret_cast<floatx4*>(ost + (jt * 16 + acc_col()) * L::kOstLd + 16 * ww + acc_row(0)) = ov;
          } else {
            // quad transpose: this lane's row 4 (lane / 16) + lane % 4, columns
            // 4 ((lane % 16) / 4) .. + 3 of the wave's 16 x 16 tile
            const floatx4 x = quad_transpose(ov);
            const int row = 4 * (lane >> 4) + (lane & 3), col = 4 * ((lane & 15) >> 2);
            char* dst = ostage(c, jt) + (row * 16 + col) * (int)sizeof(OT);
            u16x4 b;
#pragma unroll
            for (int k = 0; k < 4; ++k) b[k] = f2bf(x[k]);
            *reinterpret_cast<u16x4*>(dst) = b;
          }
        }
      }
      write_state_copies();
    } else {
      // the next chunk's DMA (and this wave's earlier stores) complete; the
      // barrier below publishes the DMA data
      wait_vmem();
      if (more) write_gates(c + 1);
      if constexpr (CKPT) store_block(c, 1, URt);
    }
    barrier_lds();
  }

  if constexpr (!CH && WRITE_O) {
    if (nch > 0) store_o(nch - 1);
  }
  if constexpr (CH) {
    if (p.S_fin || p.R_fin) {
#pragma unroll
      for (int it = 0; it < IT; ++it)
#pragma unroll
        for (int jt = 0; jt < JT; ++jt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int i = ww * (DK / 4) + it * 16 + acc_row(r), j = j0 + jt * 16 + acc_col();
            if (p.S_fin) p.S_fin[state_off + (int64_t)i * DV + j] = Sacc[it][jt][r];
            if (p.R_fin) p.R_fin[state_off + (int64_t)i * DV + j] = Racc[it][jt][r];
          }
    }
  }
  };
  if (chain) run(std::true_type{});
  else run(std::false_type{});
}

template <typename IN, int DK, int BV, bool RDN, bool WRITE_O, bool CKPT, typename OT>
hipError_t launch_fwd_t(const OpParams& p, hipStream_t stream) {
  typedef FwdLayout<IN, DK, BV, RDN> L;
  const bool var = (p.vflags & kVarOperator) || p.qk_f16;
  auto kern = var ? fwd_scan_kernel<IN, DK, BV, RDN, WRITE_O, CKPT, OT, true>
                  : fwd_scan_kernel<IN, DK, BV, RDN, WRITE_O, CKPT, OT, false>;
  int threads = kThreads, lds = L::kBytes;
  if constexpr (sizeof(IN) == 2 && DK == 128 && BV == 32) {
    if (!var) {   // the boxed operator: the wave-specialised scan
      kern = fwd_scan_ws_kernel<IN, DK, BV, RDN, WRITE_O, CKPT, OT>;
      threads = 2 * kThreads;
      lds = FwdWsLayout<IN, DK, BV, RDN>::kBytes;
    }
  }
  hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (err != hipSuccess) return err;
  const int nvb = p.DV / BV;
  const int npairs = p.st.nseq * p.H;
  const int grid = ((npairs + 7) / 8) * 8 * nvb;
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(threads), lds, stream, p);
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
