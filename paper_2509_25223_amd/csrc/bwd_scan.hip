// Reverse state-gradient scan: one 256-thread workgroup per (sequence, head,
// value block), walking the chunks from last to first with dS, dR (d_k x BV,
// fp32) in MFMA accumulators.  It produces, for every chunk, the gradient of
// the loss with respect to the chunk-END states (consumed by the chunk-
// parallel gradient kernel) and, at the sequence start, dS0 and dR0.
//
// Adjoint of one forward chunk (see fwd_scan.hip for the forward), with
// db = dO, dc = diag(gamma) dO and the clip mask m from the forward pass:
//   dUR = diag(e^{h_C-h}) K dR_end + MR^T dc
//   RDN: dYR = T^R^T dUR            RLA: dYR = dUR
//   dX  = m * (diag(gamma) dYR)     (dr = gamma dYR, then the clip's mask)
//   dKR = -diag(gamma e^{h}) dYR    (RDN only: UR depends on R0 through KR)
//   dU  = diag(e^{g_C-g}) K dS_end + MP^T db - MG^T dX
//   RDN: dY = T^S^T dU              RLA: not needed (U = diag(b) V)
//   dKS = -diag(e^{g_{t-1}}) dX - diag(b e^{g}) dY      (RLA: first term only)
//   dS_start = e^{g_C} dS_end + Q^T diag(e^{g}) db + K^T dKS
//   dR_start = e^{h_C} dR_end + Q^T diag(e^{h}) dc + K^T dKR
// Also written per chunk: dv = dX + diag(b) dY (RLA: dX + diag(b) dU), and
// the blocks dX, dY (RLA: dU), dYR (RLA: dUR) for the gradient kernel.
// Variants: ungated output db = e^{g_{t-1}}-weighted (the S_{t-1} q read-out)
// and dc = dO; decayed residual dKS with e^{g} in place of e^{g_{t-1}};
// log-cosh residual dX = (1 - (r / c)^2) gamma dYR, r read from the forward's
// saved block instead of the clip mask.
// Every column of dS, dR only sees its own value column, so value blocks are
// independent here as in the forward.  Operand precision (bf16 inputs): K x
// (dS, dR) takes fp16 K times one fp16 copy of each gradient state scaled by
// a power of two per chunk; all other products use fp16 operands (fp32 for
// fp32 inputs).  The upstream gradients dO, dS_T, dR_T of each (sequence,
// head) enter multiplied by the power of two 2^e that brings their largest
// magnitude into [4, 8) (from the per-chunk maxima of grad_scale.hip), so the
// fp16 operands derived from them keep fp16's range for any loss scale; dv,
// dS0 and dR0 are multiplied by 2^-e when written, and 2^e is left in
// grad_scale for the gradient kernel, which reads the scaled blocks and
// checkpoints.
#include <type_traits>

#include "kernels.hpp"

namespace rla {

namespace {

template <typename IN, int DK, int BV, bool RDN, bool VAR>
struct BwdScanLayout {
  static constexpr bool kBF = sizeof(IN) == 2;
  typedef typename std::conditional<kBF, f16, float>::type XT;
  // LDS buffers as padded rows (measured faster here than the swizzled
  // tiles, whose element-wise addressing costs this kernel registers):
  typedef PadRows<XT, kChunk, kBF ? 8 : 4> TT;    // per-token blocks [BV][64]
  // K, Q for the state-gradient update's K^T, Q^T operands: bf16 inputs keep
  // them row-major [64][DK] (16-byte stores at the commit, transpose reads at
  // the update); fp32 inputs store K^T, Q^T [DK][64]
  typedef typename std::conditional<kBF, TrTile<XT, DK>, PadRows<XT, kChunk, 4>>::type TKQ;
  // gradient-state copies [BV][DK] in the operand type: bf16 inputs keep one
  // fp16 copy of each state scaled by a power of two per chunk
  typedef PadRows<XT, DK, kBF ? 8 : 4> TSC;
  // matrix slots (swizzled tiles filled by LDS-DMA); with bf16 inputs MR
  // (first used) is double-buffered
  static constexpr bool kDB = kBF;
  static constexpr int kNumSlots = RDN ? (kDB ? 6 : 5) : (kDB ? 4 : 3);
  static constexpr int kNumCopies = 2;
  static constexpr int kNumBufs = 6;
  static constexpr int kKT = 0;
  static constexpr int kKQBytes = kBF ? kChunk * TKQ::kRowB : DK * TKQ::kRowB;
  static constexpr int kQT = kKT + kKQBytes;
  static constexpr int kCopies = kQT + kKQBytes;
  static constexpr int kCopyBytes = BV * TSC::kRowB;
  static constexpr int kMats = kCopies + kNumCopies * kCopyBytes;
  static constexpr int kBufs = kMats + kNumSlots * Swz<XT>::kBytes;
  static constexpr int kBufBytes = BV * TT::kRowB;
  static constexpr int kMask = kBufs + kNumBufs * kBufBytes;
  // the clip mask (BV bytes per token) or, in the variant instance (log-cosh
  // residual), the forward's r block (BV operand-type values per token)
  static constexpr int kMaskBytes = kChunk * BV * (VAR ? (int)sizeof(XT) : 1);
  static constexpr int kGraw = kMask + kMaskBytes;
  static constexpr int kGates = kGraw + kGateBlock * 4;
  static constexpr int kYst = kGates + 10 * kChunk * 4;   // dYR staging (token tile)
  static constexpr int kRed = kYst + kBufBytes;   // per-wave state maxima [2][4]
  static constexpr int kBytes = kRed + 8 * 4;
  static_assert(kMaskBytes % 1024 == 0, "mask block moved in whole DMA instructions");
  static_assert(kBytes <= 160 * 1024, "backward scan LDS");
  // RDN: TS MG MP TR MR[2]; RLA: MG MP MR[2]
  __device__ static constexpr int slot(int mat, int buf) {
    if (!RDN) {
      if (mat == kMatMG) return 0;
      if (mat == kMatMP) return 1;
      return kDB ? 2 + buf : 2;   // MR
    }
    if (mat == kMatTS) return 0;
    if (mat == kMatMG) return 1;
    if (mat == kMatMP) return 2;
    if (mat == kMatTR) return 3;
    return kDB ? 4 + buf : 4;   // MR
  }
};

// per-token block slots ([BV][64], value-major); aliases follow lifetimes:
// db is last read in P4 and dKS first written in P5; dc is last read in P2
// and dX first written in P3; dUR is last read in P3 and dU first written in
// P4.  RLA keeps dKS in the dKR slot (dKR = 0 there).
enum { bDB_DKS = 0, bDC_DX = 1, bQDB = 2, bQDC = 3, bDUR_DU = 4, bDKR = 5 };

// Writes this lane's 4 accumulator rows of a gradient-state tile into the
// transposed copy (tile rows r0 + column, columns c0 + row) in the operand
// type: 4 consecutive elements, one 8-byte (fp16) or 16-byte (fp32) store.
template <class TL, typename T>
__device__ __forceinline__ void store_state_copy(T* dst, int r0, int c0, floatx4 v) {
  // r0, c0 multiples of 16
  const int o = TL::off_split(r0, acc_col(), acc_row(0) * (int)sizeof(T), c0 * (int)sizeof(T));
  if constexpr (sizeof(T) == 2) {
    f16x4 x;
#pragma unroll
    for (int k = 0; k < 4; ++k) x[k] = (f16)v[k];
    *reinterpret_cast<f16x4*>(reinterpret_cast<char*>(dst) + o) = x;
  } else {
    *reinterpret_cast<floatx4*>(reinterpret_cast<char*>(dst) + o) = v;
  }
}

// VAR: an instance that reads the variant flags and qk_f16 (the default
// instance compiles them away)
template <typename IN, int DK, int BV, bool RDN, bool VAR>
__global__ __launch_bounds__(kThreads) void bwd_scan_kernel(OpParams p) {
  typedef BwdScanLayout<IN, DK, BV, RDN, VAR> L;
  typedef typename L::XT XT;
  typedef Mfma<IN> MI;
  typedef typename L::TT TT;
  typedef typename L::TKQ TKQ;
  typedef typename L::TSC TSC;
  constexpr bool BF = L::kBF;
  constexpr int JT = BV / 16;
  constexpr int IT = DK / 64;
  constexpr int KS_STEPS = DK / MI::kStep;
  // store instructions per wave of the two checkpointed gradient states
  // (save_state_f16: one row store and one scale store per 16-row tile;
  // fp32: one per row)
  constexpr int kCkptStores = 2 * (BF ? 2 * IT : 4 * IT * JT);
  extern __shared__ __align__(16) unsigned char smem_[];
  // LDS base, made opaque to the optimiser once per chunk (set_ptrs): the
  // per-lane addresses of every tile are then formed inside the loop from a
  // few per-lane offsets rather than each kept live across it
  unsigned char* smem = smem_;
  XT *KT, *QT, *Yst;
  XT *dSc, *dRc;
  uint32_t* smax;
  uint8_t* mask;
  float *graw, *gbt, *ggm, *egs, *egsp, *egr, *dls, *dlr, *edge, *gout;
  const float *ekp, *eqb;
  const int vf = VAR ? p.vflags : 0;
  auto set_ptrs = [&](bool opaque) {
    __attribute__((address_space(3))) unsigned char* s3 = (__attribute__((address_space(3))) unsigned char*)smem_;
    if (opaque) asm volatile("" : "+v"(s3));
    smem = (unsigned char*)s3;
    KT = reinterpret_cast<XT*>(smem + L::kKT);
    QT = reinterpret_cast<XT*>(smem + L::kQT);
    dSc = reinterpret_cast<XT*>(smem + L::kCopies);
    dRc = reinterpret_cast<XT*>(smem + L::kCopies + L::kCopyBytes);
    smax = reinterpret_cast<uint32_t*>(smem + L::kRed);
    mask = reinterpret_cast<uint8_t*>(smem + L::kMask);
    graw = reinterpret_cast<float*>(smem + L::kGraw);
    gbt = reinterpret_cast<float*>(smem + L::kGates);
    ggm = gbt + kChunk;
    egs = ggm + kChunk;
    egsp = egs + kChunk;
    egr = egsp + kChunk;
    dls = egr + kChunk;
    dlr = dls + kChunk;
    edge = dlr + kChunk;
    // output weight of c: gamma (ungated: 1); the default instance reads gamma
    gout = VAR ? edge + kChunk : ggm;
    ekp = (vf & kVarDecayed) ? egs : egsp;   // S0 factor of the residual
    eqb = (vf & kVarUngated) ? egsp : egs;   // S0 factor of the base read-out
    Yst = reinterpret_cast<XT*>(smem + L::kYst);   // dYR of this chunk
  };
  set_ptrs(false);
  auto mat = [&](int m, int buf) {
    return reinterpret_cast<XT*>(smem + L::kMats + L::slot(m, buf) * Swz<XT>::kBytes);
  };
  auto blk = [&](int b) { return reinterpret_cast<XT*>(smem + L::kBufs + b * L::kBufBytes); };
  const bool tanh_resid = (vf & kVarTanh) != 0;
  // log-cosh slope 1 - (r / c)^2 = s0 (1 - (r invc)^2): c = inf -> 1, c = 0 -> 0
  const float invc = p.clip > 0.f ? 1.f / p.clip : 0.f;
  const float s0 = p.clip == 0.f ? 0.f : 1.f;

  const int H = p.H, DV = p.DV, tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  // transposed matrix fragments, loaded ahead of the barrier before their
  // products (16-bit: transpose reads)
  auto cols_frags = [&](const XT* m) {
    if constexpr (BF) return swz_cols_frags_sync<XT>(m, 16 * w);
    else return swz_cols_frags<XT>(m, 16 * w);
  };
  const int nvb = DV / BV;
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int pair = (slot / nvb) * 8 + xcd, vb = slot % nvb;
  if (pair >= p.st.nseq * H) return;
  const int n = seq_order(p.st, pair / H), h = pair % H;
  const SeqInfo si = seq_info(p.st, n);
  const int nch = (si.len + kChunk - 1) / kChunk;
  const int j0 = vb * BV;
  const int64_t state_off = ((int64_t)n * H + h) * DK * DV;

  // scale of the upstream gradients of this (sequence, head): the largest of
  // the per-chunk maxima, brought into [4, 8) by sig = 2^e (1 if all are zero)
  float sig = 1.f, isig = 1.f;
  if (p.grad_absmax) {
    uint32_t m = 0;
    for (int c = tid; c < nch; c += kThreads)
      m = max(m, p.grad_absmax[(int64_t)(si.chunk0 + c) * H + h]);
    m = wave_absmax_bits(m);
    smax[w] = m;   // every lane stores the wave-uniform value
    barrier_lds();
    m = max(max(smax[0], smax[1]), max(smax[2], smax[3]));
    barrier_lds();
    const int be = (int)(m >> 23);
    const int e = be == 0 ? 0 : min(max(129 - be, -126), 126);
    sig = exp2_int(e);
    isig = exp2_int(-e);
    if (vb == 0 && tid == 0) p.grad_scale[(int64_t)n * H + h] = sig;
  }

  floatx4 dS[IT][JT], dR[IT][JT];
#pragma unroll
  for (int it = 0; it < IT; ++it)
#pragma unroll
    for (int jt = 0; jt < JT; ++jt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = w * (DK / 4) + it * 16 + acc_row(r), j = j0 + jt * 16 + acc_col();
        dS[it][jt][r] = p.dS_fin ? p.dS_fin[state_off + (int64_t)i * DV + j] * sig : 0.f;
        dR[it][jt][r] = p.dR_fin ? p.dR_fin[state_off + (int64_t)i * DV + j] * sig : 0.f;
      }
  // Copies of the gradient states for the next chunk's K dS, K dR products.
  // bf16 inputs: fp16, scaled by 2^-e with e from the largest magnitude of
  // each whole state (the waves' maxima meet in LDS across a barrier); the
  // products are multiplied back by 2^e (exact).  fp32 inputs: plain copies.
  float scS = 1.f, scR = 1.f;
  // largest magnitude of each of this wave's 16-row checkpoint tiles of the
  // current dS, dR (wave-uniform), kept for the next chunk's checkpoint
  // stores, which save these same values
  uint32_t tmS[IT], tmR[IT];
  auto publish_state_max = [&]() {
    if constexpr (BF) {
      state_tile_absmax<IT>(dS, tmS);
      state_tile_absmax<IT>(dR, tmR);
      uint32_t ms = tmS[0], mr = tmR[0];
#pragma unroll
      for (int it = 1; it < IT; ++it) {
        ms = max(ms, tmS[it]);
        mr = max(mr, tmR[it]);
      }
      smax[w] = ms;   // every lane stores the wave-uniform value
      smax[4 + w] = mr;
    }
  };
  auto write_copies = [&]() {   // after a barrier that follows publish_state_max
    float iS = 1.f, iR = 1.f;
    if constexpr (BF) {
      const uint32_t ms = max(max(smax[0], smax[1]), max(smax[2], smax[3]));
      const uint32_t mr = max(max(smax[4], smax[5]), max(smax[6], smax[7]));
      const int es = pow2_scale_exp(ms), er = pow2_scale_exp(mr);
      scS = exp2_int(es);
      scR = exp2_int(er);
      iS = exp2_int(-es);
      iR = exp2_int(-er);
    }
#pragma unroll
    for (int it = 0; it < IT; ++it)
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        store_state_copy<TSC>(dSc, jt * 16, w * (DK / 4) + it * 16, dS[it][jt] * iS);
        store_state_copy<TSC>(dRc, jt * 16, w * (DK / 4) + it * 16, dR[it][jt] * iR);
      }
  };
  publish_state_max();
  barrier_lds();
  write_copies();

  const IN* qg = reinterpret_cast<const IN*>(p.q);
  const IN* kg = reinterpret_cast<const IN*>(p.k);
  const IN* dog = reinterpret_cast<const IN*>(p.dO);
  const XT* matg = reinterpret_cast<const XT*>(p.mat_ws);
  XT* bblk = reinterpret_cast<XT*>(p.bwd_blk);

  // ---- staging of the next (earlier) chunk while this one computes ----
  //   K, Q, dO: register prefetch after P1 (transposed / converted at commit)
  //   gates, MR: LDS-DMA after P1 (MR double-buffered)
  //   T^R, mask: after P3;  MG, MP: after P4;  T^S: after P5 (their last uses)
  // bf16 inputs; fp32 inputs single-buffer every matrix and move them all
  // after the chunk's last barrier.
  // dO block: one 16-byte vector per thread, token = lane, columns of wave w
  constexpr int kOPerThread = 16 / (int)sizeof(IN);
  static_assert(kChunk * BV == kThreads * kOPerThread, "one dO vector per thread");
  typename MI::frag Kn[KS_STEPS], Qn[KS_STEPS];
  IN on[kOPerThread];
  auto chunk_len = [&](int c) { return min(kChunk, si.len - c * kChunk); };
  auto mat_src = [&](int c, int m) {
    return matg + ((int64_t)(si.chunk0 + c) * H + h) * kNumMats * kMatElems + m * kMatElems;
  };
  const MatDma<XT> mdo;   // this lane's matrix DMA offsets
  auto issue_regs = [&](int c) {
    const int64_t tok = si.start + (int64_t)c * kChunk;
    const int len = chunk_len(c);
    const int t = 16 * w + (lane & 15);
    const int64_t roff = ((tok + t) * H + h) * (int64_t)DK;
    load_rowfrags<IN, DK>(Kn, t < len ? kg + roff : nullptr);
    load_rowfrags<IN, DK>(Qn, t < len ? qg + roff : nullptr);
    {
      typedef IN INV __attribute__((ext_vector_type(kOPerThread)));
      const int tt = lane, j = w * kOPerThread;
      INV v = {};
      if (tt < len) v = *reinterpret_cast<const INV*>(dog + ((tok + tt) * H + h) * (int64_t)DV + j0 + j);
#pragma unroll
      for (int u = 0; u < kOPerThread; ++u) on[u] = v[u];
    }
  };
  auto issue_gates = [&](int c) {
    if (w == 0)
      dma_linear_wave(p.gate_ws + ((int64_t)(si.chunk0 + c) * H + h) * kGateBlock, graw,
                      kGateBlock * 4);
  };
  auto issue_mask = [&](int c) {   // rows of BV bytes; padding rows read row 0 (masked by 0 grads)
    if (tanh_resid) {   // the r block rows of this value block (rows past the end are zero)
      constexpr int kPerRow = BV * (int)sizeof(XT) / 16;
      static_assert(kChunk * kPerRow == kThreads, "r block = one DMA instruction per wave");
      const int P = w * 64 + lane, t = P / kPerRow, cc = P % kPerRow;
      const XT* src = reinterpret_cast<const XT*>(p.fwd_blk) + blk_off(si.chunk0 + c, h, H, 2, DV) +
                      (int64_t)t * DV + j0 + cc * (16 / (int)sizeof(XT));
      dma16(src, mask + w * 1024);
      return;
    }
    const int64_t tok = si.start + (int64_t)c * kChunk;
    const int len = chunk_len(c);
    constexpr int kPerRow = BV / 16;
#pragma unroll
    for (int m = 0; m < kChunk * BV / 1024; ++m) {
      if (w == m) {
        const int P = m * 64 + lane, t = P / kPerRow, cc = P % kPerRow;
        const int ts = t < len ? t : 0;
        const uint8_t* src = p.ck_mask + ((tok + ts) * H + h) * (int64_t)DV + j0 + cc * 16;
        dma16(src, mask + m * 1024);
      }
    }
  };
  auto issue_early = [&](int c) {   // after P1
    issue_gates(c);
    if constexpr (L::kDB) dma_mat64<XT>(mat_src(c, kMatMR), mat(kMatMR, c & 1), mdo);
  };
  auto issue_mid = [&](int c) {     // after P3
    if constexpr (L::kDB) {
      issue_mask(c);
      if constexpr (RDN) dma_mat64<XT>(mat_src(c, kMatTR), mat(kMatTR, 0), mdo);
    }
  };
  auto issue_late = [&](int c) {    // after P4
    if constexpr (L::kDB) {
      dma_mat64<XT>(mat_src(c, kMatMG), mat(kMatMG, 0), mdo);
      dma_mat64<XT>(mat_src(c, kMatMP), mat(kMatMP, 0), mdo);
    }
  };
  auto issue_after5 = [&](int c) {  // after P5 (RDN)
    if constexpr (L::kDB && RDN) dma_mat64<XT>(mat_src(c, kMatTS), mat(kMatTS, 0), mdo);
  };
  auto issue_all_single = [&](int c) {   // fp32: everything after the last barrier
    if constexpr (!L::kDB) {
      issue_mask(c);
      if constexpr (RDN) {
        dma_mat64<XT>(mat_src(c, kMatTS), mat(kMatTS, 0), mdo);
        dma_mat64<XT>(mat_src(c, kMatTR), mat(kMatTR, 0), mdo);
      }
      dma_mat64<XT>(mat_src(c, kMatMG), mat(kMatMG, 0), mdo);
      dma_mat64<XT>(mat_src(c, kMatMP), mat(kMatMP, 0), mdo);
      dma_mat64<XT>(mat_src(c, kMatMR), mat(kMatMR, 0), mdo);
    }
  };
  if (nch > 0) {
    const int c = nch - 1;
    issue_regs(c);
    issue_gates(c);
    issue_mask(c);
    if constexpr (RDN) {
      dma_mat64<XT>(mat_src(c, kMatTS), mat(kMatTS, 0), mdo);
      dma_mat64<XT>(mat_src(c, kMatTR), mat(kMatTR, 0), mdo);
    }
    dma_mat64<XT>(mat_src(c, kMatMG), mat(kMatMG, 0), mdo);
    dma_mat64<XT>(mat_src(c, kMatMP), mat(kMatMP, 0), mdo);
    dma_mat64<XT>(mat_src(c, kMatMR), mat(kMatMR, c & 1), mdo);
    wait_vmem();
  }
  barrier_lds();

  for (int c = nch - 1; c >= 0; --c) {
    set_ptrs(true);
    const int gc = si.chunk0 + c;
    const int buf = c & 1;
    const int len = chunk_len(c);
    const int64_t tok = si.start + (int64_t)c * kChunk;
    // dv = dX + diag(b) dV_tail, rows of this chunk only: this lane's 4
    // rows (one 16-byte read of b), then a transpose within each lane quad so
    // that lane 4g + i holds token t0 + i at columns 4g .. 4g + 3 of each
    // 16-column tile: one 16-byte (fp32) or 8-byte (bf16) store per tile
    auto store_dv = [&](const floatx4 (&dx)[JT], const floatx4 (&tail)[JT]) {
      const int t0 = 16 * w + acc_row(0);
      const floatx4 b4 = *reinterpret_cast<const floatx4*>(gbt + t0);
      floatx4 val[JT];
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
#pragma unroll
        for (int r = 0; r < 4; ++r) val[jt][r] = __builtin_fmaf(b4[r], tail[jt][r], dx[jt][r]) * isig;
        val[jt] = quad_transpose(val[jt]);
      }
      const int tq = t0 + (lane & 3);
      const int64_t o0 = ((tok + tq) * H + h) * (int64_t)DV + j0 + 4 * ((lane & 15) >> 2);
      if (tq < len) {
        if (p.out_bf16) {
          u16* d = reinterpret_cast<u16*>(p.dv) + o0;
#pragma unroll
          for (int jt = 0; jt < JT; ++jt) {
            u16x4 b;
#pragma unroll
            for (int e = 0; e < 4; ++e) b[e] = f2bf(val[jt][e]);
            *reinterpret_cast<u16x4*>(d + jt * 16) = b;
          }
        } else {
          float* d = reinterpret_cast<float*>(p.dv) + o0;
#pragma unroll
          for (int jt = 0; jt < JT; ++jt) *reinterpret_cast<floatx4*>(d + jt * 16) = val[jt];
        }
      }
    };

    // gradient w.r.t. this chunk's end states for the gradient kernel,
    // straight from the accumulators (bf16 inputs: fp16 scaled per (16 rows,
    // 32 columns)), stored after the chunk's last prefetch (with bf16 inputs
    // the update's transpose reads wait for them along with the prefetched
    // data).
    auto save_ckpt = [&]() {
      const int64_t off = ((int64_t)gc * H + h) * DK * DV + j0;
      if constexpr (BF) {   // blocked [DV / 32][DK][32]: each wave store is 1 KiB contiguous
        const int64_t ob = ((int64_t)gc * H + h) * DK * DV + (int64_t)j0 * DK;
        const int64_t so = ((int64_t)gc * H + h) * (DK / 16) * (DV / 32) + j0 / 32;
        // tile maxima from publish_state_max: dS, dR are unchanged since
        save_state_f16_max<IT>(dS, tmS, reinterpret_cast<f16*>(p.dS_ws) + ob, 32, p.dS_sc + so, DV / 32, w * (DK / 4));
        save_state_f16_max<IT>(dR, tmR, reinterpret_cast<f16*>(p.dR_ws) + ob, 32, p.dR_sc + so, DV / 32, w * (DK / 4));
      } else {
        save_state_f32<IT, JT>(dS, reinterpret_cast<float*>(p.dS_ws) + off, DV, w * (DK / 4));
        save_state_f32<IT, JT>(dR, reinterpret_cast<float*>(p.dR_ws) + off, DV, w * (DK / 4));
      }
    };

    // ---- commit: K fragments, K^T and Q^T (XT), dO^T, gate vectors ----
    typename Mfma<XT>::frag Kf[KS_STEPS];   // fp16 with bf16 inputs
    {
      const int t = 16 * w + (lane & 15);
#pragma unroll
      for (int s2 = 0; s2 < KS_STEPS; ++s2) {
        if constexpr (!BF) Kf[s2] = Kn[s2];
        if constexpr (BF) {   // row t, 8 columns: one 16-byte store each
          const u16x8 kv = __builtin_bit_cast(u16x8, Kn[s2]);
          const u16x8 qv = __builtin_bit_cast(u16x8, Qn[s2]);
          f16x8 kh, qh;
          if (VAR && p.qk_f16) {   // the pre-processing's fp16 rows
            kh = __builtin_bit_cast(f16x8, kv);
            qh = __builtin_bit_cast(f16x8, qv);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              kh[e] = (f16)bf2f(kv[e]);
              qh[e] = (f16)bf2f(qv[e]);
            }
          }
          const int i = s2 * 32 + (lane >> 4) * 8;
          Kf[s2] = kh;
          *reinterpret_cast<f16x8*>(TKQ::ptr(KT, t, i)) = kh;
          *reinterpret_cast<f16x8*>(TKQ::ptr(QT, t, i)) = qh;
        } else {
          const int i = s2 * 4 + (lane >> 4);
          *TKQ::ptr(KT, i, t) = Kn[s2];
          *TKQ::ptr(QT, i, t) = Qn[s2];
        }
      }
      XT* dbT = blk(bDB_DKS);
#pragma unroll
      for (int u = 0; u < kOPerThread; ++u)   // lanes write consecutive tokens
        *TT::ptr(dbT, w * kOPerThread + u, lane) = from_f<XT>(to_f<IN>(on[u]) * sig);
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

    // ---- P1: K dS_end, K dR_end (split state); scaled copies of dO ----
    floatx4 KdS[JT], KdR[JT];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      KdS[jt] = zero4();
      KdR[jt] = zero4();
      mma_rega_tile<XT, DK, TSC>(KdS[jt], Kf, dSc, jt * 16);
      mma_rega_tile<XT, DK, TSC>(KdR[jt], Kf, dRc, jt * 16);
      if constexpr (BF) {   // undo the copies' scales (powers of two: exact)
        KdS[jt] *= scS;
        KdR[jt] *= scR;
      }
      floatx4 dc, qdb, qdc;
      const floatx4 o4 = load_acc_tile<TT>(blk(bDB_DKS), jt * 16, 16 * w);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = 16 * w + acc_row(r);
        dc[r] = gout[t] * o4[r];
        qdb[r] = eqb[t] * o4[r];
        qdc[r] = egr[t] * dc[r];
      }
      store_acc_tile<TT>(blk(bDC_DX), jt * 16, 16 * w, dc);
      store_acc_tile<TT>(blk(bQDB), jt * 16, 16 * w, qdb);
      store_acc_tile<TT>(blk(bQDC), jt * 16, 16 * w, qdc);
    }
    // the transposed matrices' fragments are loaded ahead of the barriers
    // that precede their products (every matrix landed in an earlier chunk)
    const MatFrags<XT> aMR = cols_frags(mat(kMatMR, buf));
    barrier_lds();
    if (c > 0) {
      issue_regs(c - 1);
      issue_early(c - 1);
    }

    // ---- P2: dUR = diag(e^{h_C-h}) K dR_end + MR^T dc ----
    floatx4 dUR[JT];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      floatx4 a = zero4();
      mma_frags<XT, TT>(a, aMR, blk(bDC_DX), jt * 16);
#pragma unroll
      for (int r = 0; r < 4; ++r) dUR[jt][r] = dlr[16 * w + acc_row(r)] * KdR[jt][r] + a[r];
      if constexpr (RDN) store_acc_tile<TT>(blk(bDUR_DU), jt * 16, 16 * w, dUR[jt]);
    }
    MatFrags<XT> aTR;
    if constexpr (RDN) aTR = cols_frags(mat(kMatTR, 0));
    barrier_lds();

    // ---- P3: dYR, dX, dKR (RLA: dKS) ----
    floatx4 dX[JT];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      floatx4 dYR = dUR[jt];
      if constexpr (RDN) {
        dYR = zero4();
        mma_frags<XT, TT>(dYR, aTR, blk(bDUR_DU), jt * 16);
      }
      floatx4 dkr, dks;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = 16 * w + acc_row(r), j = jt * 16 + acc_col();
        if constexpr (VAR) {
          float slope;
          if (tanh_resid) {
            const float rn = to_f<XT>(reinterpret_cast<const XT*>(mask)[t * BV + j]) * invc;
            slope = s0 * __builtin_fmaf(-rn, rn, 1.f);
          } else {
            slope = mask[t * BV + j] ? 1.f : 0.f;
          }
          dX[jt][r] = slope * (ggm[t] * dYR[r]);
        } else {
          dX[jt][r] = mask[t * BV + j] ? ggm[t] * dYR[r] : 0.f;
        }
        dkr[r] = -ggm[t] * egr[t] * dYR[r];
        dks[r] = -ekp[t] * dX[jt][r];
      }
      store_acc_tile<TT>(blk(bDC_DX), jt * 16, 16 * w, dX[jt]);
      store_acc_tile<TT>(blk(bDKR), jt * 16, 16 * w, RDN ? dkr : dks);
      store_acc_tile<TT>(Yst, jt * 16, 16 * w, dYR);
    }
    const MatFrags<XT> aMP = cols_frags(mat(kMatMP, 0));
    const MatFrags<XT> aMG = cols_frags(mat(kMatMG, 0));
    barrier_lds();
    if (c > 0) issue_mid(c - 1);

    // ---- P4: dU = diag(e^{g_C-g}) K dS_end + MP^T db - MG^T dX ----
    floatx4 dU[JT];   // RLA: U = diag(b) V, so dV gets b dU
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      floatx4 a = zero4(), b = zero4();
      mma_frags<XT, TT>(a, aMP, blk(bDB_DKS), jt * 16);
      mma_frags<XT, TT>(b, aMG, blk(bDC_DX), jt * 16);
#pragma unroll
      for (int r = 0; r < 4; ++r) dU[jt][r] = dls[16 * w + acc_row(r)] * KdS[jt][r] + a[r] - b[r];
      // RLA keeps dU there for the block store
      store_acc_tile<TT>(blk(bDUR_DU), jt * 16, 16 * w, dU[jt]);
    }
    MatFrags<XT> aTS;
    if constexpr (RDN) aTS = cols_frags(mat(kMatTS, 0));
    barrier_lds();
    if (c > 0) issue_late(c - 1);
    if constexpr (!RDN) {   // last prefetch issued: dv and checkpoint stores
      store_dv(dX, dU);
      save_ckpt();
    }
    if constexpr (RDN) {
      // ---- P5: dY = T^S^T dU, dKS ----
      floatx4 dY[JT];
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        floatx4 dks;
        dY[jt] = zero4();
        mma_frags<XT, TT>(dY[jt], aTS, blk(bDUR_DU), jt * 16);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = 16 * w + acc_row(r);
          dks[r] = -ekp[t] * dX[jt][r] - gbt[t] * egs[t] * dY[jt][r];
        }
        store_acc_tile<TT>(blk(bDB_DKS), jt * 16, 16 * w, dks);
      }
      barrier_lds();
      if (c > 0) issue_after5(c - 1);
      // last prefetch issued: dv and checkpoint stores
      store_dv(dX, dY);
      save_ckpt();
      // dU is dead: its slot keeps dY for the block store (P6 does not read it)
#pragma unroll
      for (int jt = 0; jt < JT; ++jt)
        store_acc_tile<TT>(blk(bDUR_DU), jt * 16, 16 * w, dY[jt]);
    }

    // ---- P6: state gradients at the chunk start ----
    // (bf16 inputs: the Q^T, K^T fragments from transpose reads issued as
    // inline assembly, which leaves the DMA issued after P5 and the dv and
    // checkpoint stores in flight; the builtin would drain them first)
    const float eS = edge[0], eR = edge[1];
    if constexpr (BF) {
      typedef Mfma<XT> MX;
      constexpr int KS2 = kChunk / MX::kStep;
      constexpr int NF = IT * KS2;
      int fr0[NF], fk0[NF];
#pragma unroll
      for (int n = 0; n < NF; ++n) {
        fr0[n] = w * (DK / 4) + (n / KS2) * 16;
        fk0[n] = (n % KS2) * MX::kStep;
      }
      typename MX::frag qf[NF], kf[NF];
      frags_tr_sync<TKQ, XT, NF>(QT, fr0, fk0, qf);
      frags_tr_sync<TKQ, XT, NF>(KT, fr0, fk0, kf);
      auto acc = [&](floatx4& d, const typename MX::frag* a, const XT* b, int it, int jt) {
#pragma unroll
        for (int ks = 0; ks < KS2; ++ks)
          d = MX::mma(a[it * KS2 + ks], TT::template frag<MX>(b, jt * 16, ks * MX::kStep), d);
      };
#pragma unroll
      for (int it = 0; it < IT; ++it)
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) {
          dS[it][jt] *= eS;
          dR[it][jt] *= eR;
          acc(dS[it][jt], qf, blk(bQDB), it, jt);
          acc(dS[it][jt], kf, blk(RDN ? bDB_DKS : bDKR), it, jt);
          acc(dR[it][jt], qf, blk(bQDC), it, jt);
          if constexpr (RDN) acc(dR[it][jt], kf, blk(bDKR), it, jt);
        }
    } else {
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const int i0 = w * (DK / 4) + it * 16;
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) {
          dS[it][jt] *= eS;
          dR[it][jt] *= eR;
          mma_tiles<XT, kChunk, TKQ, TT>(dS[it][jt], QT, i0, blk(bQDB), jt * 16);
          mma_tiles<XT, kChunk, TKQ, TT>(dS[it][jt], KT, i0, blk(RDN ? bDB_DKS : bDKR), jt * 16);
          mma_tiles<XT, kChunk, TKQ, TT>(dR[it][jt], QT, i0, blk(bQDC), jt * 16);
          if constexpr (RDN) mma_tiles<XT, kChunk, TKQ, TT>(dR[it][jt], KT, i0, blk(bDKR), jt * 16);
        }
      }
    }
    publish_state_max();
    barrier_lds();
    if constexpr (!L::kDB) {
      if (c > 0) issue_all_single(c - 1);
    }
    // the next chunk's DMA data must have landed before anyone reads it (bf16
    // inputs: the checkpoint stores, issued after the chunk's last DMA, may
    // still be in flight; single-buffered fp32 issues its DMAs after them)
    wait_vmem_but<L::kDB ? kCkptStores : 0>();
    barrier_lds();
    {   // this chunk's dX, dY, dYR (value-major in LDS) as token-major rows in
        // 16-byte stores; rows past the end are zero.  The buffers are next
        // written after the coming chunk's first barrier.
      constexpr int kVE = 16 / (int)sizeof(XT);
      constexpr int kVPR = BV / kVE;
      static_assert(kChunk * kVPR == kThreads, "one block vector per thread");
      const int t = lane, v = w;   // lanes read consecutive tokens: no bank conflicts
#pragma unroll
      for (int b = 0; b < 3; ++b) {
        const XT* srcb = b == 0 ? blk(bDC_DX) : b == 1 ? blk(bDUR_DU) : Yst;
        uint4 x;
        if constexpr (BF) {   // two transpose reads per 16-byte row piece
          x = keep_if(tile_token_vec8<TT>(srcb, v * kVE), t < len);
        } else {
          XT vals[kVE];
#pragma unroll
          for (int k = 0; k < kVE; ++k) vals[k] = t < len ? TT::at(srcb, v * kVE + k, t) : from_f<XT>(0.f);
          x = *reinterpret_cast<const uint4*>(vals);
        }
        *reinterpret_cast<uint4*>(bblk + blk_off(gc, h, H, b, DV) + (int64_t)t * DV + j0 + v * kVE) = x;
      }
    }
    write_copies();
  }

  if (p.dS0 || p.dR0) {
#pragma unroll
    for (int it = 0; it < IT; ++it)
#pragma unroll
      for (int jt = 0; jt < JT; ++jt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = w * (DK / 4) + it * 16 + acc_row(r), j = j0 + jt * 16 + acc_col();
          if (p.dS0) p.dS0[state_off + (int64_t)i * DV + j] = dS[it][jt][r] * isig;
          if (p.dR0) p.dR0[state_off + (int64_t)i * DV + j] = dR[it][jt][r] * isig;
        }
  }
}

// ---------------------------------------------------------------------------
// Wave-specialised reverse scan: bf16 inputs, d_k = 128, 32 value columns,
// the boxed operator (no variant flags).  Eight waves per workgroup in two
// groups of four that pass the same seven barriers per chunk in the same
// order:
//   chain waves (0-3): hold dS and dR (rows 32 w' .. 32 w' + 31) and do every
//     product of the chunk (the algebra of bwd_scan_kernel) with no global
//     memory access: K comes from the K^T tile, dv and the packed chunk-end
//     checkpoints go to LDS;
//   side waves (4-7): all global memory traffic — the next (earlier)
//     chunk's K, Q, dO rows and their commit into LDS, its gate vectors, the
//     LDS-DMA of its matrices and clip mask, and the stores of the later
//     chunk's dX, dY, dYR blocks, dv and checkpoints — overlapping the chain.
// Per chunk (phase: chain waves | side waves), walking backwards:
//   0: state copies                               | commit K^T, dO^T; the later
//                                                   chunk's dX block
//   1: K dS, K dR; dc, e^g db, e^h dc             | its dY, dYR blocks and
//                                                   checkpoints; the next gate
//                                                   values; DMA of the next MR
//   2: dUR                                        | its dv
//   3: dYR, dX, dKR                               | commit Q^T; the next K, Q, dO
//                                                   rows; DMA of the next T^R
//   4: dU                                         | DMA of the next mask, MG, MP
//   5: dY, dKS; dv and checkpoints into LDS       | DMA of the next T^S
//   6: dS, dR at the chunk start; their maxima    | wait for the DMA; next gate vectors
// Each matrix is refilled once the chain has read it into registers (T^R,
// MG, MP, T^S) or, for MR, into the other buffer.
// ---------------------------------------------------------------------------
template <typename IN, int DK, int BV, bool RDN>
struct BwdWsLayout {
  typedef BwdScanLayout<IN, DK, BV, RDN, false> B;
  typedef typename B::XT XT;
  typedef typename B::TT TT;
  typedef typename B::TKQ TKQ;
  typedef typename B::TSC TSC;
  static constexpr int kKT = B::kKT, kQT = B::kQT, kCopies = B::kCopies, kCopyBytes = B::kCopyBytes;
  static constexpr int kMats = B::kMats, kBufBytes = B::kBufBytes;
  // matrix slots: the packed lower blocks (kPkBytes each)
  static constexpr int kBufs = kMats + B::kNumSlots * kPkBytes;
  static constexpr int kMask = kBufs + B::kNumBufs * kBufBytes;
  static constexpr int kGateVec = 8 * kChunk;   // floats per chunk's gate vectors
  static constexpr int kGates = kMask + B::kMaskBytes;   // two sets (chunk parity)
  static constexpr int kYst = kGates + 2 * kGateVec * 4;    // dYR (token tile)
  static constexpr int kRed = kYst + kBufBytes;             // per-wave maxima [8]
  static constexpr int kDvLd = kChunk + 4;                  // dv row stride (floats)
  static constexpr int kDv = kRed + 8 * 4;                  // dv, fp32 [BV][kDvLd] (column-major)
  // chunk-end checkpoints of dS, dR in fp16, each 16-row tile divided by its
  // power of two, in the state-copy layout ([BV][DK] padded rows, TSC), then
  // the tile scales [2][DK / 16]
  static constexpr int kCk = kDv + BV * kDvLd * 4;
  static constexpr int kCkSc = kCk + 2 * BV * TSC::kRowB;
  static constexpr int kGraw = kCkSc + 2 * (DK / 16) * 4;   // the gate block (one side wave's DMA)
  static constexpr int kZero = kGraw + kGateBlock * 4;      // 16 zero bytes (blocks above the diagonal)
  static constexpr int kBytes = kZero + 16;
  static_assert(sizeof(IN) == 2 && DK == 128 && BV == 32, "bf16, d_k 128, 32 columns");
  static_assert(kBytes <= 160 * 1024, "backward scan LDS");
  __device__ static constexpr int slot(int mat, int buf) { return B::slot(mat, buf); }
};

template <typename IN, int DK, int BV, bool RDN>
__global__ __launch_bounds__(2 * kThreads) void bwd_scan_ws_kernel(OpParams p) {
  typedef BwdWsLayout<IN, DK, BV, RDN> L;
  typedef typename L::XT XT;
  typedef typename L::TT TT;
  typedef typename L::TKQ TKQ;
  typedef typename L::TSC TSC;
  typedef Mfma<IN> MI;
  constexpr int JT = BV / 16;
  constexpr int IT = DK / 64;
  constexpr int KS_STEPS = DK / MI::kStep;
  extern __shared__ __align__(16) unsigned char smem_[];
  unsigned char* smem = smem_;
  XT* KT = reinterpret_cast<XT*>(smem + L::kKT);
  XT* QT = reinterpret_cast<XT*>(smem + L::kQT);
  XT* dSc = reinterpret_cast<XT*>(smem + L::kCopies);
  XT* dRc = reinterpret_cast<XT*>(smem + L::kCopies + L::kCopyBytes);
  uint32_t* smax = reinterpret_cast<uint32_t*>(smem + L::kRed);
  uint8_t* mask = reinterpret_cast<uint8_t*>(smem + L::kMask);
  float* gates = reinterpret_cast<float*>(smem + L::kGates);
  XT* Yst = reinterpret_cast<XT*>(smem + L::kYst);
  float* dvst = reinterpret_cast<float*>(smem + L::kDv);
  f16* ckst = reinterpret_cast<f16*>(smem + L::kCk);
  float* ckscl = reinterpret_cast<float*>(smem + L::kCkSc);
  float* graw = reinterpret_cast<float*>(smem + L::kGraw);   // prep's gate block
  auto mat = [&](int m, int buf) {
    return reinterpret_cast<XT*>(smem + L::kMats + L::slot(m, buf) * kPkBytes);
  };
  const XT* zero16 = reinterpret_cast<const XT*>(smem + L::kZero);
  auto blk = [&](int b) { return reinterpret_cast<XT*>(smem + L::kBufs + b * L::kBufBytes); };
  // gate vectors of chunk c: beta, gamma, e^{g_t}, e^{g_{t-1}}, e^{h_t},
  // e^{g_C - g_t}, e^{h_C - h_t}, then [e^{g_C}, e^{h_C}]
  auto gvec = [&](int c, int k) { return gates + (c & 1) * L::kGateVec + k * kChunk; };

  const int H = p.H, DV = p.DV, tid = threadIdx.x, lane = tid & 63;
  const int wu = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool chain = wu < kWaves;      // wave-uniform role
  const int ww = wu & (kWaves - 1);    // index within the role's four waves
  const int nvb = DV / BV;
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int pair = (slot / nvb) * 8 + xcd, vb = slot % nvb;
  if (pair >= p.st.nseq * H) return;
  const int n = seq_order(p.st, pair / H), h = pair % H;
  const SeqInfo si = seq_info(p.st, n);
  const int nch = (si.len + kChunk - 1) / kChunk;
  const int j0 = vb * BV;
  const int64_t state_off = ((int64_t)n * H + h) * DK * DV;

  // scale of the upstream gradients of this (sequence, head), as
  // bwd_scan_kernel (over all eight waves)
  float sig = 1.f, isig = 1.f;
  if (p.grad_absmax) {
    uint32_t m = 0;
    for (int c = tid; c < nch; c += 2 * kThreads)
      m = max(m, p.grad_absmax[(int64_t)(si.chunk0 + c) * H + h]);
    m = wave_absmax_bits(m);
    smax[wu] = m;   // every lane stores the wave-uniform value
    barrier_lds();
    m = 0;
#pragma unroll
    for (int k = 0; k < 2 * kWaves; ++k) m = max(m, smax[k]);
    barrier_lds();
    const int be = (int)(m >> 23);
    const int e = be == 0 ? 0 : min(max(129 - be, -126), 126);
    sig = exp2_int(e);
    isig = exp2_int(-e);
    if (vb == 0 && tid == 0) p.grad_scale[(int64_t)n * H + h] = sig;
  }

  const IN* qg = reinterpret_cast<const IN*>(p.q);
  const IN* kg = reinterpret_cast<const IN*>(p.k);
  const IN* dog = reinterpret_cast<const IN*>(p.dO);
  const XT* matg = reinterpret_cast<const XT*>(p.mat_ws);
  XT* bblk = reinterpret_cast<XT*>(p.bwd_blk);
  auto chunk_len = [&](int c) { return min(kChunk, si.len - c * kChunk); };
  auto mat_src = [&](int c, int m) {
    return matg + ((int64_t)(si.chunk0 + c) * H + h) * kNumMats * kMatElems + m * kMatElems;
  };
  constexpr int kOPerThread = 16 / (int)sizeof(IN);
  static_assert(kChunk * BV == kThreads * kOPerThread, "one dO vector per chain thread");

  // One loop body, instantiated once per role (std::true_type: chain
  // waves): both roles pass the same barriers in the same order by
  // construction, and each instance gets its own registers.
  auto run = [&](auto role) {
  constexpr bool CH = decltype(role)::value;
  floatx4 dS[IT][JT], dR[IT][JT];      // chain: the gradient states
  typename MI::frag Kn[KS_STEPS], Qn[KS_STEPS];   // side: the next chunk's K, Q rows 16 ww + (lane & 15)
  IN on[kOPerThread];                              // side: its dO vector
  float scS = 1.f, scR = 1.f;
  uint32_t tmS[IT], tmR[IT];
  auto publish_state_max = [&]() {   // chain: the four tile maxima, reduced together
    static_assert(IT == 2, "two tiles of each state per wave");
    const uint32_t lm[4] = {lane_absmax_bits(dS[0][0], dS[0][1]), lane_absmax_bits(dS[1][0], dS[1][1]),
                            lane_absmax_bits(dR[0][0], dR[0][1]), lane_absmax_bits(dR[1][0], dR[1][1])};
    const uint32_t y = wave_max4_bits(lm);
    tmS[0] = __builtin_amdgcn_readlane(y, 0);
    tmS[1] = __builtin_amdgcn_readlane(y, 2);
    tmR[0] = __builtin_amdgcn_readlane(y, 1);
    tmR[1] = __builtin_amdgcn_readlane(y, 3);
    smax[ww] = max(tmS[0], tmS[1]);   // every lane stores the wave-uniform value
    smax[4 + ww] = max(tmR[0], tmR[1]);
  };
  auto write_copies = [&]() {   // chain, after a barrier that follows publish_state_max
    const uint32_t ms = max(max(smax[0], smax[1]), max(smax[2], smax[3]));
    const uint32_t mr = max(max(smax[4], smax[5]), max(smax[6], smax[7]));
    const int es = pow2_scale_exp(ms), er = pow2_scale_exp(mr);
    scS = exp2_int(es);
    scR = exp2_int(er);
    const float iS = exp2_int(-es), iR = exp2_int(-er);
#pragma unroll
    for (int it = 0; it < IT; ++it)
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        store_state_copy<TSC>(dSc, jt * 16, ww * (DK / 4) + it * 16, dS[it][jt] * iS);
        store_state_copy<TSC>(dRc, jt * 16, ww * (DK / 4) + it * 16, dR[it][jt] * iR);
      }
  };
  // The side's global addresses are a chunk's uniform base plus a 32-bit
  // lane offset that does not change from chunk to chunk, so the memory
  // instructions take a scalar base and the lane part is formed once.
  // K or Q rows: token row 16 ww + (lane & 15) of the chunk whose rows start at base
  auto load_rows = [&](typename MI::frag (&afr)[KS_STEPS], const IN* base, bool ok) {
    const uint32_t o = (uint32_t)((16 * ww + (lane & 15)) * H * DK + (lane >> 4) * 8);
#pragma unroll
    for (int s2 = 0; s2 < KS_STEPS; ++s2) {
      u16x8 v = {0, 0, 0, 0, 0, 0, 0, 0};
      if (ok) v = *reinterpret_cast<const u16x8*>(base + o + s2 * 32);
      afr[s2] = __builtin_bit_cast(typename MI::frag, v);
    }
  };
  auto issue_regs = [&](int c) {   // side: K, Q rows and this thread's dO vector of chunk c
    const int64_t tok = si.start + (int64_t)c * kChunk;
    const int len = chunk_len(c);
    const bool ok = 16 * ww + (lane & 15) < len;
    const int64_t rb = (tok * H + h) * (int64_t)DK;
    load_rows(Kn, kg + rb, ok);
    load_rows(Qn, qg + rb, ok);
    typedef IN INV __attribute__((ext_vector_type(kOPerThread)));
    const int tt = lane, j = ww * kOPerThread;
    INV v = {};
    if (tt < len)
      v = *reinterpret_cast<const INV*>(dog + (tok * H + h) * (int64_t)DV + j0 + j + (uint32_t)(tt * H * DV));
#pragma unroll
    for (int u = 0; u < kOPerThread; ++u) on[u] = v[u];
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
  // side: chunk c's matrix m into slot buffer buf; the side wave x issues two
  // of the five DMA instructions (chosen per matrix to even out the phases)
  auto dma_mat = [&](int c, int m, int buf, int x) {
    dma_mat_packed<true>(mat_src(c, m), mat(m, buf), (ww - x) & 3, kWaves);
  };
  auto issue_mask = [&](int c) {   // side: rows of BV bytes; padding rows read row 0 (masked by 0 gradients)
    const int64_t tok = si.start + (int64_t)c * kChunk;
    const int len = chunk_len(c);
    constexpr int kPerRow = BV / 16;
    constexpr int kInst = kChunk * BV / 1024;
    static_assert(kInst <= kWaves, "one mask DMA instruction per side wave at most");
    if (ww < kInst) {
      const int P = ww * 64 + lane, t = P / kPerRow, cc = P % kPerRow;
      const int ts = t < len ? t : 0;
      dma16(p.ck_mask + (tok * H + h) * (int64_t)DV + j0 + (uint32_t)(ts * H * DV + cc * 16), mask + ww * 1024);
    }
  };
  // side: block b (0 dX, 1 dY, 2 dYR) of chunk c, tokens 16 ww .. 16 ww + 15,
  // one 64-byte segment per token; rows past the end are zero
  auto store_block = [&](int c, int b) {
    static_assert(sizeof(XT) == 2, "four lanes per 32-value token row");
    const int64_t gc = si.chunk0 + c;
    const XT* srcb = b == 0 ? blk(bDC_DX) : b == 1 ? blk(bDUR_DU) : Yst;
    const int t = 16 * ww + (lane & 15);
    const uint4 x = keep_if(tile_token_rows16_sync<TT>(srcb, 16 * ww), t < chunk_len(c));
    *reinterpret_cast<uint4*>(bblk + blk_off(gc, h, H, b, DV) + j0 + (uint32_t)(t * DV + 8 * (lane >> 4))) = x;
  };
  // side: dv rows 16 ww + 8 u + lane / 8, columns 4 (lane % 8) .. from the
  // column-major stage (four reads per 16 bytes)
  auto store_dv = [&](int c) {
    const int64_t tok = si.start + (int64_t)c * kChunk;
    const int len = chunk_len(c);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int t = 16 * ww + 8 * u + (lane >> 3), col = 4 * (lane & 7);
      const uint4 x = lds_read4x1_sync(dvst + col * L::kDvLd + t, L::kDvLd * 4);
      if (t < len) {
        const int64_t ob = (tok * H + h) * (int64_t)DV + j0;
        const uint32_t ol = (uint32_t)(t * H * DV + col);
        if (p.out_bf16) {
          const floatx4 f = {__uint_as_float(x.x), __uint_as_float(x.y), __uint_as_float(x.z), __uint_as_float(x.w)};
          u16x4 b;
#pragma unroll
          for (int e = 0; e < 4; ++e) b[e] = f2bf(f[e]);
          *reinterpret_cast<u16x4*>(reinterpret_cast<u16*>(p.dv) + ob + ol) = b;
        } else {
          *reinterpret_cast<uint4*>(reinterpret_cast<float*>(p.dv) + ob + ol) = x;
        }
      }
    }
  };
  // side: chunk c's end-state checkpoints from LDS, rows 32 ww .. 32 ww + 31
  // of each: two transpose reads give a lane 16 bytes of one row, so each
  // store writes 16 rows (1 KiB contiguous); and their tile scales
  auto store_ckpt = [&](int c) {
    const int64_t gc = si.chunk0 + c;
    const int64_t ob = ((int64_t)gc * H + h) * DK * DV + (int64_t)j0 * DK;
    const int64_t so = ((int64_t)gc * H + h) * (DK / 16) * (DV / 32) + j0 / 32;
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      f16* dst = reinterpret_cast<f16*>(st ? p.dR_ws : p.dS_ws) + ob;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int t0 = ww * (DK / 4) + 16 * u;
        const uint4 x = tile_token_rows16_sync<TSC>(ckst + st * BV * (TSC::kRowB / 2), t0);
        *reinterpret_cast<uint4*>(dst + (uint32_t)((t0 + (lane & 15)) * BV + 8 * (lane >> 4))) = x;
      }
    }
    if (lane < 2 * IT) {   // one lane per tile scale, both states in one store
      const int st = lane / IT, it = lane % IT;
      (st ? p.dR_sc : p.dS_sc)[so + (int64_t)(ww * IT + it) * (DV / 32)] = ckscl[st * (DK / 16) + ww * IT + it];
    }
  };
  // side: rows 16 ww + (lane & 15) of a K^T or Q^T tile (fp16) from the
  // prefetched bf16 rows, one 16-byte store per k-step
  auto commit_rows = [&](XT* dst, const typename MI::frag (&src)[KS_STEPS]) {
    const int t = 16 * ww + (lane & 15);
#pragma unroll
    for (int s2 = 0; s2 < KS_STEPS; ++s2) {
      const u16x8 v = __builtin_bit_cast(u16x8, src[s2]);
      f16x8 x;
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = (f16)bf2f(v[e]);
      *reinterpret_cast<f16x8*>(TKQ::ptr(dst, t, s2 * 32 + (lane >> 4) * 8)) = x;
    }
  };
  auto commit_do = [&]() {   // side: dO^T (scaled) of the chunk whose vector on holds
    XT* dbT = blk(bDB_DKS);
#pragma unroll
    for (int u = 0; u < kOPerThread; ++u)   // lanes write consecutive tokens
      *TT::ptr(dbT, ww * kOPerThread + u, lane) = from_f<XT>(to_f<IN>(on[u]) * sig);
  };

  // ---- prologue: the last chunk's staging; the end-state maxima ----
  if constexpr (CH) {
#pragma unroll
    for (int it = 0; it < IT; ++it)
#pragma unroll
      for (int jt = 0; jt < JT; ++jt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = ww * (DK / 4) + it * 16 + acc_row(r), j = j0 + jt * 16 + acc_col();
          dS[it][jt][r] = p.dS_fin ? p.dS_fin[state_off + (int64_t)i * DV + j] * sig : 0.f;
          dR[it][jt][r] = p.dR_fin ? p.dR_fin[state_off + (int64_t)i * DV + j] * sig : 0.f;
        }
    publish_state_max();
  } else {
    if (nch > 0) {
      const int c = nch - 1;
      issue_regs(c);
      issue_gates(c);
      issue_mask(c);
      if constexpr (RDN) {
        dma_mat(c, kMatTS, 0, 1);
        dma_mat(c, kMatTR, 0, 2);
      }
      dma_mat(c, kMatMG, 0, 2);
      dma_mat(c, kMatMP, 0, 3);
      dma_mat(c, kMatMR, c & 1, 3);
      wait_vmem();
      write_gates(c);
    }
  }
  if (tid == 0) *reinterpret_cast<uint4*>(smem + L::kZero) = uint4{0, 0, 0, 0};
  barrier_lds();

  floatx4 KdS[JT], KdR[JT], dUR[JT], dX[JT];
  MatFrags<XT> aMR, aTR, aMP, aMG, aTS;
  for (int c = nch - 1; c >= 0; --c) {
    const int gc = si.chunk0 + c;
    const int buf = c & 1;
    const int len = chunk_len(c);
    const int64_t tok = si.start + (int64_t)c * kChunk;
    const float* gbt = gvec(c, 0);
    const float* ggm = gvec(c, 1);
    const float* egs = gvec(c, 2);
    const float* egsp = gvec(c, 3);
    const float* egr = gvec(c, 4);
    const float* dls = gvec(c, 5);
    const float* dlr = gvec(c, 6);
    const float* edge = gvec(c, 7);

    // ======== phase 0: copies and commit | the later chunk's outputs ========
    if constexpr (CH) {
      write_copies();
    } else {
      commit_rows(KT, Kn);   // read by phase 1 (Q^T, read in phase 6 only, in phase 3)
      commit_do();
      if (c + 1 < nch) store_block(c + 1, 0);   // dX: its slot takes dc in phase 1
    }
    barrier_lds();

    // ======== phase 1: K dS_end, K dR_end; dc, e^g db, e^h dc ========
    if constexpr (CH) {
      typename Mfma<XT>::frag Kf[KS_STEPS];   // rows 16 ww + (lane & 15) of the K^T tile
#pragma unroll
      for (int s2 = 0; s2 < KS_STEPS; ++s2)
        Kf[s2] = *reinterpret_cast<const typename Mfma<XT>::frag*>(
            TKQ::ptr(KT, 16 * ww + (lane & 15), s2 * 32 + (lane >> 4) * 8));
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        KdS[jt] = zero4();
        KdR[jt] = zero4();
        mma_rega_tile<XT, DK, TSC>(KdS[jt], Kf, dSc, jt * 16);
        mma_rega_tile<XT, DK, TSC>(KdR[jt], Kf, dRc, jt * 16);
        KdS[jt] *= scS;   // undo the copies' scales (powers of two: exact)
        KdR[jt] *= scR;
        floatx4 dc, qdb, qdc;
        const floatx4 o4 = load_acc_tile<TT>(blk(bDB_DKS), jt * 16, 16 * ww);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = 16 * ww + acc_row(r);
          dc[r] = ggm[t] * o4[r];
          qdb[r] = egs[t] * o4[r];
          qdc[r] = egr[t] * dc[r];
        }
        store_acc_tile<TT>(blk(bDC_DX), jt * 16, 16 * ww, dc);
        store_acc_tile<TT>(blk(bQDB), jt * 16, 16 * ww, qdb);
        store_acc_tile<TT>(blk(bQDC), jt * 16, 16 * ww, qdc);
      }
      aMR = packed_cols_frags_sync(mat(kMatMR, buf), ww, zero16);
    } else {
      if (c + 1 < nch) {   // dY (its slot takes dUR in phase 2), dYR, checkpoints
        store_block(c + 1, 1);
        store_block(c + 1, 2);
        store_ckpt(c + 1);
      }
      if (c > 0) {
        issue_gates(c - 1);
        dma_mat(c - 1, kMatMR, (c - 1) & 1, 3);
      }
    }
    barrier_lds();

    // ======== phase 2: dUR = diag(e^{h_C-h}) K dR_end + MR^T dc ========
    if constexpr (CH) {
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        floatx4 a = zero4();
        mma_frags<XT, TT>(a, aMR, blk(bDC_DX), jt * 16);
#pragma unroll
        for (int r = 0; r < 4; ++r) dUR[jt][r] = dlr[16 * ww + acc_row(r)] * KdR[jt][r] + a[r];
        if constexpr (RDN) store_acc_tile<TT>(blk(bDUR_DU), jt * 16, 16 * ww, dUR[jt]);
      }
      if constexpr (RDN) aTR = packed_cols_frags_sync(mat(kMatTR, 0), ww, zero16);
    } else {
      if (c + 1 < nch) store_dv(c + 1);
    }
    barrier_lds();

    // ======== phase 3: dYR, dX, dKR (RLA: dKS) ========
    if constexpr (CH) {
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        floatx4 dYR = dUR[jt];
        if constexpr (RDN) {
          dYR = zero4();
          mma_frags<XT, TT>(dYR, aTR, blk(bDUR_DU), jt * 16);
        }
        floatx4 dkr, dks;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = 16 * ww + acc_row(r), j = jt * 16 + acc_col();
          dX[jt][r] = mask[t * BV + j] ? ggm[t] * dYR[r] : 0.f;
          dkr[r] = -ggm[t] * egr[t] * dYR[r];
          dks[r] = -egsp[t] * dX[jt][r];
        }
        store_acc_tile<TT>(blk(bDC_DX), jt * 16, 16 * ww, dX[jt]);
        store_acc_tile<TT>(blk(bDKR), jt * 16, 16 * ww, RDN ? dkr : dks);
        store_acc_tile<TT>(Yst, jt * 16, 16 * ww, dYR);
      }
      aMP = packed_cols_frags_sync(mat(kMatMP, 0), ww, zero16);
      aMG = packed_cols_frags_sync(mat(kMatMG, 0), ww, zero16);
    } else {
      commit_rows(QT, Qn);   // then the next chunk's rows may replace Kn, Qn, on
      if (c > 0) issue_regs(c - 1);
      if constexpr (RDN) {   // T^R was read into registers before the previous barrier
        if (c > 0) dma_mat(c - 1, kMatTR, 0, 2);
      }
    }
    barrier_lds();

    // ======== phase 4: dU = diag(e^{g_C-g}) K dS_end + MP^T db - MG^T dX ========
    floatx4 dU[JT];   // RLA: U = diag(b) V, so dV gets b dU
    if constexpr (CH) {
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        floatx4 a = zero4(), b = zero4();
        mma_frags<XT, TT>(a, aMP, blk(bDB_DKS), jt * 16);
        mma_frags<XT, TT>(b, aMG, blk(bDC_DX), jt * 16);
#pragma unroll
        for (int r = 0; r < 4; ++r) dU[jt][r] = dls[16 * ww + acc_row(r)] * KdS[jt][r] + a[r] - b[r];
        store_acc_tile<TT>(blk(bDUR_DU), jt * 16, 16 * ww, dU[jt]);
      }
      if constexpr (RDN) aTS = packed_cols_frags_sync(mat(kMatTS, 0), ww, zero16);
    } else {
      if (c > 0) {   // the mask (read in phase 3) and MG, MP (read into registers)
        issue_mask(c - 1);
        dma_mat(c - 1, kMatMG, 0, 2);
        dma_mat(c - 1, kMatMP, 0, 3);
      }
    }
    barrier_lds();

    // ======== phase 5: dY = T^S^T dU, dKS; dv; checkpoints ========
    if constexpr (CH) {
      floatx4 tail[JT];   // RDN: dY; RLA: dU
      if constexpr (RDN) {
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) {
          floatx4 dks;
          tail[jt] = zero4();
          mma_frags<XT, TT>(tail[jt], aTS, blk(bDUR_DU), jt * 16);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int t = 16 * ww + acc_row(r);
            dks[r] = -egsp[t] * dX[jt][r] - gbt[t] * egs[t] * tail[jt][r];
          }
          store_acc_tile<TT>(blk(bDB_DKS), jt * 16, 16 * ww, dks);
        }
      } else {
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) tail[jt] = dU[jt];
      }
      {   // dv = dX + diag(b) tail into the column-major stage: this lane's 4
          // tokens t0 .. t0 + 3 of column 16 jt + (lane & 15), one 16-byte store
        const int t0 = 16 * ww + acc_row(0);
        const floatx4 b4 = *reinterpret_cast<const floatx4*>(gbt + t0);
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) {
          floatx4 val;
#pragma unroll
          for (int r = 0; r < 4; ++r) val[r] = __builtin_fmaf(b4[r], tail[jt][r], dX[jt][r]) * isig;
          *reinterpret_cast<floatx4*>(dvst + (jt * 16 + acc_col()) * L::kDvLd + t0) = val;
        }
      }
      {   // gradient w.r.t. this chunk's end states (tile maxima from
          // publish_state_max: dS, dR are unchanged since), each 16-row tile
          // divided by its power of two, in the state-copy layout
#pragma unroll
        for (int st = 0; st < 2; ++st) {
#pragma unroll
          for (int it = 0; it < IT; ++it) {
            const int e = pow2_scale_exp(st ? tmR[it] : tmS[it]);
            const float sc = exp2_int(-e);
#pragma unroll
            for (int jt = 0; jt < JT; ++jt)
              store_state_copy<TSC>(ckst + st * BV * (TSC::kRowB / 2), jt * 16, ww * (DK / 4) + 16 * it,
                                    (st ? dR[it][jt] : dS[it][jt]) * sc);
            ckscl[st * (DK / 16) + ww * IT + it] = exp2_int(e);   // every lane: the wave-uniform value
          }
        }
      }
      if constexpr (RDN) {   // dU is dead: its slot keeps dY for the block store
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) store_acc_tile<TT>(blk(bDUR_DU), jt * 16, 16 * ww, tail[jt]);
      }
    } else {
      if constexpr (RDN) {   // T^S was read into registers before the previous barrier
        if (c > 0) dma_mat(c - 1, kMatTS, 0, 1);
      }
    }
    barrier_lds();

    // ======== phase 6: state gradients at the chunk start ========
    if constexpr (CH) {
      typedef Mfma<XT> MX;
      const float eS = edge[0], eR = edge[1];
      constexpr int KS2 = kChunk / MX::kStep;
      constexpr int NF = IT * KS2;
      int fr0[NF], fk0[NF];
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        fr0[f] = ww * (DK / 4) + (f / KS2) * 16;
        fk0[f] = (f % KS2) * MX::kStep;
      }
      typename MX::frag qf[NF], kf[NF];
      frags_tr_sync<TKQ, XT, NF>(QT, fr0, fk0, qf);
      frags_tr_sync<TKQ, XT, NF>(KT, fr0, fk0, kf);
      auto acc = [&](floatx4& d, const typename MX::frag* a, const XT* b, int it, int jt) {
#pragma unroll
        for (int ks = 0; ks < KS2; ++ks)
          d = MX::mma(a[it * KS2 + ks], TT::template frag<MX>(b, jt * 16, ks * MX::kStep), d);
      };
#pragma unroll
      for (int it = 0; it < IT; ++it)
#pragma unroll
        for (int jt = 0; jt < JT; ++jt) {
          dS[it][jt] *= eS;
          dR[it][jt] *= eR;
          acc(dS[it][jt], qf, blk(bQDB), it, jt);
          acc(dS[it][jt], kf, blk(RDN ? bDB_DKS : bDKR), it, jt);
          acc(dR[it][jt], qf, blk(bQDC), it, jt);
          if constexpr (RDN) acc(dR[it][jt], kf, blk(bDKR), it, jt);
        }
      publish_state_max();
    } else {
      wait_vmem();   // the next chunk's DMA; the barrier below publishes it
      if (c > 0) write_gates(c - 1);
    }
    barrier_lds();
  }

  if constexpr (CH) {
    if (p.dS0 || p.dR0) {
#pragma unroll
      for (int it = 0; it < IT; ++it)
#pragma unroll
        for (int jt = 0; jt < JT; ++jt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int i = ww * (DK / 4) + it * 16 + acc_row(r), j = j0 + jt * 16 + acc_col();
            if (p.dS0) p.dS0[state_off + (int64_t)i * DV + j] = dS[it][jt][r] * isig;
            if (p.dR0) p.dR0[state_off + (int64_t)i * DV + j] = dR[it][jt][r] * isig;
          }
    }
  } else if (nch > 0) {   // the first chunk's outputs
    store_block(0, 0);
    store_block(0, 1);
    store_block(0, 2);
    store_ckpt(0);
    store_dv(0);
  }
  };
  if (chain) run(std::true_type{});
  else run(std::false_type{});
}

template <typename IN, int DK, int BV, bool RDN, bool VAR>
hipError_t launch_bwd_scan_v(const OpParams& p, hipStream_t stream) {
  typedef BwdScanLayout<IN, DK, BV, RDN, VAR> L;
  auto kern = bwd_scan_kernel<IN, DK, BV, RDN, VAR>;
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

template <typename IN, int DK, int BV, bool RDN>
hipError_t launch_bwd_scan_ws(const OpParams& p, hipStream_t stream) {
  typedef BwdWsLayout<IN, DK, BV, RDN> L;
  auto kern = bwd_scan_ws_kernel<IN, DK, BV, RDN>;
  hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, L::kBytes);
  if (err != hipSuccess) return err;
  const int nvb = p.DV / BV;
  const int npairs = p.st.nseq * p.H;
  const int grid = ((npairs + 7) / 8) * 8 * nvb;
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(2 * kThreads), L::kBytes, stream, p);
  return hipGetLastError();
}

template <typename IN, int DK, int BV, bool RDN>
hipError_t launch_bwd_scan_t(const OpParams& p, hipStream_t stream) {
  if ((p.vflags & kVarOperator) || p.qk_f16) return launch_bwd_scan_v<IN, DK, BV, RDN, true>(p, stream);
  if constexpr (sizeof(IN) == 2 && DK == 128 && BV == 32) {
    return launch_bwd_scan_ws<IN, DK, BV, RDN>(p, stream);   // the boxed operator: wave-specialised
  }
  return launch_bwd_scan_v<IN, DK, BV, RDN, false>(p, stream);
}

}  // namespace

hipError_t launch_bwd_scan(const OpParams& p, bool bf16, hipStream_t stream) {
  if (bf16) {
    if (p.DK == 128) return p.rdn ? launch_bwd_scan_t<u16, 128, 32, true>(p, stream) : launch_bwd_scan_t<u16, 128, 32, false>(p, stream);
    return p.rdn ? launch_bwd_scan_t<u16, 64, 32, true>(p, stream) : launch_bwd_scan_t<u16, 64, 32, false>(p, stream);
  }
  return p.rdn ? launch_bwd_scan_t<float, 64, 16, true>(p, stream) : launch_bwd_scan_t<float, 64, 16, false>(p, stream);
}

}  // namespace rla
