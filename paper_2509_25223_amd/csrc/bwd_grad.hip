// Chunk-parallel gradient contractions: one 256-thread workgroup per (chunk,
// head).  Inputs per chunk: its start states S0, R0 (from the checkpointing
// forward scan), the gradients dS1, dR1 of its end states (from the reverse
// scan), the clip mask, and the prep kernel's gates and matrices.  The
// workgroup re-derives the chunk's forward intermediates (U, X, r, UR, c) and
// backward intermediates (dUR, dYR, dX, dU, dY, dKS, dKR) one block of 16
// value columns at a time, and accumulates over the blocks:
//   dQ += diag(e^g) dO S0^T + diag(e^h gamma) dO R0^T
//   dK += diag(e^{g_C-g}) U dS1^T + diag(e^{h_C-h}) UR dR1^T + dKS S0^T + dKR R0^T
//   W1 = dO U^T, W2 = diag(gamma) dO UR^T, W3 = dX U^T, W4 = dY U^T, W5 = dYR UR^T
//   dV = dX + diag(b) dY   (RLA: dX + diag(b) dU)
// and the row sums that the gates' gradients need.  Then, from W1..W5, the
// Gram G = K K^T, the scores P = Q K^T and the decays,
//   dP = E^S (.) W1 (.) L- + E^R (.) W2 (.) L
//   dG = [ -E' (.) W3 - diag(b) E^S (.) W4 - diag(gamma) E^R (.) W5 ] (.) L-
//   dQ += dP K,  dK += dP^T Q + (dG + dG^T) K
// where the E's are the decay matrices of prep.hip and dA^S = -W4, dA^R = -W5
// are the gradients of the triangular systems (A = I + ... inverted by T:
// dA = -T^T dU (T Y)^T = -dY U^T).  Gate gradients: d log a over a chunk is
// the suffix sum of the gradients of the cumulative sums g_t, h_t.
//
// Precision (bf16 inputs): all products on fp16 MFMA with fp32 accumulation.
// The state blocks are scaled by a power of two per (chunk, head, block) so
// their fp16 copies cannot overflow; the scale is undone on the products.
#include <type_traits>

#include "kernels.hpp"

namespace rla {

namespace {

constexpr int kBVG = 16;   // value columns per block

template <typename IN, int DK, bool RDN>
struct GradLayout {
  static constexpr bool kBF = sizeof(IN) == 2;
  typedef typename std::conditional<kBF, f16, float>::type XT;
  static constexpr int kPad = kBF ? 8 : 4;
  static constexpr int kLdK = DK + kPad;     // KX, QX rows
  static constexpr int kLdX = kChunk + kPad; // matrices, per-token blocks [16][64], dP, dG
  static constexpr int kLdV = kBVG + kPad;   // state blocks [DK][16]
  static constexpr int kLdZ = kChunk + 1;    // fp32 Z matrices
  static constexpr bool kMatsInLds = kBF;
  static constexpr int kNumBlocks = 16;
  static constexpr int kKX = 0;
  static constexpr int kQX = kKX + kChunk * kLdK * (int)sizeof(XT);
  static constexpr int kMats = kQX + kChunk * kLdK * (int)sizeof(XT);
  static constexpr int kMatBytes = kMatsInLds ? 5 * kChunk * kLdX * (int)sizeof(XT) : 0;
  static constexpr int kStates = kMats + kMatBytes;
  static constexpr int kStateBytes = DK * kLdV * (int)sizeof(XT);
  static constexpr int kBlocks = kStates + 4 * kStateBytes;
  static constexpr int kBlockBytes = kBVG * kLdX * (int)sizeof(XT);
  // after the value loop: Z matrices over states + blocks; dP, dG over the
  // matrices (bf16) or after the Z matrices (fp32)
  static constexpr int kZ = kStates;
  static constexpr int kZBytes = 3 * kChunk * kLdZ * 4;
  static constexpr int kDPG = kMatsInLds ? kMats : kZ + kZBytes;
  static constexpr int kDPGBytes = 2 * kChunk * kLdX * (int)sizeof(XT);
  static constexpr int kLoopEnd = kBlocks + kNumBlocks * kBlockBytes;
  static constexpr int kEndUse = kMatsInLds ? kZ + kZBytes : kDPG + kDPGBytes;
  static constexpr int kEndOfBlocks = kLoopEnd > kEndUse ? kLoopEnd : kEndUse;
  static_assert(!kMatsInLds || kDPGBytes <= kMatBytes, "dP region");
  static constexpr int kVB = kEndOfBlocks;
  static constexpr int kMask = kVB + kChunk * kBVG * (int)sizeof(IN);
  static constexpr int kGates = kMask + kChunk * kBVG;
  static constexpr int kNumGateArrays = 12;
  static constexpr int kRows = kGates + kNumGateArrays * kChunk * 4;
  static constexpr int kNumRows = 8;
  static constexpr int kRed = kRows + kNumRows * kChunk * 4;
  static constexpr int kBytes = kRed + 64 * 4;
  static_assert(kBytes <= 160 * 1024, "gradient kernel LDS");
};

// per-token block slots, each [16][64] value-major
enum {
  kYT = 0,  // Y, later YR
  kUT, kDUT, kURT, kDURT, kDBT, kDCT, kEDBT, kEDCT, kDURt, kDXT, kDKRT, kDYRT, kDUt, kDYT, kDKST
};
// row accumulator slots
enum { rBeta = 0, rGamma, rGS, rGSP, rGR, rZS, rZP, rZR };

__device__ __forceinline__ float sum16(float x) {   // over the 16 lanes sharing a lane>>4
#pragma unroll
  for (int off = 1; off < 16; off <<= 1) x += __shfl_xor(x, off, 64);
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) x += __shfl_xor(x, off, 64);
  return x;
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
  return x;
}

template <typename IN, int DK, bool RDN, typename OT>
__global__ __launch_bounds__(kThreads) void bwd_grad_kernel(OpParams p) {
  typedef GradLayout<IN, DK, RDN> L;
  typedef typename L::XT XT;
  typedef Mfma<XT> M;       // 32-deep (fp16) / 4-deep (fp32) steps
  typedef MfmaK16<XT> M16;  // 16-deep steps for contractions over a value block
  constexpr int IT = DK / 16;
  extern __shared__ __align__(16) unsigned char smem[];
  XT* KX = reinterpret_cast<XT*>(smem + L::kKX);
  XT* QX = reinterpret_cast<XT*>(smem + L::kQX);
  XT* S0N = reinterpret_cast<XT*>(smem + L::kStates);
  XT* R0N = reinterpret_cast<XT*>(smem + L::kStates + 1 * L::kStateBytes);
  XT* dS1N = reinterpret_cast<XT*>(smem + L::kStates + 2 * L::kStateBytes);
  XT* dR1N = reinterpret_cast<XT*>(smem + L::kStates + 3 * L::kStateBytes);
  auto blk = [&](int b) { return reinterpret_cast<XT*>(smem + L::kBlocks + b * L::kBlockBytes); };
  IN* VB = reinterpret_cast<IN*>(smem + L::kVB);
  uint8_t* mask = reinterpret_cast<uint8_t*>(smem + L::kMask);
  float* gbt = reinterpret_cast<float*>(smem + L::kGates);
  float* ggm = gbt + kChunk;
  float* egs = ggm + kChunk;
  float* egsp = egs + kChunk;
  float* egr = egsp + kChunk;
  float* dls = egr + kChunk;
  float* dlr = dls + kChunk;
  float* gsv = dlr + kChunk;    // g_t
  float* gspv = gsv + kChunk;   // g_{t-1}
  float* grv = gspv + kChunk;   // h_t
  float* edge = grv + kChunk;   // e^{g_C}, e^{h_C}
  float* rows = reinterpret_cast<float*>(smem + L::kRows);
  float* red = reinterpret_cast<float*>(smem + L::kRed);

  const int c = blockIdx.x, h = blockIdx.y, tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  ChunkInfo ci;
  if (!chunk_info(p.st, c, ci)) return;
  const int H = p.H, DV = p.DV, len = ci.len;
  const int64_t tok = ci.tok;
  const float clip = p.clip;

  const IN* qg = reinterpret_cast<const IN*>(p.q);
  const IN* kg = reinterpret_cast<const IN*>(p.k);
  const IN* vg = reinterpret_cast<const IN*>(p.v);
  const IN* dog = reinterpret_cast<const IN*>(p.dO);
  const XT* mg = reinterpret_cast<const XT*>(p.mat_ws) + ((int64_t)c * H + h) * kNumMats * kMatElems;
  const int64_t soff = ((int64_t)c * H + h) * DK * DV;

  // ---- per value block inputs, prefetched into registers one block ahead:
  //      V and dO rows (16-byte vectors), the clip mask rows, the four state
  //      blocks (fp32, 4 columns per vector) ----
  constexpr int kVR = kBVG * (int)sizeof(IN) / 16;            // vectors per V / dO row
  constexpr int kVPT = 2 * kChunk * kVR / kThreads;           // V + dO vectors per thread
  constexpr int kSPT = DK * (kBVG / 4) / kThreads;            // float4 per thread per state
  static_assert(kVPT >= 1 && kSPT >= 1, "block prefetch shape");
  uint4 pv[kVPT];
  uint4 pm;
  float4 ps[4][kSPT];
  auto prefetch = [&](int j0) {
#pragma unroll
    for (int u = 0; u < kVPT; ++u) {
      const int e = tid + u * kThreads, which = e / (kChunk * kVR), r = e % (kChunk * kVR);
      const int t = r / kVR, cv = r % kVR;
      const IN* src = (which ? dog : vg) + ((tok + t) * H + h) * (int64_t)DV + j0 +
                      cv * (16 / (int)sizeof(IN));
      pv[u] = t < len ? *reinterpret_cast<const uint4*>(src) : uint4{0, 0, 0, 0};
    }
    pm = uint4{0, 0, 0, 0};
    if (tid < len)
      pm = *reinterpret_cast<const uint4*>(p.ck_mask + ((tok + tid) * H + h) * (int64_t)DV + j0);
    const float* srcs[4] = {p.ck_S, p.ck_R, p.dS_ws, p.dR_ws};
#pragma unroll
    for (int u = 0; u < kSPT; ++u) {
      const int e = tid + u * kThreads, i = e / (kBVG / 4), qd = e % (kBVG / 4);
      const int64_t gi = soff + (int64_t)i * DV + j0 + 4 * qd;
#pragma unroll
      for (int m = 0; m < 4; ++m) ps[m][u] = *reinterpret_cast<const float4*>(srcs[m] + gi);
    }
  };
  prefetch(0);

  // ---- chunk-constant staging: K, Q (XT, row-major), matrices, gates ----
  {
    constexpr int kE = 16 / (int)sizeof(IN);                  // elements per vector
    constexpr int kKV = kChunk * DK / kE / kThreads;          // vectors per thread per matrix
    uint4 kv[kKV], qv[kKV];
#pragma unroll
    for (int u = 0; u < kKV; ++u) {
      const int e = tid + u * kThreads, t = e / (DK / kE), i = (e % (DK / kE)) * kE;
      const int64_t off = ((tok + t) * H + h) * (int64_t)DK + i;
      kv[u] = t < len ? *reinterpret_cast<const uint4*>(kg + off) : uint4{0, 0, 0, 0};
      qv[u] = t < len ? *reinterpret_cast<const uint4*>(qg + off) : uint4{0, 0, 0, 0};
    }
#pragma unroll
    for (int u = 0; u < kKV; ++u) {
      const int e = tid + u * kThreads, t = e / (DK / kE), i = (e % (DK / kE)) * kE;
      if constexpr (L::kBF) {   // bf16 -> fp16, 8 at a time
        const u16x8 a = __builtin_bit_cast(u16x8, kv[u]), b = __builtin_bit_cast(u16x8, qv[u]);
        f16x8 ka, qa;
#pragma unroll
        for (int x = 0; x < 8; ++x) { ka[x] = (f16)bf2f(a[x]); qa[x] = (f16)bf2f(b[x]); }
        *reinterpret_cast<f16x8*>(KX + t * L::kLdK + i) = ka;
        *reinterpret_cast<f16x8*>(QX + t * L::kLdK + i) = qa;
      } else {
        *reinterpret_cast<uint4*>(KX + t * L::kLdK + i) = kv[u];
        *reinterpret_cast<uint4*>(QX + t * L::kLdK + i) = qv[u];
      }
    }
  }
  const XT *mTS, *mMG, *mMP, *mTR, *mMR;
  int ldm;
  if constexpr (L::kMatsInLds) {
    XT* mats = reinterpret_cast<XT*>(smem + L::kMats);
    constexpr int kVecM = 16 / sizeof(XT);
    constexpr int kMV = 5 * kMatElems / kVecM / kThreads;   // vectors per thread
    uint4 mv[kMV];
#pragma unroll
    for (int u = 0; u < kMV; ++u) {
      const int e = tid + u * kThreads;
      mv[u] = *reinterpret_cast<const uint4*>(mg + e * kVecM);
    }
#pragma unroll
    for (int u = 0; u < kMV; ++u) {
      const int e = tid + u * kThreads;
      const int m = e / (kMatElems / kVecM), r = e % (kMatElems / kVecM);
      const int t = r / (kChunk / kVecM), s = (r % (kChunk / kVecM)) * kVecM;
      *reinterpret_cast<uint4*>(mats + (m * kChunk + t) * L::kLdX + s) = mv[u];
    }
    ldm = L::kLdX;
    mTS = mats + kMatTS * kChunk * L::kLdX;
    mMG = mats + kMatMG * kChunk * L::kLdX;
    mMP = mats + kMatMP * kChunk * L::kLdX;
    mTR = mats + kMatTR * kChunk * L::kLdX;
    mMR = mats + kMatMR * kChunk * L::kLdX;
  } else {
    ldm = kChunk;
    mTS = mg + kMatTS * kMatElems;
    mMG = mg + kMatMG * kMatElems;
    mMP = mg + kMatMP * kMatElems;
    mTR = mg + kMatTR * kMatElems;
    mMR = mg + kMatMR * kMatElems;
  }
  if (tid < kChunk) {
    const float* gb = p.gate_ws + ((int64_t)c * H + h) * kGateBlock;
    const int t = tid;
    const float gs = gb[t], gsl = gb[kChunk - 1], gsp = t > 0 ? gb[t - 1] : 0.f;
    const float gr = gb[64 + t], grl = gb[64 + kChunk - 1];
    gbt[t] = gb[128 + t];
    ggm[t] = gb[192 + t];
    egs[t] = __expf(gs);
    egsp[t] = __expf(gsp);
    egr[t] = __expf(gr);
    dls[t] = __expf(gsl - gs);
    dlr[t] = __expf(grl - gr);
    gsv[t] = gs;
    gspv[t] = gsp;
    grv[t] = gr;
    if (t == 0) {
      edge[0] = __expf(gsl);
      edge[1] = __expf(grl);
    }
  }

  // accumulators: dQ, dK rows of this wave; W1..W5 rows of this wave
  floatx4 dQ[IT], dK[IT], W1[4], W2[4], W3[4], W4[4], W5[4];
#pragma unroll
  for (int it = 0; it < IT; ++it) { dQ[it] = zero4(); dK[it] = zero4(); }
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    W1[st] = zero4(); W2[st] = zero4(); W3[st] = zero4(); W4[st] = zero4(); W5[st] = zero4();
  }
  float rb[4] = {0, 0, 0, 0}, rgm[4] = {0, 0, 0, 0}, rgs[4] = {0, 0, 0, 0};
  float rgsp[4] = {0, 0, 0, 0}, rgr[4] = {0, 0, 0, 0};
  float gsC = 0.f, grC = 0.f;   // gradients w.r.t. g_C, h_C (partial, this thread)
  const int trow0 = 16 * w;
  barrier_lds();   // staged K, Q, matrices and gates

  for (int j0 = 0; j0 < DV; j0 += kBVG) {
    // ---- this block's inputs from the prefetch registers into LDS; the
    //      state blocks scaled to fp16 ----
#pragma unroll
    for (int u = 0; u < kVPT; ++u) {
      const int e = tid + u * kThreads, which = e / (kChunk * kVR), r = e % (kChunk * kVR);
      const int t = r / kVR, cv = r % kVR, j = cv * (16 / (int)sizeof(IN));
      if (which == 0) {
        *reinterpret_cast<uint4*>(VB + t * kBVG + j) = pv[u];
      } else {
        const IN* x = reinterpret_cast<const IN*>(&pv[u]);
#pragma unroll
        for (int y = 0; y < 16 / (int)sizeof(IN); ++y)
          blk(kDBT)[(j + y) * L::kLdX + t] = from_f<XT>(to_f<IN>(x[y]));
      }
    }
    if (tid < kChunk) *reinterpret_cast<uint4*>(mask + tid * kBVG) = pm;
    float mx[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < kSPT; ++u) {
#pragma unroll
      for (int m = 0; m < 4; ++m)
        mx[m] = fmaxf(mx[m], fmaxf(fmaxf(fabsf(ps[m][u].x), fabsf(ps[m][u].y)),
                                   fmaxf(fabsf(ps[m][u].z), fabsf(ps[m][u].w))));
      // states at the chunk start times their end gradients (for g_C, h_C)
      gsC += edge[0] * (ps[0][u].x * ps[2][u].x + ps[0][u].y * ps[2][u].y +
                        ps[0][u].z * ps[2][u].z + ps[0][u].w * ps[2][u].w);
      grC += edge[1] * (ps[1][u].x * ps[3][u].x + ps[1][u].y * ps[3][u].y +
                        ps[1][u].z * ps[3][u].z + ps[1][u].w * ps[3][u].w);
    }
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const float wm = wave_max(mx[m]);
      if (lane == 0) red[w * 4 + m] = wm;
    }
    barrier_lds();
    float scl[4];   // power-of-two scale: value = scl * stored
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const float bmax = fmaxf(fmaxf(red[m], red[4 + m]), fmaxf(red[8 + m], red[12 + m]));
      float sc = 1.f;
      if constexpr (L::kBF) {
        if (bmax > 16384.f) {
          int ex;
          frexpf(bmax / 16384.f, &ex);
          sc = ldexpf(1.f, ex);
        }
      }
      scl[m] = sc;
    }
    {
      XT* dst[4] = {S0N, R0N, dS1N, dR1N};
#pragma unroll
      for (int u = 0; u < kSPT; ++u) {
        const int e = tid + u * kThreads, i = e / (kBVG / 4), qd = e % (kBVG / 4);
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const float inv = 1.f / scl[m];
          XT* d = dst[m] + i * L::kLdV + 4 * qd;
          d[0] = from_f<XT>(ps[m][u].x * inv);
          d[1] = from_f<XT>(ps[m][u].y * inv);
          d[2] = from_f<XT>(ps[m][u].z * inv);
          d[3] = from_f<XT>(ps[m][u].w * inv);
        }
      }
    }
    barrier_lds();
    if (j0 + kBVG < DV) prefetch(j0 + kBVG);

    // ---- A: state products, elementwise Y / dO copies ----
    floatx4 KS, QS, KR, QR, KdS, KdR;
    {
      KS = zero4(); QS = zero4(); KR = zero4(); QR = zero4(); KdS = zero4(); KdR = zero4();
      const XT* Kw = KX + trow0 * L::kLdK;
      const XT* Qw = QX + trow0 * L::kLdK;
      mma_with<M, DK, true, false>(KS, Kw, L::kLdK, S0N, L::kLdV);
      mma_with<M, DK, true, false>(QS, Qw, L::kLdK, S0N, L::kLdV);
      mma_with<M, DK, true, false>(KR, Kw, L::kLdK, R0N, L::kLdV);
      mma_with<M, DK, true, false>(QR, Qw, L::kLdK, R0N, L::kLdV);
      mma_with<M, DK, true, false>(KdS, Kw, L::kLdK, dS1N, L::kLdV);
      mma_with<M, DK, true, false>(KdR, Kw, L::kLdK, dR1N, L::kLdV);
      KS *= scl[0]; QS *= scl[0]; KR *= scl[1]; QR *= scl[1]; KdS *= scl[2]; KdR *= scl[3];
    }
    float vv[4], dob[4], yarg[4];
    {
      floatx4 y, dc, edb, edc;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = trow0 + acc_row(r), j = acc_col();
        vv[r] = to_f<IN>(VB[t * kBVG + j]);
        dob[r] = to_f<XT>(blk(kDBT)[j * L::kLdX + t]);
        yarg[r] = RDN ? vv[r] - egs[t] * KS[r] : vv[r];
        y[r] = gbt[t] * yarg[r];
        dc[r] = ggm[t] * dob[r];
        edb[r] = egs[t] * dob[r];
        edc[r] = egr[t] * dc[r];
      }
      if constexpr (RDN) {
        store_acc_t<XT>(blk(kYT) + trow0, L::kLdX, y);
      } else {
        floatx4 du;
#pragma unroll
        for (int r = 0; r < 4; ++r) du[r] = dls[trow0 + acc_row(r)] * y[r];
        store_acc_t<XT>(blk(kUT) + trow0, L::kLdX, y);
        store_acc_t<XT>(blk(kDUT) + trow0, L::kLdX, du);
      }
      store_acc_t<XT>(blk(kDCT) + trow0, L::kLdX, dc);
      store_acc_t<XT>(blk(kEDBT) + trow0, L::kLdX, edb);
      store_acc_t<XT>(blk(kEDCT) + trow0, L::kLdX, edc);
    }
    barrier_lds();

    // ---- B: U = T^S Y (RDN) ----
    floatx4 U;
    if constexpr (RDN) {
      U = zero4();
      mma_with<M, kChunk, true, true>(U, mTS + trow0 * ldm, ldm, blk(kYT), L::kLdX);
      floatx4 du;
#pragma unroll
      for (int r = 0; r < 4; ++r) du[r] = dls[trow0 + acc_row(r)] * U[r];
      store_acc_t<XT>(blk(kUT) + trow0, L::kLdX, U);
      store_acc_t<XT>(blk(kDUT) + trow0, L::kLdX, du);
      barrier_lds();
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) U[r] = gbt[trow0 + acc_row(r)] * vv[r];
    }

    // ---- C: residual and the R path's right-hand side ----
    float rr[4], yrarg[4];
    {
      floatx4 mgu = zero4(), y;
      mma_with<M, kChunk, true, true>(mgu, mMG + trow0 * ldm, ldm, blk(kUT), L::kLdX);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = trow0 + acc_row(r);
        const float x = vv[r] - egsp[t] * KS[r] - mgu[r];
        rr[r] = clip < 0.f ? x : fminf(fmaxf(x, -clip), clip);
        yrarg[r] = RDN ? rr[r] - egr[t] * KR[r] : rr[r];
        y[r] = ggm[t] * yrarg[r];
      }
      if constexpr (RDN) {
        store_acc_t<XT>(blk(kYT) + trow0, L::kLdX, y);
      } else {
        floatx4 du;
#pragma unroll
        for (int r = 0; r < 4; ++r) du[r] = dlr[trow0 + acc_row(r)] * y[r];
        store_acc_t<XT>(blk(kURT) + trow0, L::kLdX, y);
        store_acc_t<XT>(blk(kDURT) + trow0, L::kLdX, du);
      }
    }
    barrier_lds();

    // ---- D: UR = T^R YR (RDN) ----
    floatx4 UR;
    if constexpr (RDN) {
      UR = zero4();
      mma_with<M, kChunk, true, true>(UR, mTR + trow0 * ldm, ldm, blk(kYT), L::kLdX);
      floatx4 du;
#pragma unroll
      for (int r = 0; r < 4; ++r) du[r] = dlr[trow0 + acc_row(r)] * UR[r];
      store_acc_t<XT>(blk(kURT) + trow0, L::kLdX, UR);
      store_acc_t<XT>(blk(kDURT) + trow0, L::kLdX, du);
      barrier_lds();
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) UR[r] = ggm[trow0 + acc_row(r)] * rr[r];
    }

    // ---- E: correction read-out c, and dUR = e^{h_C-h} K dR1 + MR^T dc ----
    floatx4 cc = zero4(), dUR = zero4();
    mma_with<M, kChunk, true, true>(cc, mMR + trow0 * ldm, ldm, blk(kURT), L::kLdX);
    mma_with<M, kChunk, false, true>(dUR, mMR + trow0, ldm, blk(kDCT), L::kLdX);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = trow0 + acc_row(r);
      cc[r] += egr[t] * QR[r];
      dUR[r] += dlr[t] * KdR[r];
    }
    if constexpr (RDN) {
      store_acc_t<XT>(blk(kDURt) + trow0, L::kLdX, dUR);
      barrier_lds();
    }

    // ---- F: dYR, dX, dKR ----
    floatx4 dYR = dUR, dX, dKR;
    if constexpr (RDN) {
      dYR = zero4();
      mma_with<M, kChunk, false, true>(dYR, mTR + trow0, ldm, blk(kDURt), L::kLdX);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = trow0 + acc_row(r), j = acc_col();
      dX[r] = mask[t * kBVG + j] ? ggm[t] * dYR[r] : 0.f;
      dKR[r] = RDN ? -ggm[t] * egr[t] * dYR[r] : 0.f;
      // gamma: o = b + gamma c, and (RDN) YR = gamma (r - e^h KR) / (RLA) UR = gamma r
      rgm[r] += dob[r] * cc[r] + dYR[r] * yrarg[r];
      // h_t through e^{h_t} in c and (RDN) in YR; h_t, h_C through the R update
      const float kdu = KdR[r] * UR[r] * dlr[t];
      rgr[r] += ggm[t] * dob[r] * egr[t] * QR[r] - kdu;
      if constexpr (RDN) rgr[r] += -ggm[t] * egr[t] * dYR[r] * KR[r];
      grC += kdu;
    }
    store_acc_t<XT>(blk(kDXT) + trow0, L::kLdX, dX);
    store_acc_t<XT>(blk(kDKRT) + trow0, L::kLdX, dKR);
    store_acc_t<XT>(blk(kDYRT) + trow0, L::kLdX, dYR);
    barrier_lds();

    // ---- G: dU = e^{g_C-g} K dS1 + MP^T dO - MG^T dX ----
    floatx4 dU = zero4();
    {
      floatx4 b = zero4();
      mma_with<M, kChunk, false, true>(dU, mMP + trow0, ldm, blk(kDBT), L::kLdX);
      mma_with<M, kChunk, false, true>(b, mMG + trow0, ldm, blk(kDXT), L::kLdX);
#pragma unroll
      for (int r = 0; r < 4; ++r) dU[r] += dls[trow0 + acc_row(r)] * KdS[r] - b[r];
    }
    if constexpr (RDN) {
      store_acc_t<XT>(blk(kDUt) + trow0, L::kLdX, dU);
      barrier_lds();
    }

    // ---- H: dY, dKS, dV, row sums of the S path ----
    {
      floatx4 dY = dU, dKS;
      if constexpr (RDN) {
        dY = zero4();
        mma_with<M, kChunk, false, true>(dY, mTS + trow0, ldm, blk(kDUt), L::kLdX);
      }
      OT* dvg = reinterpret_cast<OT*>(p.dv);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = trow0 + acc_row(r);
        dKS[r] = -egsp[t] * dX[r] - (RDN ? gbt[t] * egs[t] * dY[r] : 0.f);
        if (t < len)
          dvg[((tok + t) * H + h) * (int64_t)DV + j0 + acc_col()] = from_f<OT>(dX[r] + gbt[t] * dY[r]);
        rb[r] += dY[r] * yarg[r];
        const float kdu = KdS[r] * U[r] * dls[t];
        rgs[r] += egs[t] * dob[r] * QS[r] - kdu;
        if constexpr (RDN) rgs[r] += -gbt[t] * egs[t] * dY[r] * KS[r];
        rgsp[r] += -egsp[t] * dX[r] * KS[r];
        gsC += kdu;
      }
      if constexpr (RDN) store_acc_t<XT>(blk(kDYT) + trow0, L::kLdX, dY);
      store_acc_t<XT>(blk(kDKST) + trow0, L::kLdX, dKS);
    }
    barrier_lds();

    // ---- I: contractions over this value block ----
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int io = it * 16 * L::kLdV;
      floatx4 t0 = zero4(), t1 = zero4(), t2 = zero4(), t3 = zero4(), t4 = zero4(), t5 = zero4();
      mma_with<M16, kBVG, false, true>(t0, blk(kEDBT) + trow0, L::kLdX, S0N + io, L::kLdV);
      mma_with<M16, kBVG, false, true>(t1, blk(kEDCT) + trow0, L::kLdX, R0N + io, L::kLdV);
      mma_with<M16, kBVG, false, true>(t2, blk(kDUT) + trow0, L::kLdX, dS1N + io, L::kLdV);
      mma_with<M16, kBVG, false, true>(t3, blk(kDURT) + trow0, L::kLdX, dR1N + io, L::kLdV);
      mma_with<M16, kBVG, false, true>(t4, blk(kDKST) + trow0, L::kLdX, S0N + io, L::kLdV);
      if constexpr (RDN) mma_with<M16, kBVG, false, true>(t5, blk(kDKRT) + trow0, L::kLdX, R0N + io, L::kLdV);
      dQ[it] += scl[0] * t0 + scl[1] * t1;
      dK[it] += scl[2] * t2 + scl[3] * t3 + scl[0] * t4 + scl[1] * t5;
    }
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      mma_with<M16, kBVG, false, false>(W1[st], blk(kDBT) + trow0, L::kLdX, blk(kUT) + 16 * st, L::kLdX);
      mma_with<M16, kBVG, false, false>(W2[st], blk(kDCT) + trow0, L::kLdX, blk(kURT) + 16 * st, L::kLdX);
      mma_with<M16, kBVG, false, false>(W3[st], blk(kDXT) + trow0, L::kLdX, blk(kUT) + 16 * st, L::kLdX);
      if constexpr (RDN) {
        mma_with<M16, kBVG, false, false>(W4[st], blk(kDYT) + trow0, L::kLdX, blk(kUT) + 16 * st, L::kLdX);
        mma_with<M16, kBVG, false, false>(W5[st], blk(kDYRT) + trow0, L::kLdX, blk(kURT) + 16 * st, L::kLdX);
      }
    }
    barrier_lds();
  }

  // ---- row sums of the value loop ----
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const float a = sum16(rb[r]), b = sum16(rgm[r]), s1 = sum16(rgs[r]), s2 = sum16(rgsp[r]),
                s3 = sum16(rgr[r]);
    if ((lane & 15) == 0) {
      const int t = trow0 + acc_row(r);
      rows[rBeta * kChunk + t] = a;
      rows[rGamma * kChunk + t] = b;
      rows[rGS * kChunk + t] = s1;
      rows[rGSP * kChunk + t] = s2;
      rows[rGR * kChunk + t] = s3;
    }
  }
  {
    const float a = wave_sum(gsC), b = wave_sum(grC);
    if (lane == 0) { red[16 + w] = a; red[20 + w] = b; }
  }

  // ---- E1: Gram / scores, decay matrices, dP, dG and the Z matrices ----
  XT* dPm = reinterpret_cast<XT*>(smem + L::kDPG);
  XT* dGm = dPm + kChunk * L::kLdX;
  float* ZS = reinterpret_cast<float*>(smem + L::kZ);
  float* ZP = ZS + kChunk * L::kLdZ;
  float* ZR = ZP + kChunk * L::kLdZ;
  barrier_lds();   // matrices / states / blocks are dead beyond this point
  {
    float pb[4] = {0, 0, 0, 0}, pg[4] = {0, 0, 0, 0};
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      floatx4 G = zero4(), P = zero4();
      mma_with<M, DK, true, true>(G, KX + trow0 * L::kLdK, L::kLdK, KX + 16 * st * L::kLdK, L::kLdK);
      mma_with<M, DK, true, true>(P, QX + trow0 * L::kLdK, L::kLdK, KX + 16 * st * L::kLdK, L::kLdK);
      floatx4 dp, dg;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = trow0 + acc_row(r), s = 16 * st + acc_col();
        const bool lower = s < t, diag = s <= t;
        const float es = __expf(fminf(gsv[t] - gsv[s], 0.f));
        const float ep = __expf(fminf(gspv[t] - gsv[s], 0.f));
        const float er = __expf(fminf(grv[t] - grv[s], 0.f));
        const float dAs = RDN ? -W4[st][r] : 0.f, dAr = RDN ? -W5[st][r] : 0.f;
        dp[r] = (lower ? es * W1[st][r] : 0.f) + (diag ? er * W2[st][r] : 0.f);
        dg[r] = lower ? (-ep * W3[st][r] + gbt[t] * es * dAs + ggm[t] * er * dAr) : 0.f;
        ZS[t * L::kLdZ + s] = lower ? es * (P[r] * W1[st][r] + gbt[t] * G[r] * dAs) : 0.f;
        ZP[t * L::kLdZ + s] = lower ? -ep * G[r] * W3[st][r] : 0.f;
        ZR[t * L::kLdZ + s] = (diag ? er * P[r] * W2[st][r] : 0.f) + (lower ? ggm[t] * er * G[r] * dAr : 0.f);
        pb[r] += lower ? dAs * es * G[r] : 0.f;
        pg[r] += lower ? dAr * er * G[r] : 0.f;
      }
      store_acc<XT>(dPm + trow0 * L::kLdX + 16 * st, L::kLdX, dp);
      store_acc<XT>(dGm + trow0 * L::kLdX + 16 * st, L::kLdX, dg);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float a = sum16(pb[r]), b = sum16(pg[r]);
      if ((lane & 15) == 0) {
        const int t = trow0 + acc_row(r);
        rows[rBeta * kChunk + t] += a;
        rows[rGamma * kChunk + t] += b;
      }
    }
  }
  barrier_lds();

  // ---- E2: gate gradients (wave 0) ----
  if (tid < kChunk) {
    const int t = tid;
    float rzs = 0.f, czs = 0.f, rzp = 0.f, czp = 0.f, rzr = 0.f, czr = 0.f, rzp1 = 0.f;
    for (int s = 0; s < kChunk; ++s) {
      rzs += ZS[t * L::kLdZ + s];
      czs += ZS[s * L::kLdZ + t];
      rzp += ZP[t * L::kLdZ + s];
      czp += ZP[s * L::kLdZ + t];
      rzr += ZR[t * L::kLdZ + s];
      czr += ZR[s * L::kLdZ + t];
      if (t + 1 < kChunk) rzp1 += ZP[(t + 1) * L::kLdZ + s];
    }
    const float gsC_all = red[16] + red[17] + red[18] + red[19];
    const float grC_all = red[20] + red[21] + red[22] + red[23];
    float dgs = rows[rGS * kChunk + t] + rzs - czs - czp +
                (t + 1 < kChunk ? rows[rGSP * kChunk + t + 1] + rzp1 : 0.f) +
                (t == kChunk - 1 ? gsC_all : 0.f);
    float dgr = rows[rGR * kChunk + t] + rzr - czr + (t == kChunk - 1 ? grC_all : 0.f);
    (void)rzp;
    // suffix sums over the chunk: d log a_j = sum_{t >= j} d g_t
    float ss = dgs, sr = dgr;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float a = __shfl_down(ss, off, 64), b = __shfl_down(sr, off, 64);
      if (t + off < 64) { ss += a; sr += b; }
    }
    if (t < len) {
      const int64_t gi = (tok + t) * H + h;
      const float as = p.alpha_s[gi], ar = p.alpha_r[gi];
      p.dalpha_s[gi] = as >= 1.17549435e-38f ? ss / as : 0.f;
      p.dalpha_r[gi] = ar >= 1.17549435e-38f ? sr / ar : 0.f;
      p.dbeta[gi] = rows[rBeta * kChunk + t];
      p.dgamma[gi] = rows[rGamma * kChunk + t];
    }
  }

  // ---- E2: dQ += dP K, dK += dP^T Q + dG K + dG^T K ----
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const XT* Ki = KX + 16 * it;
    const XT* Qi = QX + 16 * it;
    mma_with<M, kChunk, true, false>(dQ[it], dPm + trow0 * L::kLdX, L::kLdX, Ki, L::kLdK);
    mma_with<M, kChunk, false, false>(dK[it], dPm + trow0, L::kLdX, Qi, L::kLdK);
    mma_with<M, kChunk, true, false>(dK[it], dGm + trow0 * L::kLdX, L::kLdX, Ki, L::kLdK);
    mma_with<M, kChunk, false, false>(dK[it], dGm + trow0, L::kLdX, Ki, L::kLdK);
  }
  OT* dqg = reinterpret_cast<OT*>(p.dq);
  OT* dkg = reinterpret_cast<OT*>(p.dk);
#pragma unroll
  for (int it = 0; it < IT; ++it)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = trow0 + acc_row(r);
      if (t < len) {
        const int64_t gi = ((tok + t) * H + h) * (int64_t)DK + 16 * it + acc_col();
        dqg[gi] = from_f<OT>(dQ[it][r]);
        dkg[gi] = from_f<OT>(dK[it][r]);
      }
    }
}

template <typename IN, int DK, bool RDN, typename OT>
hipError_t launch_grad_t(const OpParams& p, hipStream_t stream) {
  typedef GradLayout<IN, DK, RDN> L;
  auto kern = bwd_grad_kernel<IN, DK, RDN, OT>;
  hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, L::kBytes);
  if (err != hipSuccess) return err;
  if (p.max_chunks == 0) return hipSuccess;
  hipLaunchKernelGGL(kern, dim3(p.max_chunks, p.H), dim3(kThreads), L::kBytes, stream, p);
  return hipGetLastError();
}

template <typename IN, int DK, typename OT>
hipError_t launch_grad_dk(const OpParams& p, hipStream_t s) {
  return p.rdn ? launch_grad_t<IN, DK, true, OT>(p, s) : launch_grad_t<IN, DK, false, OT>(p, s);
}

}  // namespace

hipError_t launch_bwd_grad(const OpParams& p, bool bf16, hipStream_t stream) {
  if (bf16) {
    if (p.out_bf16)
      return p.DK == 128 ? launch_grad_dk<u16, 128, u16>(p, stream) : launch_grad_dk<u16, 64, u16>(p, stream);
    return p.DK == 128 ? launch_grad_dk<u16, 128, float>(p, stream) : launch_grad_dk<u16, 64, float>(p, stream);
  }
  return launch_grad_dk<float, 64, float>(p, stream);
}

}  // namespace rla
