// Chunk-parallel gradient contractions: one 256-thread workgroup per (chunk,
// head).  The forward scan saved, per chunk, the start states S0, R0 and the
// blocks U, UR and r (clipped residual); the reverse scan saved the end-state
// gradients dS1, dR1 and the blocks dX, dY, dYR (RLA: dU, dUR in the dY, dYR
// places) and already wrote dv.  What is left are contractions over the value
// dimension plus chunk-local products; nothing of the scans is recomputed.
//
// With E^S, E', E^R the decay matrices of prep.hip and the row scalings e^g,
// e^{g_{t-1}}, e^h, dls = e^{g_C-g}, dlr = e^{h_C-h}:
//   F1 = dO S0^T, F2 = dO R0^T, FK1 = dX S0^T, FK2 = dY S0^T, FK3 = dYR R0^T,
//   FK4 = U dS1^T, FK5 = UR dR1^T                      (RLA: no FK2, FK3)
//   dQ = e^g F1 + gamma e^h F2 + dP K
//   dK = -e^{g_{t-1}} FK1 - b e^g FK2 - gamma e^h FK3 + dls FK4 + dlr FK5
//        + dP^T Q + (dG + dG^T) K
//   W1 = dO U^T, W2 = dO UR^T, W3 = dX U^T, W4 = dY U^T, W5 = dYR UR^T
//   dP = E^S (.) W1 (.) L- + diag(gamma) E^R (.) W2 (.) L
//   dG = [-E' (.) W3 - diag(b) E^S (.) W4 - diag(gamma) E^R (.) W5] (.) L-
// (dA^S = -W4 and dA^R = -W5 are the gradients of the triangular systems.)
// Variants: the ungated output weights its S0 and U read-out by e^{g_{t-1}}
// (E' in dP, F1 with e^{g_{t-1}}: their gate terms move to g_{t-1}) and drops
// gamma from the output (dQ's F2 term, dP's W2 term and dgamma's output
// terms); the decayed residual weights FK1 and W3 by e^{g} and E^S (their
// gate terms move from g_{t-1} to g_t).  The log-cosh residual changes
// nothing here: the reverse scan applied its slope to dX.
// The gate gradients need per-token sums over the value dimension of
// products of a backward and a forward quantity.  Those that involve a state
// are row-dots of Q or K with the F matrices above, e.g.
// sum_j dO_tj (Q S0)_tj = sum_i Q_ti F1_ti, so they come out of the same
// contractions; sum_j dY_tj V_tj and sum_j dYR_tj r_tj (RLA: dU V, dUR r) are
// taken elementwise.  d log a over a chunk is the suffix sum of the gradients
// of the cumulative sums g_t, h_t.
//
// Work split: d_k / 16 waves; wave w owns d_k tile w (16 state rows) for the
// F contractions, dQ and dK, over all 64 tokens; the 10 lower 16 x 16 tiles
// of the chunk's token x token matrices are dealt round-robin for W,
// G = K K^T, P = Q K^T, dP and dG.  State rows stream from HBM (fp32) straight into MFMA B
// fragments; the token blocks are moved into LDS by LDS-DMA.
//
// Precision (bf16 inputs): fp16 MFMA operands with fp32 accumulation.  The
// scans store the states in fp16 scaled by a power of two per (16 rows, 32
// columns); here each row is brought to one scale (its largest) when loaded,
// and a contraction multiplies its result by that scale.  The reverse scan's
// blocks and gradient states carry the (sequence, head)'s upstream-gradient
// scale 2^e (grad_scale); dO is multiplied by it here too, so everything is in
// one scale, and every gradient written is multiplied by 2^-e.
#include <type_traits>

#include "kernels.hpp"

namespace rla {

namespace {

// token blocks in LDS
enum { bDO = 0, bU, bUR, bDX, bDY, bDYR, kNumTokBlk };
// per-token sums (LDS, fp32, one set per wave, each entry written once so
// that plain stores suffice): direct gate terms of g_t, g_{t-1}, h_t, beta,
// gamma from the F contractions; row / column sums of the Z matrices and the
// beta / gamma terms of the decay-matrix products
enum { sGS = 0, sGSP, sGR, sB, sGM, sZRS, sZCS, sZRP, sZCP, sZRR, sZCR, sZB, sZGM, kNumSums };

template <typename IN, int DK, int DV>
struct GradLayout {
  static constexpr bool kBF = sizeof(IN) == 2;
  static constexpr int kNW = DK / 16;        // one wave per 16-row d_k tile
  static constexpr int kNT = 64 * kNW;       // threads per workgroup
  typedef typename std::conditional<kBF, f16, float>::type XT;
  typedef Tile<XT, DK> TK;    // K, Q rows
  typedef Tile<XT, DV> TV;    // token blocks
  static constexpr int kLdP = kChunk + (kBF ? 8 : 4);   // padded rows of dP, dP^T, dG+dG^T, K^T, Q^T
  static constexpr int kK = 0;
  static constexpr int kQ = kK + kChunk * TK::kRowB;
  static constexpr int kBlk = kQ + kChunk * TK::kRowB;
  static constexpr int kBlkBytes = kChunk * TV::kRowB;
  // after the W / G / P products the token blocks are dead; their region then
  // holds dP, dP^T, dG + dG^T ([64][kLdP]) and K^T, Q^T ([DK][kLdP])
  static constexpr int kDP = kBlk;
  static constexpr int kDPT = kDP + kChunk * kLdP * (int)sizeof(XT);
  static constexpr int kDG = kDPT + kChunk * kLdP * (int)sizeof(XT);
  static constexpr int kKT = kDG + kChunk * kLdP * (int)sizeof(XT);
  static constexpr int kQT = kKT + DK * kLdP * (int)sizeof(XT);
  static constexpr int kOvlEnd = kQT + DK * kLdP * (int)sizeof(XT);
  static constexpr int kBlkEnd = kBlk + kNumTokBlk * kBlkBytes;
  // the per-token sums totalled over the waves ([kNumSums][64]), written
  // when the token blocks are dead: in place of K^T (16-bit operands, which
  // read K, Q transposed instead) or past the overlay
  static constexpr int kTot = kBF ? kKT : kOvlEnd;
  static constexpr int kGates = kBlkEnd > kOvlEnd ? kBlkEnd : kOvlEnd;
  static_assert(kTot + kNumSums * kChunk * 4 <= kGates, "totals inside the dead token blocks");
  static constexpr int kNumGateArrays = 11;
  static constexpr int kSums = kGates + kNumGateArrays * kChunk * 4;
  static constexpr int kElem = kSums + kNW * kNumSums * kChunk * 4;  // per-wave sums
  static constexpr int kRed = kElem + 2 * kChunk * 4;   // elementwise beta / gamma sums
  static constexpr int kBytes = kRed + 16 * 4;
  static_assert(kBytes <= 160 * 1024, "gradient kernel LDS");
};

__device__ __forceinline__ float wave_sum(float x) {
  x = group_sum<16>(x);
  x += __shfl_xor(x, 16, 64);
  x += __shfl_xor(x, 32, 64);
  return x;
}

// Per-wave per-token sums in LDS, written branch-free: all lanes that hold
// the same sum store the same value to the same address.
// Row sums of a tile quantity (lane: rows 4*(lane>>4)+r) into dst[t0 + row],
// by a transpose-reduce: exchanges with lanes c ^ 1 and c ^ 2 leave lane c
// (c = lane % 16) with the sum over its quad of row 2 (c & 1) + ((c >> 1) & 1);
// rotations by 8 and then 4 inside the 16-lane row add the four quads (after
// the first the values repeat with period 8, so the four lanes of a row end
// with the same bits and store the same value).
__device__ __forceinline__ void put_rows(float* dst, int t0, const float (&v)[4]) {
  const int lane = threadIdx.x & 63;
  const bool b0 = lane & 1, b1 = lane & 2;
  const float x0 = (b0 ? v[2] : v[0]) + dpp<0xB1>(b0 ? v[0] : v[2]);   // quad_perm [1,0,3,2]
  const float x1 = (b0 ? v[3] : v[1]) + dpp<0xB1>(b0 ? v[1] : v[3]);
  float y = (b1 ? x1 : x0) + dpp<0x4E>(b1 ? x0 : x1);                  // quad_perm [2,3,0,1]
  y += dpp<0x128>(y);   // row_ror:8
  y += dpp<0x124>(y);   // row_ror:4
  dst[t0 + 4 * (lane >> 4) + 2 * (lane & 1) + ((lane >> 1) & 1)] = y;
}

// Column sums of a tile quantity (lane: column lane & 15) into dst[s0 + column].
__device__ __forceinline__ void put_cols(float* dst, int s0, const float (&v)[4]) {
  float s = v[0] + v[1] + v[2] + v[3];
  s += __shfl_xor(s, 16, 64);
  s += __shfl_xor(s, 32, 64);
  dst[s0 + (threadIdx.x & 15)] = s;
}

// VAR: an instance that reads the variant flags and qk_f16 (the default
// instance compiles them away)
template <typename IN, int DK, int DV, bool RDN, typename OT, bool VAR>
__global__ __launch_bounds__(64 * (DK / 16)) void bwd_grad_kernel(OpParams p) {
  typedef GradLayout<IN, DK, DV> L;
  constexpr int NW = L::kNW, NT = L::kNT;
  typedef typename L::XT XT;
  typedef typename L::TK TK;
  typedef PadRows<XT, kChunk, L::kLdP - kChunk> TDP;   // dP [64][kLdP]
  typedef typename L::TV TV;
  typedef Mfma<XT> M;
  typedef typename M::frag Frag;
  constexpr bool BF = L::kBF;
  constexpr int KSV = DV / M::kStep;   // k-steps over the value dimension
  constexpr int KSK = DK / M::kStep;   // k-steps over d_k
  constexpr int KSC = kChunk / M::kStep;
  constexpr int kIT = DK / 16 / NW;    // d_k tiles per wave
  static_assert(sizeof(IN) == sizeof(XT), "bf16 inputs pair with fp16 operands, fp32 with fp32");
  constexpr int kE = 16 / (int)sizeof(IN);   // elements per 16-byte vector
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* Kl = smem + L::kK;
  unsigned char* Ql = smem + L::kQ;
  auto tokblk = [&](int b) { return smem + L::kBlk + b * L::kBlkBytes; };
  XT* dPm = reinterpret_cast<XT*>(smem + L::kDP);
  XT* dPTm = reinterpret_cast<XT*>(smem + L::kDPT);
  XT* dGm = reinterpret_cast<XT*>(smem + L::kDG);
  XT* KTm = reinterpret_cast<XT*>(smem + L::kKT);
  XT* QTm = reinterpret_cast<XT*>(smem + L::kQT);
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
  const int vf = VAR ? p.vflags : 0;
  const bool ung = (vf & kVarUngated) != 0, dec = (vf & kVarDecayed) != 0;
  const float* eqb = ung ? egsp : egs;   // S0 factor of the base read-out
  const float* ekp = dec ? egs : egsp;   // S0 factor of the residual
  float* sums = reinterpret_cast<float*>(smem + L::kSums);   // [wave][kNumSums][64]
  float* esum = reinterpret_cast<float*>(smem + L::kElem);   // [2][64]: dY.V, dYR.r
  float* red = reinterpret_cast<float*>(smem + L::kRed);

  // heads vary fastest over consecutive workgroups, which then read one
  // contiguous stretch of the token rows (every head of the chunk)
  const int h = blockIdx.x, c = blockIdx.y, tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  float* wsum = sums + w * kNumSums * kChunk;   // this wave's sums
  auto sum_row = [&](int q) { return wsum + q * kChunk; };
  ChunkInfo ci;
  if (!chunk_info(p.st, c, ci)) return;
  const int H = p.H, len = ci.len;
  const int64_t tok = ci.tok;
  // upstream-gradient scale of this (sequence, head) (a power of two) and its inverse
  const float sig = p.grad_scale ? p.grad_scale[(int64_t)ci.seq * H + h] : 1.f;
  const float isig = 1.f / sig;

  const IN* qg = reinterpret_cast<const IN*>(p.q);
  const IN* kg = reinterpret_cast<const IN*>(p.k);
  const IN* vg = reinterpret_cast<const IN*>(p.v);
  const IN* dog = reinterpret_cast<const IN*>(p.dO);
  const XT* fb = reinterpret_cast<const XT*>(p.fwd_blk);
  const XT* bb = reinterpret_cast<const XT*>(p.bwd_blk);
  const int64_t soff = ((int64_t)c * H + h) * DK * DV;

  // ---------------- phase 0: staging ----------------
  // A state's rows i0 .. i0+15 as MFMA B fragments (row = lane & 15), with
  // the power-of-two scale of each (16-row tile, 32-column k-step) for fp16
  // states.
  // The row's fp16 blocks are brought to one scale, the largest of its blocks
  // (power-of-two factors <= 1, applied in fp16): a block 2^10 or more below
  // the row's largest loses only entries under 2^-14 of that scale, far below
  // what fp16 operands resolve in the contraction.
  struct StateRows {
    Frag fr[KSV];
    float sc;         // the row's scale
  };
  const void* srcs[4] = {p.ck_S, p.ck_R, p.dS_ws, p.dR_ws};
  const float* scs[4] = {p.ck_S_sc, p.ck_R_sc, p.dS_sc, p.dR_sc};
  const int64_t sco = ((int64_t)c * H + h) * (DK / 16) * (DV / 32);
  auto load_rows = [&](StateRows& x, int st, int i0) {
    const int i = i0 + (lane & 15);
    if constexpr (BF) {
      // blocked layout [DV / 32][DK][32]: k-step ks is column block ks
      static_assert(M::kStep == 32, "one 32-column block per k-step");
      // the state's uniform base plus a 32-bit lane offset (scalar-base loads)
      const f16* rowp = reinterpret_cast<const f16*>(srcs[st]) + soff;
      const uint32_t ro = (uint32_t)(i * 32 + 8 * (lane >> 4));
      const float* scp = scs[st] + sco + (i0 >> 4) * (DV / 32);
      float sc[KSV], mx = 0.f;
#pragma unroll
      for (int ks = 0; ks < KSV; ++ks) {
        x.fr[ks] = *reinterpret_cast<const Frag*>(rowp + ro + ks * DK * 32);
        sc[ks] = scp[ks];
        mx = fmaxf(mx, sc[ks]);
      }
      // sc / mx: exact power of two <= 1 (from the exponent bits; f16 0 below 2^-24)
      const uint32_t emx = __float_as_uint(mx) >> 23;
#pragma unroll
      for (int ks = 0; ks < KSV; ++ks) {
        const int d = (int)(__float_as_uint(sc[ks]) >> 23) - (int)emx;   // <= 0
        const f16 f = d < -24 ? (f16)0.f : (f16)__uint_as_float((uint32_t)(127 + d) << 23);
        x.fr[ks] = x.fr[ks] * f;
      }
      x.sc = mx;
    } else {
      const float* rowp = reinterpret_cast<const float*>(srcs[st]) + soff + (int64_t)i * DV;
#pragma unroll
      for (int ks = 0; ks < KSV; ++ks) {
        x.fr[ks] = rowp[ks * M::kStep + (lane >> 4)];
      }
      x.sc = 1.f;
    }
  };
  // Every global load of the staging is issued at once: K, Q, dO rows and
  // the gate block (converted / exponentiated before the barrier), the V and
  // r rows (the elementwise sums) and the token blocks' LDS-DMA.  The
  // compiler's waits for register loads issued alongside an LDS-DMA are full
  // drains, so the first state rows are issued after the conversions and the
  // drain: their latency then overlaps the barrier and the W / G / P products.
  constexpr int kKV = kChunk * DK / kE / NT;
  constexpr int kOV = kChunk * DV / kE / NT;
  // Rows past the chunk's end (len >= 1) are read at the last row and zeroed
  // where they are used: unconditional loads keep the waits for them at
  // their uses.
  auto in_row = [&](int t) { return t < len ? t : len - 1; };
  uint4 kv[kKV], qv[kKV], ov[kOV];
#pragma unroll
  for (int u = 0; u < kKV; ++u) {
    const int e = tid + u * NT, t = in_row(e / (DK / kE)), i = (e % (DK / kE)) * kE;
    const int64_t off = (tok * H + h) * (int64_t)DK + (uint32_t)(t * H * DK + i);
    kv[u] = *reinterpret_cast<const uint4*>(kg + off);
    qv[u] = *reinterpret_cast<const uint4*>(qg + off);
  }
#pragma unroll
  for (int u = 0; u < kOV; ++u) {
    const int e = tid + u * NT, t = in_row(e / (DV / kE)), j = (e % (DV / kE)) * kE;
    ov[u] = *reinterpret_cast<const uint4*>(dog + (tok * H + h) * (int64_t)DV + (uint32_t)(t * H * DV + j));
  }
  // this token's decay inputs for the gate gradients of wave 0 (lane = token),
  // loaded now so that their latency is not left to the kernel's end
  float a_s = 0.f, a_r = 0.f;
  if (w == 0) {
    const int64_t gi = tok * H + h + (uint32_t)(in_row(lane) * H);
    a_s = p.alpha_s[gi];
    a_r = p.alpha_r[gi];
  }
  // the gate block (every wave reads it; wave 0 stores the derived arrays)
  const float* gb = p.gate_ws + ((int64_t)c * H + h) * kGateBlock;
  const float gs = gb[lane], gsl = gb[kChunk - 1], gspr = gb[lane > 0 ? lane - 1 : 0];
  const float gr = gb[64 + lane], grl = gb[64 + kChunk - 1];
  const float gbe = gb[128 + lane], ggme = gb[192 + lane];
  dma_tile64<TV, NW>(fb + blk_off(c, h, H, 0, DV), tokblk(bU));
  dma_tile64<TV, NW>(fb + blk_off(c, h, H, 1, DV), tokblk(bUR));
  dma_tile64<TV, NW>(bb + blk_off(c, h, H, 0, DV), tokblk(bDX));
  dma_tile64<TV, NW>(bb + blk_off(c, h, H, 1, DV), tokblk(bDY));
  dma_tile64<TV, NW>(bb + blk_off(c, h, H, 2, DV), tokblk(bDYR));

  // V and r rows for the elementwise sums (consumed after the staging barrier)
  constexpr int kVV = kChunk * DV / kE / NT;
  uint4 vrow[kVV], rrow[kVV];
#pragma unroll
  for (int u = 0; u < kVV; ++u) {
    const int e = tid + u * NT, t = e / (DV / kE), j = (e % (DV / kE)) * kE;
    vrow[u] = *reinterpret_cast<const uint4*>(vg + (tok * H + h) * (int64_t)DV + (uint32_t)(in_row(t) * H * DV + j));
    rrow[u] = *reinterpret_cast<const uint4*>(fb + blk_off(c, h, H, 2, DV) + (uint32_t)(t * DV + j));
  }
  // K, Q, dO rows: converted to the operand type (dO multiplied by the
  // upstream-gradient scale), stored swizzled
  {
    auto conv = [&](uint4 x, float scale) -> uint4 {
      if constexpr (BF) {
        const u16x8 a = __builtin_bit_cast(u16x8, x);
        f16x8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (f16)(bf2f(a[e]) * scale);
        return __builtin_bit_cast(uint4, o);
      } else {
        return x;
      }
    };
#pragma unroll
    for (int u = 0; u < kKV; ++u) {
      const int e = tid + u * NT, t = e / (DK / kE), i = (e % (DK / kE)) * kE;
      if (VAR && p.qk_f16) {   // the pre-processing's fp16 rows
        *reinterpret_cast<uint4*>(Kl + TK::off(t, i)) = keep_if(kv[u], t < len);
        *reinterpret_cast<uint4*>(Ql + TK::off(t, i)) = keep_if(qv[u], t < len);
      } else {
        *reinterpret_cast<uint4*>(Kl + TK::off(t, i)) = conv(keep_if(kv[u], t < len), 1.f);
        *reinterpret_cast<uint4*>(Ql + TK::off(t, i)) = conv(keep_if(qv[u], t < len), 1.f);
      }
    }
#pragma unroll
    for (int u = 0; u < kOV; ++u) {
      const int e = tid + u * NT, t = e / (DV / kE), j = (e % (DV / kE)) * kE;
      *reinterpret_cast<uint4*>(tokblk(bDO) + TV::off(t, j)) = conv(keep_if(ov[u], t < len), sig);
    }
  }
  if (tid < kChunk) {
    const int t = tid;
    const float gsp = t > 0 ? gspr : 0.f;
    gbt[t] = gbe;
    ggm[t] = ggme;
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
  for (int e = tid; e < NW * kNumSums * kChunk; e += NT) sums[e] = 0.f;
  wait_vmem();   // this wave's DMAs have landed (published by the barrier)
  asm volatile("" ::: "memory");
  StateRows rowA, rowB;
  load_rows(rowA, 0, 16 * w);
  load_rows(rowB, 2, 16 * w);
  barrier_lds();

  // elementwise sums: dY . V (RLA: dU . V) for beta, dYR . r (RLA: dUR . r) for gamma
  {
    constexpr int kPerRow = DV / kE;   // threads sharing a row
#pragma unroll
    for (int u = 0; u < kVV; ++u) {
      const int e = tid + u * NT, t = e / kPerRow, j = (e % kPerRow) * kE;
      const uint4 dy = *reinterpret_cast<const uint4*>(tokblk(bDY) + TV::off(t, j));
      const uint4 dyr = *reinterpret_cast<const uint4*>(tokblk(bDYR) + TV::off(t, j));
      const XT* a = reinterpret_cast<const XT*>(&dy);
      const XT* b = reinterpret_cast<const XT*>(&dyr);
      const uint4 vr = keep_if(vrow[u], t < len);
      const IN* x = reinterpret_cast<const IN*>(&vr);
      const XT* y = reinterpret_cast<const XT*>(&rrow[u]);
      float s1 = 0.f, s2 = 0.f;
#pragma unroll
      for (int k = 0; k < kE; ++k) {
        s1 += to_f<XT>(a[k]) * to_f<IN>(x[k]);
        s2 += to_f<XT>(b[k]) * to_f<XT>(y[k]);
      }
      s1 = group_sum<kPerRow>(s1);
      s2 = group_sum<kPerRow>(s2);
      esum[t] = s1;
      esum[kChunk + t] = s2;
    }
  }

  // ---------------- phase 2: W, G, P on the lower token tiles ----------------
  constexpr int kMyTiles = (10 + NW - 1) / NW;   // share of the 10 lower tiles per wave
  floatx4 tW1[kMyTiles], tW2[kMyTiles], tW3[kMyTiles], tW4[kMyTiles], tW5[kMyTiles];
  floatx4 tG[kMyTiles], tP[kMyTiles];
  // Lower tiles (token block rows tt >= st). With eight waves, waves 0 and 1
  // take two tiles each: those four are strictly below the diagonal (no
  // masks, the cheaper decay step), the four diagonal tiles go to waves 2-5,
  // and each wave's tiles differ in both row and column block (every per-wave
  // sum entry is written once).  Other wave counts: row by row.
  auto tile_of = [](int idx, int& tt, int& st) {
    if constexpr (NW == 8) {   // (tt, st) of idx 0..9, two bits each
      constexpr int kT = 0xfee49, kS = 0x91e40;
      tt = (kT >> (2 * idx)) & 3;
      st = (kS >> (2 * idx)) & 3;
    } else {
      tt = idx >= 6 ? 3 : idx >= 3 ? 2 : idx >= 1 ? 1 : 0;
      st = idx - (tt * (tt + 1)) / 2;
    }
  };
#pragma unroll
  for (int x = 0; x < kMyTiles; ++x) {
    asm volatile("" ::: "memory");
    const int idx = w + NW * x;
    tW1[x] = zero4(); tW2[x] = zero4(); tW3[x] = zero4(); tW4[x] = zero4(); tW5[x] = zero4();
    tG[x] = zero4(); tP[x] = zero4();
    if (idx < 10) {
      int tt, st;
      tile_of(idx, tt, st);
#pragma unroll
      for (int ks = 0; ks < KSV; ++ks) {
        const int k0 = ks * M::kStep;
        const Frag fo = TV::template frag<M>(tokblk(bDO), 16 * tt, k0);
        const Frag fx = TV::template frag<M>(tokblk(bDX), 16 * tt, k0);
        const Frag fu = TV::template frag<M>(tokblk(bU), 16 * st, k0);
        const Frag fur = TV::template frag<M>(tokblk(bUR), 16 * st, k0);
        tW1[x] = M::mma(fo, fu, tW1[x]);
        tW2[x] = M::mma(fo, fur, tW2[x]);
        tW3[x] = M::mma(fx, fu, tW3[x]);
        if constexpr (RDN) {
          tW4[x] = M::mma(TV::template frag<M>(tokblk(bDY), 16 * tt, k0), fu, tW4[x]);
          tW5[x] = M::mma(TV::template frag<M>(tokblk(bDYR), 16 * tt, k0), fur, tW5[x]);
        }
      }
#pragma unroll
      for (int ks = 0; ks < KSK; ++ks) {
        const int k0 = ks * M::kStep;
        const Frag fk = TK::template frag<M>(Kl, 16 * st, k0);
        tG[x] = M::mma(TK::template frag<M>(Kl, 16 * tt, k0), fk, tG[x]);
        tP[x] = M::mma(TK::template frag<M>(Ql, 16 * tt, k0), fk, tP[x]);
      }
    }
  }
  // ---- dP, dG (into registers) and the sums over the decay-matrix products ----
  float edp[kMyTiles][4], edg[kMyTiles][4];
#pragma unroll
  for (int x = 0; x < kMyTiles; ++x) {
    const int idx = w + NW * x;
    if (idx < 10) {
      int tt, st;
      tile_of(idx, tt, st);
      float zs[4], zp[4], zr[4], zb[4], zg[4];
      // SL: a tile strictly below the diagonal (s < t everywhere: no masks,
      // and every exponent is already <= 0)
      auto decay_step = [&](auto strict) {
      constexpr bool SL = decltype(strict)::value;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = 16 * tt + acc_row(r), s = 16 * st + acc_col();
        const bool lower = SL || s < t, diag = SL || s <= t;
        const float es = __expf(SL ? gsv[t] - gsv[s] : fminf(gsv[t] - gsv[s], 0.f));
        const float ep = __expf(SL ? gspv[t] - gsv[s] : fminf(gspv[t] - gsv[s], 0.f));
        const float er = __expf(SL ? grv[t] - grv[s] : fminf(grv[t] - grv[s], 0.f));
        const float W1 = tW1[x][r], W2 = tW2[x][r], W3 = tW3[x][r];
        const float G = tG[x][r], P = tP[x][r];
        const float dAs = RDN ? -tW4[x][r] : 0.f, dAr = RDN ? -tW5[x][r] : 0.f;
        // decays of the base read-out (W1) and residual (W3) terms: e^{g_t - g_s}
        // or e^{g_{t-1} - g_s}, by variant; their gate terms follow them to
        // the g_t (zs) or the g_{t-1} (zp) sums
        const float ew1 = ung ? ep : es, ew3 = dec ? es : ep;
        const float gw2 = (ung ? 1.f : ggm[t]) * W2;
        const float dp = (lower ? ew1 * W1 : 0.f) + (diag ? er * gw2 : 0.f);
        const float dg = lower ? (-ew3 * W3 + gbt[t] * es * dAs + ggm[t] * er * dAr) : 0.f;
        const float t1 = lower ? ew1 * P * W1 : 0.f, t3 = lower ? -ew3 * G * W3 : 0.f;
        zs[r] = (lower ? es * gbt[t] * G * dAs : 0.f) + (ung ? 0.f : t1) + (dec ? t3 : 0.f);
        zp[r] = (ung ? t1 : 0.f) + (dec ? 0.f : t3);
        zr[r] = (diag ? er * P * gw2 : 0.f) + (lower ? ggm[t] * er * G * dAr : 0.f);
        zb[r] = lower ? dAs * es * G : 0.f;
        zg[r] = (lower ? dAr * er * G : 0.f) + ((diag && !ung) ? er * P * W2 : 0.f);
        edp[x][r] = dp;
        edg[x][r] = dg;
      }
      };
      if (tt > st) decay_step(std::true_type{});
      else decay_step(std::false_type{});
      put_rows(sum_row(sZRS), 16 * tt, zs);
      put_rows(sum_row(sZRP), 16 * tt, zp);
      put_rows(sum_row(sZRR), 16 * tt, zr);
      put_rows(sum_row(sZB), 16 * tt, zb);
      put_rows(sum_row(sZGM), 16 * tt, zg);
      put_cols(sum_row(sZCS), 16 * st, zs);
      put_cols(sum_row(sZCP), 16 * st, zp);
      put_cols(sum_row(sZCR), 16 * st, zr);
    }
  }
  // ---------------- phase 1: contractions over the value dimension ----------------
  floatx4 dQ[kIT][4], dK[kIT][4];
#pragma unroll
  for (int m = 0; m < kIT; ++m)
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) { dQ[m][tt] = zero4(); dK[m][tt] = zero4(); }
  float gsC = 0.f, grC = 0.f;

  // sum over this lane's elements of a (.) b (fp16 pairs by v_dot2_f32_f16:
  // fp16 products are exact in fp32, accumulated in fp32)
  auto frag_dot = [&](const StateRows& a, const StateRows& b) {
    float s = 0.f;
#pragma unroll
    for (int ks = 0; ks < KSV; ++ks) {
      if constexpr (BF) {
        typedef _Float16 h2 __attribute__((ext_vector_type(2)));
#pragma unroll
        for (int e = 0; e < 8; e += 2)
          s = __builtin_amdgcn_fdot2(h2{a.fr[ks][e], a.fr[ks][e + 1]}, h2{b.fr[ks][e], b.fr[ks][e + 1]}, s, false);
      } else {
        s += a.fr[ks] * b.fr[ks];
      }
    }
    return s * (a.sc * b.sc);
  };
  // [16 tokens x 16 state rows] tile: token block rows 16 tt times the state
  // rows, contracted over the value dimension; each k-step's scale is applied
  // by rescaling the accumulator (powers of two: exact)
  auto contract = [&](int b, int tt, const StateRows& x) {
    floatx4 acc = zero4();
#pragma unroll
    for (int ks = 0; ks < KSV; ++ks) {
      acc = M::mma(TV::template frag<M>(tokblk(b), 16 * tt, ks * M::kStep), x.fr[ks], acc);
    }
    return BF ? acc * x.sc : acc;
  };

  // per d_k tile: S0 with dS1, then R0 with dR1; the next pair's rows are
  // loaded while the current pair's products run
#pragma unroll
  for (int m = 0; m < kIT; ++m) {
    // the token-block fragments are reloaded per d_k tile: keeping them
    // across tiles would need ~400 registers
    asm volatile("" ::: "memory");
    const int i0 = 16 * (w + NW * m);
    const int icol = i0 + (lane & 15);   // this lane's output column
    // K, Q at this lane's output positions of token tile tt
    auto kq_of = [&](int tt, float (&kq)[4], float (&qq)[4]) {
      if constexpr (BF) {   // one transpose read each
        // (whole-vector casts: a bit cast of one vector element miscompiles)
        const f16x4 k4 = __builtin_bit_cast(f16x4, acc_tile_tr<TK>(Kl, 16 * tt, i0));
        const f16x4 q4 = __builtin_bit_cast(f16x4, acc_tile_tr<TK>(Ql, 16 * tt, i0));
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          kq[r] = (float)k4[r];
          qq[r] = (float)q4[r];
        }
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          kq[r] = to_f<XT>(TK::at(Kl, 16 * tt + acc_row(r), icol));
          qq[r] = to_f<XT>(TK::at(Ql, 16 * tt + acc_row(r), icol));
        }
      }
    };
    // ---- S0 (rowA) and dS1 (rowB) ----
    {
      const StateRows s0 = rowA, d1 = rowB;
      gsC += edge[0] * frag_dot(s0, d1);   // e^{g_C} <S0, dS1>
      load_rows(rowA, 1, i0);
      load_rows(rowB, 3, i0);
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        asm volatile("" ::: "memory");   // bounds how far fragment loads are hoisted
        // F1 = dO S0^T, FK1 = dX S0^T, FK2 = dY S0^T, FK4 = U dS1^T
        const floatx4 F1 = contract(bDO, tt, s0);
        const floatx4 FK1 = contract(bDX, tt, s0);
        floatx4 FK2 = zero4();
        if constexpr (RDN) FK2 = contract(bDY, tt, s0);
        const floatx4 FK4 = contract(bU, tt, d1);
        float kq[4], qq[4], ags[4], agsp[4], ab[4];
        kq_of(tt, kq, qq);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = 16 * tt + acc_row(r);
          const float c1 = eqb[t] * F1[r], c2 = -ekp[t] * FK1[r], c6 = dls[t] * FK4[r];
          dQ[m][tt][r] += c1;
          dK[m][tt][r] += c2 + c6;
          // c1 is a g_t term (g_{t-1} when ungated), c2 a g_{t-1} term (g_t when decayed)
          ags[r] = (ung ? 0.f : qq[r] * c1) + (dec ? kq[r] * c2 : 0.f) - kq[r] * c6;
          agsp[r] = (ung ? qq[r] * c1 : 0.f) + (dec ? 0.f : kq[r] * c2);
          gsC += kq[r] * c6;
          ab[r] = 0.f;
          if constexpr (RDN) {
            const float e2 = -egs[t] * FK2[r];
            dK[m][tt][r] += gbt[t] * e2;
            ags[r] += kq[r] * gbt[t] * e2;
            ab[r] = kq[r] * e2;
          }
        }
        put_rows(sum_row(sGS), 16 * tt, ags);
        put_rows(sum_row(sGSP), 16 * tt, agsp);
        if constexpr (RDN) put_rows(sum_row(sB), 16 * tt, ab);
      }
    }
    // ---- R0 (rowA) and dR1 (rowB) ----
    {
      const StateRows r0 = rowA, e1 = rowB;
      grC += edge[1] * frag_dot(r0, e1);   // e^{h_C} <R0, dR1>
      if (m + 1 < kIT) {
        load_rows(rowA, 0, i0 + 16 * NW);
        load_rows(rowB, 2, i0 + 16 * NW);
      }
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        asm volatile("" ::: "memory");
        // F2 = dO R0^T, FK3 = dYR R0^T, FK5 = UR dR1^T
        const floatx4 F2 = contract(bDO, tt, r0);
        floatx4 FK3 = zero4();
        if constexpr (RDN) FK3 = contract(bDYR, tt, r0);
        const floatx4 FK5 = contract(bUR, tt, e1);
        float kq[4], qq[4], agr[4], agm[4];
        kq_of(tt, kq, qq);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = 16 * tt + acc_row(r);
          const float e4 = egr[t] * F2[r], c4 = (ung ? 1.f : ggm[t]) * e4, c7 = dlr[t] * FK5[r];
          dQ[m][tt][r] += c4;
          dK[m][tt][r] += c7;
          agr[r] = qq[r] * c4 - kq[r] * c7;
          agm[r] = ung ? 0.f : qq[r] * e4;   // gamma's output term
          grC += kq[r] * c7;
          if constexpr (RDN) {
            const float e5 = -egr[t] * FK3[r], c5 = ggm[t] * e5;
            dK[m][tt][r] += c5;
            agr[r] += kq[r] * c5;
            agm[r] += kq[r] * e5;
          }
        }
        put_rows(sum_row(sGR), 16 * tt, agr);
        put_rows(sum_row(sGM), 16 * tt, agm);
      }
    }
  }
  {
    const float a = wave_sum(gsC), b = wave_sum(grC);
    if (lane == 0) { red[w] = a; red[NW + w] = b; }
  }

  barrier_lds();   // token blocks dead: their region becomes dP, dP^T, dG + dG^T, K^T, Q^T

  // ---- dP, dP^T and dG + dG^T (kept in registers since the decay step) ----
  constexpr int ldp = L::kLdP;
#pragma unroll
  for (int x = 0; x < kMyTiles; ++x) {
    const int idx = w + NW * x;
    if (idx < 10) {
      int tt, st;
      tile_of(idx, tt, st);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = 16 * tt + acc_row(r), s = 16 * st + acc_col();
        dPm[t * ldp + s] = from_f<XT>(edp[x][r]);
        if constexpr (!BF) dPTm[s * ldp + t] = from_f<XT>(edp[x][r]);
        if (s < t) {   // dG + dG^T: the two halves have disjoint supports
          dGm[t * ldp + s] = from_f<XT>(edg[x][r]);
          dGm[s * ldp + t] = from_f<XT>(edg[x][r]);
        } else if (s == t) {
          dGm[t * ldp + t] = from_f<XT>(0.f);
        }
      }
    }
  }
  // dP above the diagonal and dP^T below it are zero: the 6 upper tiles
  for (int x = w; x < 6; x += NW) {
    const int tt = x < 3 ? 0 : x < 5 ? 1 : 2;
    const int st = tt + 1 + x - (tt == 0 ? 0 : tt == 1 ? 3 : 5);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = 16 * tt + acc_row(r), s = 16 * st + acc_col();
      dPm[t * ldp + s] = from_f<XT>(0.f);
      if constexpr (!BF) dPTm[s * ldp + t] = from_f<XT>(0.f);
    }
  }
  // the per-token sums over the waves, shared out over all threads (in the
  // order of the waves, so every total is rounded alike)
  {
    float* tot = reinterpret_cast<float*>(smem + L::kTot);
    for (int e = tid; e < kNumSums * kChunk; e += NT) {
      float x = 0.f;
#pragma unroll
      for (int v = 0; v < NW; ++v) x += sums[v * kNumSums * kChunk + e];
      tot[e] = x;
    }
  }
  // K^T, Q^T for the final products (fp32; 16-bit operands read K, Q and
  // dP transposed with transpose reads)
  if constexpr (!BF)
  for (int e = tid; e < kChunk * DK / kE; e += NT) {
    const int s = e / (DK / kE), i = (e % (DK / kE)) * kE;
    const uint4 kv = *reinterpret_cast<const uint4*>(Kl + TK::off(s, i));
    const uint4 qv = *reinterpret_cast<const uint4*>(Ql + TK::off(s, i));
    const XT* a = reinterpret_cast<const XT*>(&kv);
    const XT* b = reinterpret_cast<const XT*>(&qv);
#pragma unroll
    for (int k = 0; k < kE; ++k) {
      KTm[(i + k) * ldp + s] = a[k];
      QTm[(i + k) * ldp + s] = b[k];
    }
  }
  barrier_lds();

  // ---------------- phase 3: gate gradients; dQ += dP K, dK += dP^T Q + (dG + dG^T) K ----------------
  if (tid < kChunk) {
    const float* tot = reinterpret_cast<const float*>(smem + L::kTot);
    auto tot_at = [&](int q, int t) { return tot[q * kChunk + t]; };
    const int t = tid;
    float gsC_all = 0.f, grC_all = 0.f;
#pragma unroll
    for (int v = 0; v < NW; ++v) { gsC_all += red[v]; grC_all += red[NW + v]; }
    const float dgs = tot_at(sGS, t) + tot_at(sZRS, t) - tot_at(sZCS, t) - tot_at(sZCP, t) +
                      (t + 1 < kChunk ? tot_at(sGSP, t + 1) + tot_at(sZRP, t + 1) : 0.f) +
                      (t == kChunk - 1 ? gsC_all : 0.f);
    const float dgr = tot_at(sGR, t) + tot_at(sZRR, t) - tot_at(sZCR, t) +
                      (t == kChunk - 1 ? grC_all : 0.f);
    // suffix sums over the chunk: d log a_j = sum_{t >= j} d g_t
    float ss = dgs, sr = dgr;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float a = __shfl_down(ss, off, 64), b = __shfl_down(sr, off, 64);
      if (t + off < 64) { ss += a; sr += b; }
    }
    ss *= isig;   // out of the upstream-gradient scale
    sr *= isig;
    // ss, sr: gradients of log aS_t, log aR_t
    float pa = 0.f, pb = 0.f;   // this token's share of d/da_h, d/db_h (pre-activations)
    if (t < len) {
      const int64_t gi = tok * H + h + (uint32_t)(t * H);
      const float db = (esum[t] + tot_at(sB, t) + tot_at(sZB, t)) * isig;
      const float dgm = (esum[kChunk + t] + tot_at(sGM, t) + tot_at(sZGM, t)) * isig;
      if (vf & kVarGatePreact) {
        // log a = -A softplus(z + Bb): d/dz = -A sigmoid(z + Bb), d/dA = -softplus(z + Bb);
        // beta = sigmoid(z): d/dz = beta (1 - beta), likewise gamma
        const float A = p.decay_param[h], Bb = p.decay_param[H + h];
        const float zs = a_s + Bb, zr = a_r + Bb;
        const float dzs = ss * (-A * sigmoid_f(zs)), dzr = sr * (-A * sigmoid_f(zr));
        p.dalpha_s[gi] = dzs;
        p.dalpha_r[gi] = dzr;
        pa = -(ss * softplus_f(zs) + sr * softplus_f(zr));
        pb = dzs + dzr;
        p.dbeta[gi] = db * gbt[t] * (1.f - gbt[t]);
        p.dgamma[gi] = dgm * ggm[t] * (1.f - ggm[t]);
      } else {
        p.dalpha_s[gi] = a_s >= 1.17549435e-38f ? ss / a_s : 0.f;
        p.dalpha_r[gi] = a_r >= 1.17549435e-38f ? sr / a_r : 0.f;
        p.dbeta[gi] = db;
        p.dgamma[gi] = dgm;
      }
    }
    if (vf & kVarGatePreact) {   // the chunk's (a, b) partials, summed over its tokens
      pa = wave_sum(pa);
      pb = wave_sum(pb);
      if (t == 0) {
        p.decay_partials[((int64_t)c * H + h) * 2 + 0] = pa;
        p.decay_partials[((int64_t)c * H + h) * 2 + 1] = pb;
      }
    }
  }
#pragma unroll
  for (int m = 0; m < kIT; ++m) {
    const int i0 = 16 * (w + NW * m);
#pragma unroll
    for (int ks = 0; ks < KSC; ++ks) {
      const int k0 = ks * M::kStep;
      Frag fk, fq;
      if constexpr (BF) {
        fk = frag_tr<TK, M>(Kl, i0, k0);
        fq = frag_tr<TK, M>(Ql, i0, k0);
      } else {
        fk = M::template load<true>(KTm + i0 * ldp, ldp, k0);
        fq = M::template load<true>(QTm + i0 * ldp, ldp, k0);
      }
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        Frag fpt;
        if constexpr (BF) fpt = frag_tr<TDP, M>(dPm, 16 * tt, k0);   // dP^T rows from dP
        else fpt = M::template load<true>(dPTm + 16 * tt * ldp, ldp, k0);
        dQ[m][tt] = M::mma(M::template load<true>(dPm + 16 * tt * ldp, ldp, k0), fk, dQ[m][tt]);
        dK[m][tt] = M::mma(fpt, fq, dK[m][tt]);
        dK[m][tt] = M::mma(M::template load<true>(dGm + 16 * tt * ldp, ldp, k0), fk, dK[m][tt]);
      }
    }
  }
  OT* dqg = reinterpret_cast<OT*>(p.dq);
  OT* dkg = reinterpret_cast<OT*>(p.dk);
#pragma unroll
  for (int m = 0; m < kIT; ++m)
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = 16 * tt + acc_row(r);
        if (t < len) {
          const int64_t gi = (tok * H + h) * (int64_t)DK + 16 * (w + NW * m) + (uint32_t)(t * H * DK + acc_col());
          dqg[gi] = from_f<OT>(dQ[m][tt][r] * isig);
          dkg[gi] = from_f<OT>(dK[m][tt][r] * isig);
        }
      }
}

template <typename IN, int DK, int DV, bool RDN, typename OT>
hipError_t launch_grad_t(const OpParams& p, hipStream_t stream) {
  typedef GradLayout<IN, DK, DV> L;
  auto kern = ((p.vflags & (kVarOperator | kVarGatePreact)) || p.qk_f16)
                  ? bwd_grad_kernel<IN, DK, DV, RDN, OT, true>
                  : bwd_grad_kernel<IN, DK, DV, RDN, OT, false>;
  hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, L::kBytes);
  if (err != hipSuccess) return err;
  if (p.max_chunks == 0) return hipSuccess;
  hipLaunchKernelGGL(kern, dim3(p.H, p.max_chunks), dim3(L::kNT), L::kBytes, stream, p);
  return hipGetLastError();
}

template <typename IN, int DK, typename OT>
hipError_t launch_grad_dk(const OpParams& p, hipStream_t s) {
  if (p.DV == 128)
    return p.rdn ? launch_grad_t<IN, DK, 128, true, OT>(p, s) : launch_grad_t<IN, DK, 128, false, OT>(p, s);
  return p.rdn ? launch_grad_t<IN, DK, 64, true, OT>(p, s) : launch_grad_t<IN, DK, 64, false, OT>(p, s);
}

}  // namespace

hipError_t launch_bwd_grad(const OpParams& p, bool bf16, hipStream_t stream) {
  if (bf16) {
    if (p.out_bf16)
      return p.DK == 128 ? launch_grad_dk<u16, 128, u16>(p, stream) : launch_grad_dk<u16, 64, u16>(p, stream);
    return p.DK == 128 ? launch_grad_dk<u16, 128, float>(p, stream) : launch_grad_dk<u16, 64, float>(p, stream);
  }
  // fp32: d_k = d_v = 64 (checked by the host API)
  return p.rdn ? launch_grad_t<float, 64, 64, true, float>(p, stream)
               : launch_grad_t<float, 64, 64, false, float>(p, stream);
}

}  // namespace rla
