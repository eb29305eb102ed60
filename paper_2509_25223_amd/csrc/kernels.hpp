// Internal interface between the host API (api.cpp) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

namespace rla {

constexpr int kNumBlk = 3;   // per-token blocks per (chunk, head) in fwd_blk / bwd_blk

// Element offset of block b of (global chunk gc, head h) in fwd_blk / bwd_blk.
__host__ __device__ inline int64_t blk_off(int64_t gc, int h, int H, int b, int DV) {
  return ((gc * H + h) * kNumBlk + b) * (int64_t)kChunk * DV;
}

// Variants of the residual and of the output (bits of OpParams::vflags):
//   kVarTanh     r = c tanh(x / c) instead of the clip (c < 0: r = x; c = 0: r = 0)
//   kVarUngated  o = S_{t-1} q + R_t q
//   kVarDecayed  x = v - aS S_{t-1} k
//   kVarGatePreact gates given as pre-activations (prep, gradient kernel, decoding)
//   kVarQkNorm     q, k given raw: SiLU + L2 normalisation (decoding; the host
//                  runs the pre-processing kernels for the chunked path)
constexpr int kVarTanh = 1, kVarUngated = 2, kVarDecayed = 4;
constexpr int kVarOperator = kVarTanh | kVarUngated | kVarDecayed;   // bits the scans read
constexpr int kVarGatePreact = 8, kVarQkNorm = 16;

// Everything a launch needs; passed by value to the kernels.
struct OpParams {
  int32_t H = 0, DK = 0, DV = 0;
  int64_t ntok = 0;
  float clip = -1.f;            // < 0: no clipping
  int32_t rdn = 1;              // 1: RDN, 0: RLA
  int32_t vflags = 0;           // kVar* bits
  int32_t out_bf16 = 0;         // o, dq, dk, dv in bf16 (else fp32)
  int32_t max_chunks = 0;       // upper bound on chunks (grid size of chunk-parallel kernels)
  int32_t qk_f16 = 0;           // bf16 inputs: q, k are fp16 rows (the pre-processing's output)
  SeqTable st{};

  const void* q = nullptr;
  const void* k = nullptr;
  const void* v = nullptr;
  const float* alpha_s = nullptr;
  const float* beta = nullptr;
  const float* alpha_r = nullptr;
  const float* gamma = nullptr;
  const float* S0 = nullptr;
  const float* R0 = nullptr;
  const float* decay_param = nullptr;   // [2][H] a, b (kVarGatePreact)
  float* decay_partials = nullptr;      // [max_chunks][H][2] per-chunk d/da, d/db (backward)

  void* o = nullptr;
  float* S_fin = nullptr;
  float* R_fin = nullptr;

  // workspace regions
  float* gate_ws = nullptr;     // [max_chunks][H][kGateBlock]
  void* mat_ws = nullptr;       // [max_chunks][H][kNumMats][kMatElems]: packed lower blocks (mm type)
  // chunk states saved for the gradient kernel, [max_chunks][H][DK][DV]: fp32
  // for fp32 inputs; fp16 for bf16 inputs, each (row, 32 columns) scaled by a
  // power of two held in the matching *_sc array [max_chunks][H][DK][DV / 32]
  void* ck_S = nullptr;         // chunk-start S
  void* ck_R = nullptr;         // chunk-start R
  void* dS_ws = nullptr;        // grad of chunk-end S
  void* dR_ws = nullptr;        // grad of chunk-end R
  float* ck_S_sc = nullptr;
  float* ck_R_sc = nullptr;
  float* dS_sc = nullptr;
  float* dR_sc = nullptr;
  uint8_t* ck_mask = nullptr;   // [ntok][H][DV] 1 where |x| <= clip
  // per-token blocks saved for the gradient kernel, [max_chunks][H][3][64][DV]
  // (mm type, token-major, rows past the end of a sequence are zero):
  void* fwd_blk = nullptr;      // U, UR, r (clipped residual) from the forward scan
  void* bwd_blk = nullptr;      // dX, dY (RLA: dU), dYR (RLA: dUR) from the reverse scan

  // backward
  const void* dO = nullptr;
  const float* dS_fin = nullptr;
  const float* dR_fin = nullptr;
  void* dq = nullptr;
  void* dk = nullptr;
  void* dv = nullptr;
  float* dalpha_s = nullptr;
  float* dbeta = nullptr;
  float* dalpha_r = nullptr;
  float* dgamma = nullptr;
  float* dS0 = nullptr;
  float* dR0 = nullptr;
  // bf16 inputs: per (chunk, head) largest magnitude of dO (and, for a
  // sequence's first chunk, of dS_T and dR_T) as fp32 bits, [max_chunks][H];
  // and the power-of-two scale of the upstream gradients of each (sequence,
  // head), [nseq][H], written by the reverse scan, read by the gradient kernel
  // (NULL: scale 1)
  const uint32_t* grad_absmax = nullptr;
  float* grad_scale = nullptr;
};

// Zeroes `bytes` (a multiple of 4) at dst with a kernel rather than a memset
// node, so that a caller may capture the call in a HIP graph.
hipError_t launch_zero_fill(void* dst, size_t bytes, hipStream_t stream);

// Builds SeqInfo / ChunkInfo / order tables from device cu_seqlens.
hipError_t launch_seq_table(const int32_t* cu, int32_t nseq, int64_t ntok, int32_t max_chunks,
                            SeqInfo* seqs, ChunkInfo* chunks, int32_t* nchunks, int32_t* order,
                            hipStream_t stream);

// Chunk-parallel preparation: gate cumsums, masked decayed Gram/score
// matrices and (RDN) the two triangular inverses.
hipError_t launch_prep(const OpParams& p, bool bf16, hipStream_t stream);

// Forward state-passing scan.  write_o: produce o; ckpt: store chunk-start
// states, clip masks and the U, UR, r blocks for the backward.
hipError_t launch_fwd_scan(const OpParams& p, bool bf16, bool write_o, bool ckpt,
                           hipStream_t stream);

// Per (chunk, head) largest magnitude of the upstream gradients (dO; dS_T and
// dR_T folded into a sequence's first chunk) into out[max_chunks][H].
hipError_t launch_grad_absmax(const OpParams& p, uint32_t* out, hipStream_t stream);

// Reverse state-gradient scan (RDN / RLA); also writes dv and the dX, dY,
// dYR blocks.
hipError_t launch_bwd_scan(const OpParams& p, bool bf16, hipStream_t stream);

// Chunk-parallel gradient contractions.
hipError_t launch_bwd_grad(const OpParams& p, bool bf16, hipStream_t stream);

// SiLU + L2 normalisation of the q and k rows ([rows][DK] each) into qh, kh.
hipError_t launch_qk_norm_fwd(const void* q, const void* k, void* qh, void* kh, int64_t rows,
                              int DK, bool bf16, hipStream_t stream);

// Gradient through the SiLU + L2 normalisation: dq = J^T dqh (raw q, fp32
// dqh), likewise k; dq, dk in the output type.
hipError_t launch_qk_norm_bwd(const void* q, const void* k, const float* dqh, const float* dkh,
                              void* dq, void* dk, int64_t rows, int DK, bool bf16, bool out_bf16,
                              hipStream_t stream);

// Sums the gradient kernel's per-chunk (a, b) partials over chunks per head:
// out[h] = sum_c partials[c][h][0], out[H + h] = sum_c partials[c][h][1].
hipError_t launch_decay_grad_reduce(const float* partials, int nch, int H, float* out,
                                    hipStream_t stream);

// Recurrent step over T tokens per sequence (dense layout, st.dense_T = T,
// st.nseq = B) with S0/R0 in (NULL = zeros) and S_fin/R_fin out.
hipError_t launch_decode(const OpParams& p, bool bf16, hipStream_t stream);

}  // namespace rla
