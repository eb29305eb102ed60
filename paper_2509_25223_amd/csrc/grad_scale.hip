// Largest magnitude of the backward's upstream gradients, per (chunk, head):
// over the chunk's rows of dO and, for the first chunk of a sequence, over
// that (sequence, head)'s final-state gradients dS_T and dR_T.
//
// The backward is linear in (dO, dS_T, dR_T) jointly, and its fp16 operands
// (dO itself, the gate-weighted copies of it, the blocks dX, dY, dYR) inherit
// the magnitude of the loss gradient, which in bf16 training without loss
// scaling is often far below fp16's normal range.  The reverse scan therefore
// reduces these maxima over each (sequence, head) and multiplies dO, dS_T and
// dR_T by one power of two 2^e that brings their largest magnitude into
// [4, 8) (the range of N(0, 1) data); every output of the backward is
// multiplied by 2^-e when written.  Powers of two are exact, so the result is
// the unscaled computation wherever no fp16 value underflows or overflows.
#include "kernels.hpp"

namespace rla {

namespace {

__device__ __forceinline__ uint32_t bf16_mag_bits(uint32_t two) {
  // the two bf16 values of a 32-bit word as fp32 magnitude bit patterns
  return max((two & 0x7FFFu) << 16, two & 0x7FFF0000u);
}

// One wave per (chunk, head), eight chunks of one head per workgroup (half
// the workgroups of four-wave groups, ~4% faster); heads vary fastest over
// consecutive workgroups, which then read contiguous stretches of dO.  Every
// load of a wave is issued before any is used.  The loads are ordinary
// (cached): the reverse scan reads dO next, and non-temporal loads, though
// they speed this pass up by a third, cost the reverse scan more.
constexpr int kAbsWaves = 8;

template <int DV>
__global__ __launch_bounds__(64 * kAbsWaves) void grad_absmax_kernel(OpParams p, uint32_t* out) {
  const int h = blockIdx.x, w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c = blockIdx.y * kAbsWaves + w;
  ChunkInfo ci;
  if (c >= p.max_chunks || !chunk_info(p.st, c, ci)) return;
  const int H = p.H, DK = p.DK;
  uint32_t m = 0;
  {   // the chunk's dO rows, 16 bytes (8 bf16) per load; rows past the
      // chunk's end re-read its last row (no effect on a maximum)
    constexpr int kPerRow = DV / 8;
    constexpr int kIter = kChunk * kPerRow / 64;
    const uint4* src = reinterpret_cast<const uint4*>(p.dO);
    uint4 x[kIter];
#pragma unroll
    for (int u = 0; u < kIter; ++u) {
      const int e = lane + u * 64, t = min(e / kPerRow, ci.len - 1), j = e % kPerRow;
      x[u] = src[((ci.tok + t) * H + h) * (int64_t)kPerRow + j];
    }
#pragma unroll
    for (int u = 0; u < kIter; ++u)
      m = max(m, max(max(bf16_mag_bits(x[u].x), bf16_mag_bits(x[u].y)),
                     max(bf16_mag_bits(x[u].z), bf16_mag_bits(x[u].w))));
  }
  const SeqInfo si = seq_info(p.st, ci.seq);
  if (ci.tok == si.start) {   // first chunk: the final-state gradients of (sequence, head)
    const int64_t off = ((int64_t)ci.seq * H + h) * DK * DV;
    const float* st[2] = {p.dS_fin, p.dR_fin};
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      if (!st[s]) continue;
      const float4* src = reinterpret_cast<const float4*>(st[s] + off);
      for (int e = lane; e < DK * (DV / 4); e += 64) {
        const float4 x = src[e];
        m = max(m, max(max(__float_as_uint(x.x) & 0x7FFFFFFFu, __float_as_uint(x.y) & 0x7FFFFFFFu),
                       max(__float_as_uint(x.z) & 0x7FFFFFFFu, __float_as_uint(x.w) & 0x7FFFFFFFu)));
      }
    }
  }
  m = wave_absmax_bits(m);
  if (lane == 0) out[(int64_t)c * H + h] = m;
}

}  // namespace

hipError_t launch_grad_absmax(const OpParams& p, uint32_t* out, hipStream_t stream) {
  if (p.max_chunks == 0) return hipSuccess;
  auto kern = p.DV == 128 ? grad_absmax_kernel<128> : grad_absmax_kernel<64>;
  hipLaunchKernelGGL(kern, dim3(p.H, (p.max_chunks + kAbsWaves - 1) / kAbsWaves), dim3(64 * kAbsWaves), 0,
                     stream, p, out);
  return hipGetLastError();
}

}  // namespace rla
