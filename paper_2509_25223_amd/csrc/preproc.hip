// Input pre-processing of the operator (the closing paragraph of Sec. 3.4:
// SiLU and L2 normalisation of queries and keys) and the reduction of the
// decay re-parameterisation's per-head gradients.
//
// qk_norm_fwd: one wave per token-head row, y = SiLU(x) = x sigmoid(x),
//   x_hat = y / max(||y||, 1e-12), stored as fp32 for fp32 inputs and as fp16
//   for bf16 inputs (|x_hat| <= 1, so fp16's 11 significant bits lose
//   nothing to range; bf16's 8 would cost about 2e-2 of max|error|/RMS on o
//   by themselves); the chunked kernels read these rows in place of q, k.
// qk_norm_bwd: dx = SiLU'(x) (dx_hat - x_hat (x_hat . dx_hat)) / ||y||, with
//   SiLU'(x) = s (1 + x (1 - s)), s = sigmoid(x); below the 1e-12 floor the
//   normalisation is the fixed scale 1e12 and dy = dx_hat 1e12.  x_hat is
//   recomputed in fp32 from the raw row.
// decay_grad_reduce: one workgroup per head sums the per-chunk partials in a
//   fixed order (deterministic).
#include <type_traits>

#include "kernels.hpp"

namespace rla {

namespace {

constexpr float kNormEps = 1e-12f;

__device__ __forceinline__ float silu_sig(float x, float& s) {
  s = 1.f / (1.f + __expf(-x));
  return x * s;
}

__device__ __forceinline__ float wave_allsum(float v) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) v += __shfl_xor(v, m);
  return v;
}

template <typename IN, typename NT, int DK>
__global__ __launch_bounds__(kThreads) void qk_norm_fwd_kernel(const IN* __restrict__ q,
                                                               const IN* __restrict__ k,
                                                               NT* __restrict__ qh, NT* __restrict__ kh,
                                                               int64_t rows) {
  constexpr int PL = DK / 64;   // values per lane
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kWaves + w;
  if (row >= rows) return;
  const IN* src = (blockIdx.y == 0 ? q : k) + row * DK + lane * PL;
  NT* dst = (blockIdx.y == 0 ? qh : kh) + row * DK + lane * PL;
  float y[PL], ss = 0.f;
#pragma unroll
  for (int e = 0; e < PL; ++e) {
    float s;
    y[e] = silu_sig(to_f<IN>(src[e]), s);
    ss = __builtin_fmaf(y[e], y[e], ss);
  }
  const float inv = 1.f / fmaxf(sqrtf(wave_allsum(ss)), kNormEps);
#pragma unroll
  for (int e = 0; e < PL; ++e) dst[e] = from_f<NT>(y[e] * inv);
}

template <typename IN, typename OT, int DK>
__global__ __launch_bounds__(kThreads) void qk_norm_bwd_kernel(const IN* __restrict__ q,
                                                               const IN* __restrict__ k,
                                                               const float* __restrict__ dqh,
                                                               const float* __restrict__ dkh,
                                                               OT* __restrict__ dq, OT* __restrict__ dk,
                                                               int64_t rows) {
  constexpr int PL = DK / 64;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kWaves + w;
  if (row >= rows) return;
  const int64_t off = row * DK + lane * PL;
  const IN* src = (blockIdx.y == 0 ? q : k) + off;
  const float* g = (blockIdx.y == 0 ? dqh : dkh) + off;
  OT* dst = (blockIdx.y == 0 ? dq : dk) + off;
  float x[PL], s[PL], y[PL], gh[PL], ss = 0.f;
#pragma unroll
  for (int e = 0; e < PL; ++e) {
    x[e] = to_f<IN>(src[e]);
    y[e] = silu_sig(x[e], s[e]);
    gh[e] = g[e];
    ss = __builtin_fmaf(y[e], y[e], ss);
  }
  const float nrm = sqrtf(wave_allsum(ss));
  const bool floor = nrm < kNormEps;
  const float inv = 1.f / fmaxf(nrm, kNormEps);
  float dot = 0.f;
#pragma unroll
  for (int e = 0; e < PL; ++e) dot = __builtin_fmaf(y[e] * inv, gh[e], dot);
  dot = wave_allsum(dot);
#pragma unroll
  for (int e = 0; e < PL; ++e) {
    const float dy = floor ? gh[e] * inv : (gh[e] - y[e] * inv * dot) * inv;
    dst[e] = from_f<OT>(dy * s[e] * __builtin_fmaf(x[e], 1.f - s[e], 1.f));
  }
}

__global__ __launch_bounds__(kThreads) void decay_grad_reduce_kernel(const float* __restrict__ part,
                                                                     int nch, int H,
                                                                     float* __restrict__ out) {
  __shared__ float ra[kThreads], rb[kThreads];
  const int h = blockIdx.x, tid = threadIdx.x;
  float a = 0.f, b = 0.f;
  for (int c = tid; c < nch; c += kThreads) {
    a += part[((int64_t)c * H + h) * 2 + 0];
    b += part[((int64_t)c * H + h) * 2 + 1];
  }
  ra[tid] = a;
  rb[tid] = b;
  __syncthreads();
  for (int s = kThreads / 2; s > 0; s >>= 1) {
    if (tid < s) {
      ra[tid] += ra[tid + s];
      rb[tid] += rb[tid + s];
    }
    __syncthreads();
  }
  if (tid == 0) {
    out[h] = ra[0];
    out[H + h] = rb[0];
  }
}

template <typename IN, int DK>
hipError_t qk_fwd_t(const void* q, const void* k, void* qh, void* kh, int64_t rows, hipStream_t s) {
  typedef typename std::conditional<sizeof(IN) == 2, f16, float>::type NT;
  const dim3 grid((unsigned)((rows + kWaves - 1) / kWaves), 2);
  hipLaunchKernelGGL((qk_norm_fwd_kernel<IN, NT, DK>), grid, dim3(kThreads), 0, s,
                     reinterpret_cast<const IN*>(q), reinterpret_cast<const IN*>(k),
                     reinterpret_cast<NT*>(qh), reinterpret_cast<NT*>(kh), rows);
  return hipGetLastError();
}

template <typename IN, typename OT, int DK>
hipError_t qk_bwd_t(const void* q, const void* k, const float* dqh, const float* dkh, void* dq,
                    void* dk, int64_t rows, hipStream_t s) {
  const dim3 grid((unsigned)((rows + kWaves - 1) / kWaves), 2);
  hipLaunchKernelGGL((qk_norm_bwd_kernel<IN, OT, DK>), grid, dim3(kThreads), 0, s,
                     reinterpret_cast<const IN*>(q), reinterpret_cast<const IN*>(k), dqh, dkh,
                     reinterpret_cast<OT*>(dq), reinterpret_cast<OT*>(dk), rows);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_qk_norm_fwd(const void* q, const void* k, void* qh, void* kh, int64_t rows,
                              int DK, bool bf16, hipStream_t stream) {
  if (rows == 0) return hipSuccess;
  if (bf16) return DK == 128 ? qk_fwd_t<u16, 128>(q, k, qh, kh, rows, stream)
                             : qk_fwd_t<u16, 64>(q, k, qh, kh, rows, stream);
  return DK == 128 ? qk_fwd_t<float, 128>(q, k, qh, kh, rows, stream)
                   : qk_fwd_t<float, 64>(q, k, qh, kh, rows, stream);
}

hipError_t launch_qk_norm_bwd(const void* q, const void* k, const float* dqh, const float* dkh,
                              void* dq, void* dk, int64_t rows, int DK, bool bf16, bool out_bf16,
                              hipStream_t stream) {
  if (rows == 0) return hipSuccess;
  if (bf16) {
    if (out_bf16) return DK == 128 ? qk_bwd_t<u16, u16, 128>(q, k, dqh, dkh, dq, dk, rows, stream)
                                   : qk_bwd_t<u16, u16, 64>(q, k, dqh, dkh, dq, dk, rows, stream);
    return DK == 128 ? qk_bwd_t<u16, float, 128>(q, k, dqh, dkh, dq, dk, rows, stream)
                     : qk_bwd_t<u16, float, 64>(q, k, dqh, dkh, dq, dk, rows, stream);
  }
  return DK == 128 ? qk_bwd_t<float, float, 128>(q, k, dqh, dkh, dq, dk, rows, stream)
                   : qk_bwd_t<float, float, 64>(q, k, dqh, dkh, dq, dk, rows, stream);
}

hipError_t launch_decay_grad_reduce(const float* partials, int nch, int H, float* out,
                                    hipStream_t stream) {
  if (H == 0) return hipSuccess;
  hipLaunchKernelGGL(decay_grad_reduce_kernel, dim3(H), dim3(kThreads), 0, stream, partials, nch,
                     H, out);
  return hipGetLastError();
}

}  // namespace rla
