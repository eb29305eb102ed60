// Device-side tables for variable-length packing: per-sequence start, length
// and first chunk; per-chunk token range; and a longest-first order of the
// sequences for the state-passing scans.  The host never reads cu_seqlens.
#include "kernels.hpp"

namespace rla {

namespace {

constexpr int kMaxRankedSeqs = 2048;

__device__ __forceinline__ int64_t clamp_tok(int64_t x, int64_t ntok) {
  return x < 0 ? 0 : (x > ntok ? ntok : x);
}

// Sequence n is [m_n, m_{n+1}) where m_i is the running maximum of the
// clamped offsets cu[0..i]: for increasing cu_seqlens this is the usual
// [cu[n], cu[n+1]); any other input yields disjoint (possibly empty)
// sequences, so the chunk count never exceeds ceil(ntok / 64) + nseq.
__global__ __launch_bounds__(kThreads) void seq_table_kernel(const int32_t* cu, int32_t nseq,
                                                             int64_t ntok, SeqInfo* seqs,
                                                             int32_t* nchunks, int32_t* order) {
  __shared__ int64_t mscan[kThreads];
  __shared__ int32_t cscan[kThreads];
  __shared__ int64_t carry_max, last_m;
  __shared__ int32_t carry;
  const int tid = threadIdx.x;
  if (tid == 0) { carry_max = 0; carry = 0; last_m = 0; }
  __syncthreads();
  // pass 1: running maximum of the N+1 clamped offsets -> seqs[n].start
  for (int base = 0; base <= nseq; base += kThreads) {
    const int i = base + tid;
    int64_t x = i <= nseq ? clamp_tok(cu[i], ntok) : 0;
    mscan[tid] = x;
    __syncthreads();
    for (int off = 1; off < kThreads; off <<= 1) {
      const int64_t y = tid >= off ? mscan[tid - off] : 0;
      __syncthreads();
      if (y > mscan[tid]) mscan[tid] = y;
      __syncthreads();
    }
    const int64_t m = mscan[tid] > carry_max ? mscan[tid] : carry_max;
    if (i < nseq) seqs[i].start = m;
    if (i == nseq) last_m = m;
    __syncthreads();
    if (tid == kThreads - 1) carry_max = m;
    __syncthreads();
  }
  __threadfence();
  __syncthreads();
  // pass 2: lengths and first chunks (exclusive scan of chunk counts)
  for (int base = 0; base < nseq; base += kThreads) {
    const int n = base + tid;
    int32_t len = 0;
    if (n < nseq) len = (int32_t)((n + 1 < nseq ? seqs[n + 1].start : last_m) - seqs[n].start);
    const int32_t nch = (len + kChunk - 1) / kChunk;
    cscan[tid] = nch;
    __syncthreads();
    for (int off = 1; off < kThreads; off <<= 1) {   // inclusive Hillis-Steele scan
      const int32_t y = tid >= off ? cscan[tid - off] : 0;
      __syncthreads();
      cscan[tid] += y;
      __syncthreads();
    }
    if (n < nseq) {
      seqs[n].len = len;
      seqs[n].chunk0 = carry + cscan[tid] - nch;
    }
    __syncthreads();
    if (tid == kThreads - 1) carry += cscan[tid];
    __syncthreads();
  }
  if (tid == 0) *nchunks = carry;
  __threadfence();
  __syncthreads();
  // Longest-first order (ties by index); identity beyond kMaxRankedSeqs.
  for (int n = tid; n < nseq; n += kThreads) {
    if (nseq > kMaxRankedSeqs) {
      order[n] = n;
      continue;
    }
    const int32_t len = seqs[n].len;
    int rank = 0;
    for (int m = 0; m < nseq; ++m) {
      const int32_t lm = seqs[m].len;
      rank += (lm > len) || (lm == len && m < n);
    }
    order[rank] = n;
  }
}

__global__ __launch_bounds__(kThreads) void chunk_table_kernel(const SeqInfo* seqs, int32_t nseq,
                                                               const int32_t* nchunks,
                                                               int32_t max_chunks,
                                                               ChunkInfo* chunks) {
  const int c = blockIdx.x * kThreads + threadIdx.x;
  if (c >= max_chunks || c >= *nchunks) return;
  // last sequence whose first chunk is <= c (empty sequences share chunk0
  // with their successor, so the last one found is never empty)
  int lo = 0, hi = nseq - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (seqs[mid].chunk0 <= c) lo = mid;
    else hi = mid - 1;
  }
  const SeqInfo si = seqs[lo];
  const int j = c - si.chunk0;
  const int32_t rem = si.len - j * kChunk;
  chunks[c] = ChunkInfo{si.start + (int64_t)j * kChunk, rem < kChunk ? rem : kChunk, lo};
}

// dst[0 .. n) = 0 for n 4-byte words (16-byte words when aligned).
template <typename W>
__global__ __launch_bounds__(kThreads) void zero_fill_kernel(W* dst, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) dst[i] = W{};
}

}  // namespace

hipError_t launch_zero_fill(void* dst, size_t bytes, hipStream_t stream) {
  if (bytes == 0) return hipSuccess;
  const bool wide = ((uintptr_t)dst % 16 == 0) && (bytes % 16 == 0);
  const int64_t n = (int64_t)(bytes / (wide ? 16 : 4));
  const int64_t blocks = (n + kThreads - 1) / kThreads;
  const unsigned grid = (unsigned)(blocks < 4096 ? blocks : 4096);
  if (wide)
    hipLaunchKernelGGL(zero_fill_kernel<uint4>, dim3(grid), dim3(kThreads), 0, stream,
                       reinterpret_cast<uint4*>(dst), n);
  else
    hipLaunchKernelGGL(zero_fill_kernel<uint32_t>, dim3(grid), dim3(kThreads), 0, stream,
                       reinterpret_cast<uint32_t*>(dst), n);
  return hipGetLastError();
}

hipError_t launch_seq_table(const int32_t* cu, int32_t nseq, int64_t ntok, int32_t max_chunks,
                            SeqInfo* seqs, ChunkInfo* chunks, int32_t* nchunks, int32_t* order,
                            hipStream_t stream) {
  hipLaunchKernelGGL(seq_table_kernel, dim3(1), dim3(kThreads), 0, stream, cu, nseq, ntok, seqs,
                     nchunks, order);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  if (max_chunks > 0) {
    hipLaunchKernelGGL(chunk_table_kernel, dim3((max_chunks + kThreads - 1) / kThreads),
                       dim3(kThreads), 0, stream, seqs, nseq, nchunks, max_chunks, chunks);
  }
  return hipGetLastError();
}

}  // namespace rla
