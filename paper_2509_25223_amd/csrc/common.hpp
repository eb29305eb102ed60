// Device-side building blocks shared by the gfx950 kernels: element types,
// bf16 conversion, MFMA fragment loads from LDS, and the per-launch
// descriptors of sequences and chunks.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace rla {

constexpr int kChunk = 64;      // tokens per chunk
constexpr int kThreads = 256;   // 4 waves of 64 lanes per workgroup
constexpr int kWaves = 4;

typedef unsigned short u16;     // bf16 bit pattern
typedef _Float16 f16;           // fp16
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef u16 u16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef u16 u16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float bf2f(u16 x) { return __uint_as_float(((uint32_t)x) << 16); }

// fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ u16 f2bf(float f) { return __builtin_bit_cast(u16, (__bf16)f); }

// Conversions between the storage type of an operand and fp32.
template <typename T> __device__ __forceinline__ float to_f(T x);
template <> __device__ __forceinline__ float to_f<float>(float x) { return x; }
template <> __device__ __forceinline__ float to_f<u16>(u16 x) { return bf2f(x); }
template <> __device__ __forceinline__ float to_f<f16>(f16 x) { return (float)x; }
template <typename T> __device__ __forceinline__ T from_f(float x);
template <> __device__ __forceinline__ float from_f<float>(float x) { return x; }
template <> __device__ __forceinline__ u16 from_f<u16>(float x) { return f2bf(x); }
// fp32 -> fp16, round to nearest even.  (The build disables the mixed-precision
// FMA instructions, so a preceding fp32 product is never folded into the
// conversion with a single rounding in some template instances only.)
__device__ __forceinline__ f16 to_f16(float x) { return (f16)x; }
template <> __device__ __forceinline__ f16 from_f<f16>(float x) { return to_f16(x); }

// bf16 residual of x after its bf16 rounding hi: x ~= hi + lo to ~16 bits,
// with fp32 range.  Used for state operands (split-bf16 products).
__device__ __forceinline__ u16 bf16_lo(float x, u16 hi) { return f2bf(x - bf2f(hi)); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
// The same split for a pair, as two packed words (first element in the low
// half): hi by one v_cvt_pk_bf16_f32; each residual x - hi, exact in fp32, as
// the bf16 dot product hi . (-1, -0) + x (v_dot2_f32_bf16: bf16 products are
// exact), in place of a shift or mask and a subtraction; lo by one more
// pair conversion.  The zero is -0 so that neither constant matches an
// inline constant: (-1, +0) is emitted as the inline -1.0, which the
// two-operand form reads as the fp32 word 0xBF800000, the pair (0, -1).
__device__ __forceinline__ void bf16_split2(float a, float b, uint32_t& hi, uint32_t& lo) {
  const bf16x2 h = {(__bf16)a, (__bf16)b};
  const float ra = __builtin_amdgcn_fdot2_f32_bf16(h, bf16x2{(__bf16)-1.f, (__bf16)-0.f}, a, false);
  const float rb = __builtin_amdgcn_fdot2_f32_bf16(h, bf16x2{(__bf16)-0.f, (__bf16)-1.f}, b, false);
  hi = __builtin_bit_cast(uint32_t, h);
  lo = __builtin_bit_cast(uint32_t, bf16x2{(__bf16)ra, (__bf16)rb});
}

// ---------------------------------------------------------------------------
// MFMA 16x16 tiles.  One wave computes D[16 x 16] += A[16 x K] * B[K x 16].
//   bf16 (T = u16): v_mfma_f32_16x16x32_bf16, 8 k-values per lane per step.
//   fp32 (T = float): v_mfma_f32_16x16x4_f32, 1 k-value per lane per step.
// A lane supplies row/column (lane & 15) and k-group (lane >> 4) of both
// operands; the sum over k does not depend on which k a (group, slot) pair
// stands for as long as A and B agree, so the k-order inside a step is ours.
// The result lane holds D[4 * (lane >> 4) + r][lane & 15], r = 0..3.
//
// Operands live in LDS and are addressed as logical (r, k) with r the output
// row (A) or column (B) inside the tile:
//   KC layout: element (r, k) at base[r * ld + k]  (k contiguous, vector loads)
//   KS layout: element (r, k) at base[k * ld + r]  (r contiguous, gathers)
// ---------------------------------------------------------------------------
template <typename T> struct Mfma;

template <> struct Mfma<u16> {
  static constexpr int kStep = 32;
  typedef bf16x8 frag;
  template <bool KC>
  __device__ __forceinline__ static frag load(const u16* base, int ld, int k0) {
    const int lane = threadIdx.x & 63;
    const int r = lane & 15, kg = (lane >> 4) * 8;
    if constexpr (KC) {
      const u16x8 v = *reinterpret_cast<const u16x8*>(base + r * ld + k0 + kg);
      return __builtin_bit_cast(frag, v);
    } else {
      u16x8 v;
      const u16* p = base + (k0 + kg) * ld + r;
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = p[e * ld];
      return __builtin_bit_cast(frag, v);
    }
  }
  __device__ __forceinline__ static floatx4 mma(frag a, frag b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};

template <> struct Mfma<f16> {
  static constexpr int kStep = 32;
  typedef f16x8 frag;
  template <bool KC>
  __device__ __forceinline__ static frag load(const f16* base, int ld, int k0) {
    const int lane = threadIdx.x & 63;
    const int r = lane & 15, kg = (lane >> 4) * 8;
    if constexpr (KC) {
      return *reinterpret_cast<const frag*>(base + r * ld + k0 + kg);
    } else {
      frag v;
      const f16* p = base + (k0 + kg) * ld + r;
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = p[e * ld];
      return v;
    }
  }
  __device__ __forceinline__ static floatx4 mma(frag a, frag b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
  }
};

template <> struct Mfma<float> {
  static constexpr int kStep = 4;
  typedef float frag;
  template <bool KC>
  __device__ __forceinline__ static frag load(const float* base, int ld, int k0) {
    const int lane = threadIdx.x & 63;
    const int r = lane & 15, kg = lane >> 4;
    if constexpr (KC) return base[r * ld + k0 + kg];
    else return base[(k0 + kg) * ld + r];
  }
  __device__ __forceinline__ static floatx4 mma(frag a, frag b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

// fp16 MFMA with a 16-deep k step (v_mfma_f32_16x16x16_f16): 4 k-values per
// lane, for contractions over 16-wide blocks.  fp32 uses the 4-deep fp32 MFMA.
template <typename T> struct MfmaK16;

template <> struct MfmaK16<f16> {
  static constexpr int kStep = 16;
  typedef f16x4 frag;
  template <bool KC>
  __device__ __forceinline__ static frag load(const f16* base, int ld, int k0) {
    const int lane = threadIdx.x & 63;
    const int r = lane & 15, kg = (lane >> 4) * 4;
    if constexpr (KC) {
      return *reinterpret_cast<const frag*>(base + r * ld + k0 + kg);
    } else {
      frag v;
      const f16* p = base + (k0 + kg) * ld + r;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = p[e * ld];
      return v;
    }
  }
  __device__ __forceinline__ static floatx4 mma(frag a, frag b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16f16(a, b, c, 0, 0, 0);
  }
};

template <> struct MfmaK16<float> : Mfma<float> {};

// acc += A(16 x K) * B(K x 16) with the MFMA traits M.
template <class M, int K, bool AKC, bool BKC, typename T>
__device__ __forceinline__ void mma_with(floatx4& acc, const T* A, int lda, const T* B, int ldb) {
#pragma unroll
  for (int k0 = 0; k0 < K; k0 += M::kStep) {
    acc = M::mma(M::template load<AKC>(A, lda, k0), M::template load<BKC>(B, ldb, k0), acc);
  }
}

// acc += A(16 x K) * B(K x 16); A and B point at the tile's first row/column.
template <typename T, int K, bool AKC, bool BKC>
__device__ __forceinline__ void mma_tile(floatx4& acc, const T* A, int lda, const T* B, int ldb) {
  typedef Mfma<T> M;
#pragma unroll
  for (int k0 = 0; k0 < K; k0 += M::kStep) {
    acc = M::mma(M::template load<AKC>(A, lda, k0), M::template load<BKC>(B, ldb, k0), acc);
  }
}

// acc += A * B with the A fragments already in registers (afr[k-step]).
template <typename T, int K, bool BKC>
__device__ __forceinline__ void mma_rega(floatx4& acc, const typename Mfma<T>::frag* afr,
                                        const T* B, int ldb) {
  typedef Mfma<T> M;
#pragma unroll
  for (int s = 0; s < K / M::kStep; ++s)
    acc = M::mma(afr[s], M::template load<BKC>(B, ldb, s * M::kStep), acc);
}

// A-operand fragments of a 16-row tile straight from global memory: this
// lane's row pointer (nullptr -> zero row), row-major with k contiguous.
template <typename T, int K>
__device__ __forceinline__ void load_rowfrags(typename Mfma<T>::frag* afr, const T* row) {
  typedef Mfma<T> M;
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int s = 0; s < K / M::kStep; ++s) {
    if constexpr (sizeof(T) == 2) {
      const int k = s * M::kStep + (lane >> 4) * 8;
      u16x8 v = {0, 0, 0, 0, 0, 0, 0, 0};
      if (row) v = *reinterpret_cast<const u16x8*>(row + k);
      afr[s] = __builtin_bit_cast(typename M::frag, v);
    } else {
      const int k = s * M::kStep + (lane >> 4);
      afr[s] = row ? row[k] : 0.f;
    }
  }
}

__device__ __forceinline__ floatx4 zero4() { return floatx4{0.f, 0.f, 0.f, 0.f}; }

// x where ok, else zero, as four bitwise ANDs.  The mask is opaque to the
// optimiser, which would otherwise turn the selection of a loaded value into
// a branch and wait for every outstanding load at its join.
__device__ __forceinline__ uint4 keep_if(uint4 x, bool ok) {
  uint32_t m = ok ? 0xFFFFFFFFu : 0u;
  asm volatile("" : "+v"(m));
  return uint4{x.x & m, x.y & m, x.z & m, x.w & m};
}


// ---------------------------------------------------------------------------
// Row-major LDS tiles without padding: rows of COLS elements of T whose
// 16-byte chunks are XOR-swizzled with sw(row):
//   logical (row r, chunk c) -> physical byte r * kRowB + ((c ^ sw(r)) << 4)
// 128-byte rows: sw(r) = (r & 7) ^ ((r >> 2) & 6); longer rows: sw(r) = r mod
// chunks.  On gfx950 (measured with the LDS bank-conflict counter) this keeps
// conflict-free both the 16-byte MFMA fragment reads (16 rows at one chunk)
// and the 2-byte column gathers of transposed fragments (lane groups reading
// rows 8 apart), where padded rows conflict 2-way.  The swizzle moves whole
// chunks, so 8- and 16-byte pieces stay contiguous.  64 x 64 matrices are
// staged into such tiles by LDS-DMA (the hardware writes lane i's 16 bytes at
// base + 16 i; the lanes pick their global sources to match).
// ---------------------------------------------------------------------------
template <typename T, int COLS> struct Tile {
  static constexpr int kRowB = COLS * (int)sizeof(T);     // bytes per row
  static constexpr int kCpr = kRowB / 16;                 // 16-byte chunks per row
  static_assert(kCpr >= 4 && (kCpr & (kCpr - 1)) == 0, "power-of-two chunks per row");
  static constexpr int kBytes = kChunk * kRowB;           // a 64-row tile
  __device__ __forceinline__ static int sw(int r) {
    return kCpr == 8 ? (r & 7) ^ ((r >> 2) & 6) : r & (kCpr - 1);
  }
  __device__ __forceinline__ static int off(int r, int col) {   // byte offset of element
    const int b = col * (int)sizeof(T);
    return r * kRowB + (((b >> 4) ^ sw(r)) << 4) + (b & 15);
  }
  // For r0 a multiple of 16 and n < 16: sw(r0 + n) = sw(n) ^ sw_hi(r0).
  __device__ __forceinline__ static int sw_hi(int r0) { return kCpr == 8 ? (r0 >> 2) & 4 : 0; }
  // Byte offset of element (r0 + n, column byte cb_lane + cb_uni), r0 a
  // multiple of 16, n < 16, cb_uni a multiple of 16 whose chunk bits do not
  // overlap those of cb_lane: a per-lane part XOR a per-block part, so that
  // every fragment of a tile is one lane offset, one XOR with a wave-uniform
  // value and an immediate offset.
  __device__ __forceinline__ static int off_split(int r0, int n, int cb_lane, int cb_uni) {
    const int lane = n * kRowB + (((cb_lane >> 4) ^ sw(n)) << 4) + (cb_lane & 15);
    return r0 * kRowB + (lane ^ (((cb_uni >> 4) ^ sw_hi(r0)) << 4));
  }
  __device__ __forceinline__ static T* ptr(void* base, int r, int col) {
    return reinterpret_cast<T*>(reinterpret_cast<char*>(base) + off(r, col));
  }
  __device__ __forceinline__ static T at(const void* base, int r, int col) {
    return *reinterpret_cast<const T*>(reinterpret_cast<const char*>(base) + off(r, col));
  }
  // MFMA fragment of rows r0 .. r0+15 (r0 a multiple of 16) at k = k0 (k runs
  // along a row, k0 a multiple of the MFMA k-step)
  template <typename M>
  __device__ __forceinline__ static typename M::frag frag(const void* base, int r0, int k0) {
    constexpr int kPL = M::kStep / 4;   // k-values per lane
    const int lane = threadIdx.x & 63;
    return *reinterpret_cast<const typename M::frag*>(
        reinterpret_cast<const char*>(base) +
        off_split(r0, lane & 15, kPL * (lane >> 4) * (int)sizeof(T), k0 * (int)sizeof(T)));
  }
};
template <typename T> using Swz = Tile<T, kChunk>;   // 64 x 64 matrices

// The chunk matrices are lower block-triangular in 16 x 16 blocks.  Only the
// 10 blocks on and below the diagonal are stored, each row-major, block
// (bi, bj), bj <= bi, at index bi (bi + 1) / 2 + bj; the blocks above the
// diagonal are zero.  Each stored matrix is followed by 64 zero elements,
// the source of the LDS-DMA lanes that fill the blocks above the diagonal.
constexpr int kMatBlocks = 10;
constexpr int kMatPacked = kMatBlocks * 256;   // elements of the stored blocks
constexpr int kMatElems = kMatPacked + 64;     // per matrix, with the zero pad
__host__ __device__ constexpr int tri_off(int t, int s) {
  return (((t >> 4) * ((t >> 4) + 1)) / 2 + (s >> 4)) * 256 + (t & 15) * 16 + (s & 15);
}

// LDS transpose read of 16-bit elements (gfx950 ds_read_b64_tr_b16).  In each
// 16-lane group, the 8-byte pieces the lanes address form a 16 x 4 array D
// (row j: the group's lane j); lane i of the group receives D[i / 4 + 4 e][i % 4]
// for e = 0 .. 3.
__device__ __forceinline__ u16x4 lds_read_tr16(const void* p) {
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  const s16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(p));
  return __builtin_bit_cast(u16x4, r);
}

// Token-major 16 bytes from a value-major tile of 16-bit elements (tile rows
// = values, columns = 64 tokens): lane L receives rows j0 .. j0+7 of column L
// (j0 a multiple of 4).  Two transpose reads: the group of lanes 16 g .. 16 g
// + 15 addresses 4 rows x 16 columns from column 16 g, 4 columns per lane.
template <class TL>
__device__ __forceinline__ uint4 tile_token_vec8(const void* base, int j0) {
  static_assert(sizeof(typename std::remove_pointer<decltype(TL::ptr(nullptr, 0, 0))>::type) == 2,
                "16-bit tile");
  const int lane = threadIdx.x & 63, jj = lane & 15;
  const int t = 16 * (lane >> 4) + 4 * (jj & 3), j = j0 + (jj >> 2);
  const char* b = reinterpret_cast<const char*>(base);
  const u16x4 a = lds_read_tr16(b + TL::off(j, t));
  const u16x4 c = lds_read_tr16(b + TL::off(j + 4, t));
  return uint4{a[0] | ((uint32_t)a[1] << 16), a[2] | ((uint32_t)a[3] << 16),
               c[0] | ((uint32_t)c[1] << 16), c[2] | ((uint32_t)c[3] << 16)};
}

// tile_token_vec8 with its two transpose reads issued as inline assembly, so
// that the compiler does not drain the wave's in-flight LDS-DMA before them;
// the function waits for its own reads (lgkmcnt(0), tied to their registers).
template <class TL>
__device__ __forceinline__ uint4 tile_token_vec8_sync(const void* base, int j0) {
  typedef __attribute__((address_space(3))) const char* lds_ptr;
  const int lane = threadIdx.x & 63, jj = lane & 15;
  const int t = 16 * (lane >> 4) + 4 * (jj & 3), j = j0 + (jj >> 2);
  const char* b = reinterpret_cast<const char*>(base);
  const uint32_t a0 = (uint32_t)(uintptr_t)(lds_ptr)(b + TL::off(j, t));
  const uint32_t a1 = (uint32_t)(uintptr_t)(lds_ptr)(b + TL::off(j + 4, t));
  u16x4 a, c;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(a) : "v"(a0));
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(c) : "v"(a1));
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(c));
  return uint4{a[0] | ((uint32_t)a[1] << 16), a[2] | ((uint32_t)a[3] << 16),
               c[0] | ((uint32_t)c[1] << 16), c[2] | ((uint32_t)c[3] << 16)};
}

// Token-major 16 bytes of a value-major tile of 16-bit elements (tile rows =
// values, columns = 64 tokens), 16 tokens per instruction: lane (g, i) (g =
// lane / 16, i = lane % 16) receives rows 8 g .. 8 g + 7 of column t0 + i, so
// the four lanes of a token hold 32 consecutive values (a 64-byte store
// segment).  Two transpose reads as inline assembly (no drain of in-flight
// LDS-DMA), waited for by the function.
template <class TL>
__device__ __forceinline__ uint4 tile_token_rows16_sync(const void* base, int t0) {
  typedef __attribute__((address_space(3))) const char* lds_ptr;
  const int lane = threadIdx.x & 63, jj = lane & 15;
  const int t = t0 + 4 * (jj & 3), j = 8 * (lane >> 4) + (jj >> 2);
  const char* b = reinterpret_cast<const char*>(base);
  const uint32_t a0 = (uint32_t)(uintptr_t)(lds_ptr)(b + TL::off(j, t));
  const uint32_t a1 = (uint32_t)(uintptr_t)(lds_ptr)(b + TL::off(j + 4, t));
  u16x4 a, c;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(a) : "v"(a0));
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(c) : "v"(a1));
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(c));
  return uint4{a[0] | ((uint32_t)a[1] << 16), a[2] | ((uint32_t)a[3] << 16),
               c[0] | ((uint32_t)c[1] << 16), c[2] | ((uint32_t)c[3] << 16)};
}

// Four 4-byte LDS values at p, p + stride, p + 2 stride, p + 3 stride (bytes)
// as 16 bytes, issued as inline assembly like lds_read16_sync (no drain of
// in-flight LDS-DMA) and waited for by the function.
__device__ __forceinline__ uint4 lds_read4x1_sync(const void* p, int stride) {
  typedef __attribute__((address_space(3))) const char* lds_ptr;
  const uint32_t a = (uint32_t)(uintptr_t)(lds_ptr)(reinterpret_cast<const char*>(p));
  uint32_t x, y, z, w;
  asm volatile("ds_read_b32 %0, %1" : "=v"(x) : "v"(a));
  asm volatile("ds_read_b32 %0, %1" : "=v"(y) : "v"(a + stride));
  asm volatile("ds_read_b32 %0, %1" : "=v"(z) : "v"(a + 2 * stride));
  asm volatile("ds_read_b32 %0, %1" : "=v"(w) : "v"(a + 3 * stride));
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(x), "+v"(y), "+v"(z), "+v"(w));
  return uint4{x, y, z, w};
}

// 16 bytes from LDS, issued as inline assembly so that the compiler does not
// drain the wave's in-flight LDS-DMA before it (it cannot always prove the
// addresses disjoint); waits for its own read.
__device__ __forceinline__ uint4 lds_read16_sync(const void* p) {
  typedef __attribute__((address_space(3))) const char* lds_ptr;
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const uint32_t a = (uint32_t)(uintptr_t)(lds_ptr)(reinterpret_cast<const char*>(p));
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a));
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(v));
  return uint4{v[0], v[1], v[2], v[3]};
}

// A 64-row tile of 16-bit elements stored row-major (COLS per row, written
// in 16-byte pieces) and read back as MFMA fragments of its transpose:
// frag(base, r0, k0) holds rows r0 .. r0+15 of the transpose (tile columns)
// at k = k0 .. k0+31 (tile rows), from two transpose reads.  The 16-byte
// chunks of row r are XOR-swizzled by 2 (r & 7) (within the row's chunks):
// the four rows that each 16-lane group of a transpose read touches, and
// eight consecutive rows of one chunk column, fall in distinct banks.
template <typename T, int COLS> struct TrTile {
  static_assert(sizeof(T) == 2, "16-bit elements");
  static constexpr int kRowB = COLS * 2;
  static constexpr int kCpr = kRowB / 16;
  static_assert(kCpr >= 8 && (kCpr & (kCpr - 1)) == 0, "power-of-two chunks per row");
  __device__ __forceinline__ static int sw(int r) { return (2 * (r & 7)) & (kCpr - 1); }
  __device__ __forceinline__ static int off(int r, int col) {
    const int b = col * 2;
    return r * kRowB + (((b >> 4) ^ sw(r)) << 4) + (b & 15);
  }
  __device__ __forceinline__ static T* ptr(void* base, int r, int col) {
    return reinterpret_cast<T*>(reinterpret_cast<char*>(base) + off(r, col));
  }
  template <typename M>
  __device__ __forceinline__ static typename M::frag frag(const void* base, int r0, int k0);
};

// MFMA fragment (16-bit, k-step 32) of the transpose of a row-major tile TL:
// rows r0 .. r0+15 of the transpose (tile columns) at k = k0 .. k0+31 (tile
// rows), from two transpose reads.  Lane j of each 16-lane group g addresses
// tile row k0 + 8 g + j / 4 (and 4 rows further for the second read) at
// columns r0 + 4 (j % 4) .. +3, which TL must keep in one aligned 8 bytes.
template <class TL, typename M>
__device__ __forceinline__ typename M::frag frag_tr(const void* base, int r0, int k0) {
  static_assert(M::kStep == 32, "8 k-values per lane");
  const int lane = threadIdx.x & 63, jj = lane & 15;
  const int row = k0 + 8 * (lane >> 4) + (jj >> 2), col = r0 + 4 * (jj & 3);
  const char* b = reinterpret_cast<const char*>(base);
  const u16x4 x = lds_read_tr16(b + TL::off(row, col));
  const u16x4 y = lds_read_tr16(b + TL::off(row + 4, col));
  const u16x8 v = {x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
  return __builtin_bit_cast(typename M::frag, v);
}

// Rows r0 .. r0+15, columns c0 .. c0+15 of a row-major 16-bit tile TL in the
// MFMA accumulator layout (lane: rows r0 + 4 (lane / 16) + 0..3, column
// c0 + lane % 16), from one transpose read: lane j of group g addresses row
// r0 + 4 g + j / 4 at columns c0 + 4 (j % 4) .. +3.
template <class TL>
__device__ __forceinline__ u16x4 acc_tile_tr(const void* base, int r0, int c0) {
  const int lane = threadIdx.x & 63, jj = lane & 15;
  const int row = r0 + 4 * (lane >> 4) + (jj >> 2), col = c0 + 4 * (jj & 3);
  return lds_read_tr16(reinterpret_cast<const char*>(base) + TL::off(row, col));
}

template <typename T, int COLS>
template <typename M>
__device__ __forceinline__ typename M::frag TrTile<T, COLS>::frag(const void* base, int r0, int k0) {
  return frag_tr<TrTile<T, COLS>, M>(base, r0, k0);
}

// Same interface over plain rows padded to COLS + PAD elements: cheaper
// addressing for buffers written element by element (transposes).
template <typename T, int COLS, int PAD> struct PadRows {
  static constexpr int kRowB = (COLS + PAD) * (int)sizeof(T);
  __device__ __forceinline__ static int off(int r, int col) { return r * kRowB + col * (int)sizeof(T); }
  __device__ __forceinline__ static int off_split(int r0, int n, int cb_lane, int cb_uni) {
    return (r0 + n) * kRowB + cb_lane + cb_uni;
  }
  __device__ __forceinline__ static T* ptr(void* base, int r, int col) {
    return reinterpret_cast<T*>(reinterpret_cast<char*>(base) + off(r, col));
  }
  __device__ __forceinline__ static T at(const void* base, int r, int col) {
    return *reinterpret_cast<const T*>(reinterpret_cast<const char*>(base) + off(r, col));
  }
  template <typename M>
  __device__ __forceinline__ static typename M::frag frag(const void* base, int r0, int k0) {
    constexpr int kPL = M::kStep / 4;
    const int lane = threadIdx.x & 63;
    return *reinterpret_cast<const typename M::frag*>(
        reinterpret_cast<const char*>(base) + off(r0 + (lane & 15), k0 + kPL * (lane >> 4)));
  }
};

// One LDS-DMA instruction: lane i copies 16 bytes from `src` (its own global
// address) to `lds` + 16 i.  (Pointers go through char* so that the builtin
// type-checks in the host pass too.)
__device__ __forceinline__ void dma16(const void* src, void* lds) {
  __builtin_amdgcn_global_load_lds(reinterpret_cast<const char*>(src),
                                   reinterpret_cast<char*>(lds), 16, 0, 0);
}

// LDS-DMA of 64 contiguous rows (global, row-major, unswizzled) into a tile;
// each of the NW waves of the workgroup issues an equal share of the 1 KiB
// instructions.  Completion: s_waitcnt vmcnt + barrier.
template <class TL, int NW>
__device__ __forceinline__ void dma_tile64(const void* gsrc, void* lds) {
  constexpr int kInst = kChunk * TL::kRowB / 1024;
  static_assert(kInst % NW == 0, "equal DMA share per wave");
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int m = 0; m < kInst / NW; ++m) {
    const int blk = w * (kInst / NW) + m;
    const int P = blk * 64 + lane;                  // physical 16-byte chunk
    const int r = P / TL::kCpr, c = (P % TL::kCpr) ^ TL::sw(r);   // logical chunk stored there
    dma16(reinterpret_cast<const char*>(gsrc) + (uint32_t)(r * TL::kRowB + c * 16),
          reinterpret_cast<char*>(lds) + blk * 1024);
  }
}

// This lane's source offsets (bytes, from the start of a stored matrix) for
// the LDS-DMA of a packed matrix into a swizzled 64 x 64 tile by NW waves:
// the element of tri_off at the lane's 16-byte chunk, or the zero pad for
// the chunks above the diagonal blocks.  The same for every matrix and
// chunk, so computed once.
template <typename T, int NW = kWaves>
struct MatDma {
  static constexpr int kInst = kChunk * Swz<T>::kRowB / 1024;
  static constexpr int kPerWave = kInst / NW;
  static_assert(kInst % NW == 0, "equal DMA share per wave");
  int off[kPerWave];
  __device__ __forceinline__ MatDma() : MatDma(threadIdx.x >> 6) {}
  // w: this wave's index among the NW waves that issue the copy
  __device__ __forceinline__ explicit MatDma(int w) {
    typedef Swz<T> TL;
    constexpr int kEpc = 16 / (int)sizeof(T);   // elements per 16-byte chunk
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int m = 0; m < kPerWave; ++m) {
      const int P = (w * kPerWave + m) * 64 + lane;   // physical 16-byte chunk
      const int r = P / TL::kCpr, col = ((P % TL::kCpr) ^ TL::sw(r)) * kEpc;   // its logical position
      off[m] = ((col >> 4) <= (r >> 4) ? tri_off(r, col) : kMatPacked) * (int)sizeof(T);
    }
  }
};

// DMA of one packed lower block-triangular 64 x 64 matrix (global, tri_off
// layout, followed by its zero pad) into a swizzled LDS tile by the NW waves
// of the workgroup: no lane is masked and no branch is taken.
template <typename T, int NW = kWaves>
__device__ __forceinline__ void dma_mat64(const T* gsrc, T* lds, const MatDma<T, NW>& md, int w) {
#pragma unroll
  for (int m = 0; m < MatDma<T, NW>::kPerWave; ++m)
    dma16(reinterpret_cast<const char*>(gsrc) + md.off[m],
          reinterpret_cast<char*>(lds) + (w * MatDma<T, NW>::kPerWave + m) * 1024);
}

template <typename T, int NW = kWaves>
__device__ __forceinline__ void dma_mat64(const T* gsrc, T* lds, const MatDma<T, NW>& md) {
  dma_mat64<T, NW>(gsrc, lds, md, threadIdx.x >> 6);
}

// DMA of `bytes` contiguous bytes (a multiple of 1 KiB) by wave `wave` only.
__device__ __forceinline__ void dma_linear_wave(const void* gsrc, void* lds, int bytes) {
  const int lane = threadIdx.x & 63;
  for (int b = 0; b < bytes; b += 1024)
    dma16(reinterpret_cast<const char*>(gsrc) + (uint32_t)(b + lane * 16), reinterpret_cast<char*>(lds) + b);
}

// Waits for this wave's outstanding vector memory operations (loads, stores
// and LDS-DMA): s_waitcnt vmcnt(0).  A barrier afterwards makes every wave's
// DMA data visible.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// s_waitcnt vmcnt(N): waits until at most N of this wave's vector memory
// operations are outstanding.  They complete in issue order (loads, stores
// and LDS-DMA share the counter), so with the last N operations being stores
// this waits for every earlier load but not for those stores' acknowledgement.
template <int N>
__device__ __forceinline__ void wait_vmem_but() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
  asm volatile("" ::: "memory");
}

// Workgroup barrier for LDS data: waits for this wave's LDS operations
// (lgkmcnt(0)) and meets the other waves, but leaves global loads, stores and
// LDS-DMA in flight (__syncthreads' release fence would drain them).  LDS-DMA
// data is published by wait_vmem() before such a barrier.
__device__ __forceinline__ void barrier_lds() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// A-operand fragment of a swizzled matrix: rows r0..r0+15 ("KC": row-major use).
template <typename T>
__device__ __forceinline__ typename Mfma<T>::frag swz_load_rows(const T* base, int r0, int k0) {
  typedef Mfma<T> M;
  const int lane = threadIdx.x & 63;
  const int r = r0 + (lane & 15);
  const char* b = reinterpret_cast<const char*>(base);
  if constexpr (sizeof(T) == 2) {
    return *reinterpret_cast<const typename M::frag*>(b + Swz<T>::off(r, k0 + (lane >> 4) * 8));
  } else {
    return *reinterpret_cast<const float*>(b + Swz<T>::off(r, k0 + (lane >> 4)));
  }
}

// A-operand fragment of the TRANSPOSE of a swizzled matrix: A(t, s) = M[s][t]
// for t = t0..t0+15 (gathers).
template <typename T>
__device__ __forceinline__ typename Mfma<T>::frag swz_load_cols(const T* base, int t0, int k0) {
  typedef Mfma<T> M;
  const int lane = threadIdx.x & 63;
  const int t = t0 + (lane & 15);
  const char* b = reinterpret_cast<const char*>(base);
  if constexpr (sizeof(T) == 2) {
    typename M::frag v;
    const int s0 = k0 + (lane >> 4) * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = *reinterpret_cast<const T*>(b + Swz<T>::off(s0 + e, t));
    return v;
  } else {
    return *reinterpret_cast<const float*>(b + Swz<T>::off(k0 + (lane >> 4), t));
  }
}

// acc += M[r0.., :] * B, M a swizzled 64 x 64 matrix, B^T rows b0.. of a
// 64-token tile (row n of B^T = column n of B)
template <typename T, class TB = Swz<T>>
__device__ __forceinline__ void mma_swz_rows(floatx4& acc, const T* M, int r0, const void* B, int b0) {
  typedef Mfma<T> F;
#pragma unroll
  for (int k0 = 0; k0 < kChunk; k0 += F::kStep)
    acc = F::mma(swz_load_rows<T>(M, r0, k0), TB::template frag<F>(B, b0, k0), acc);
}

// acc += M^T[t0.., :] * B
template <typename T, class TB = Swz<T>>
__device__ __forceinline__ void mma_swz_cols(floatx4& acc, const T* M, int t0, const void* B, int b0) {
  typedef Mfma<T> F;
#pragma unroll
  for (int k0 = 0; k0 < kChunk; k0 += F::kStep)
    acc = F::mma(swz_load_cols<T>(M, t0, k0), TB::template frag<F>(B, b0, k0), acc);
}

// The A fragments of rows r0..r0+15 of a swizzled 64 x 64 matrix (or of its
// transpose), every k-step, loaded ahead of use (e.g. before a barrier).
template <typename T> struct MatFrags {
  typename Mfma<T>::frag f[kChunk / Mfma<T>::kStep];
};
template <typename T>
__device__ __forceinline__ MatFrags<T> swz_rows_frags(const T* M, int r0) {
  MatFrags<T> a;
#pragma unroll
  for (int s = 0; s < kChunk / Mfma<T>::kStep; ++s) a.f[s] = swz_load_rows<T>(M, r0, s * Mfma<T>::kStep);
  return a;
}
// ---------------------------------------------------------------------------
// Chunk matrices kept in LDS as stored in global memory: the ten 16 x 16
// blocks on and below the diagonal (tri_off order, 512 bytes each in fp16),
// copied by five 1 KiB LDS-DMA instructions.  Inside a block, row r's two
// 16-byte halves sit at 16-byte positions pk_pos<COLS>(r, h), arranged for
// the one kind of read the matrix gets.  For row fragments (COLS false) rows
// 8 .. 15 swap their halves, so that the 16 rows a read touches at one half
// fall in distinct banks; for transposed column fragments (COLS true) rows
// 8 .. 11 and 12 .. 15 trade places, so that rows 0..3 and 8..11 (4..7 and
// 12..15), read together, fall in distinct banks.  Reads of blocks above the
// diagonal go to a shared 16-byte zero region.
// ---------------------------------------------------------------------------
constexpr int kPkBytes = kMatPacked * 2;   // fp16 matrix in LDS (5 KiB)

// 16-byte position inside a block of row r's half h (an involution)
template <bool COLS>
__device__ __forceinline__ int pk_pos(int r, int h) {
  return COLS ? (r ^ ((r >> 3) << 2)) * 2 + h : r * 2 + (h ^ (r >> 3));
}

// LDS-DMA of one packed fp16 matrix (global tri_off layout) into LDS by wave
// w (0 .. nw - 1) of the nw waves sharing the copy: the wave issues the
// instructions w, w + nw, .. of the five.
template <bool COLS>
__device__ __forceinline__ void dma_mat_packed(const f16* gsrc, f16* lds, int w, int nw) {
  const int lane = threadIdx.x & 63;
  for (int i = w; i < kPkBytes / 1024; i += nw) {
    const int P = i * 64 + lane;                    // LDS 16-byte chunk
    const int b = P >> 5, rh = pk_pos<COLS>((P & 31) >> 1, P & 1);   // the (row, half) stored there
    dma16(reinterpret_cast<const char*>(gsrc) + (uint32_t)((b * 32 + rh) * 16),
          reinterpret_cast<char*>(lds) + i * 1024);
  }
}

// A-operand fragments (MatFrags) of rows 16 bi .. 16 bi + 15 of a packed
// fp16 matrix in LDS; `zero` is 16 zero bytes in LDS.
__device__ __forceinline__ MatFrags<f16> packed_rows_frags(const f16* M, int bi, const f16* zero) {
  const int lane = threadIdx.x & 63, r = lane & 15, q = lane >> 4;
  MatFrags<f16> a;
#pragma unroll
  for (int s = 0; s < kChunk / 32; ++s) {
    const int bj = 2 * s + (q >> 1);
    const int off = ((bi * (bi + 1) / 2 + bj) * 32 + pk_pos<false>(r, q & 1)) * 16;
    const char* src = bj <= bi ? reinterpret_cast<const char*>(M) + off : reinterpret_cast<const char*>(zero);
    a.f[s] = *reinterpret_cast<const typename Mfma<f16>::frag*>(src);
  }
  return a;
}

// A-operand fragments of rows 16 bj .. 16 bj + 15 of the transpose of a
// packed fp16 matrix in LDS (its columns 16 bj ..), from transpose reads as
// in swz_cols_frags_sync (inline assembly, waited for inside, so that the
// compiler does not drain in-flight LDS-DMA first); `zero` is 16 zero bytes
// in LDS.  Lane (q, j) of the read for k-rows 32 s + 8 q + 4 n .. addresses
// 4 elements of matrix row 32 s + 8 q + (j >> 2) + 4 n at column
// 16 bj + 4 (j & 3).
__device__ __forceinline__ MatFrags<f16> packed_cols_frags_sync(const f16* M, int bj, const f16* zero) {
  typedef __attribute__((address_space(3))) const char* lds_ptr;
  const int lane = threadIdx.x & 63, j = lane & 15, q = lane >> 4;
  const int h = (j & 3) >> 1, sub = (j & 1) * 8;
  const char* b = reinterpret_cast<const char*>(M);
  u16x4 x[2], y[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int bi = 2 * s + (q >> 1), r = 8 * (q & 1) + (j >> 2);
    const int blk = (bi * (bi + 1) / 2 + bj) * 512;
    const char* p0 = bj <= bi ? b + blk + pk_pos<true>(r, h) * 16 + sub : reinterpret_cast<const char*>(zero);
    const char* p1 = bj <= bi ? b + blk + pk_pos<true>(r + 4, h) * 16 + sub : reinterpret_cast<const char*>(zero);
    const uint32_t a0 = (uint32_t)(uintptr_t)(lds_ptr)(p0);
    const uint32_t a1 = (uint32_t)(uintptr_t)(lds_ptr)(p1);
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(x[s]) : "v"(a0));
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(y[s]) : "v"(a1));
  }
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(x[0]), "+v"(y[0]), "+v"(x[1]), "+v"(y[1]));
  MatFrags<f16> a;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const u16x8 v = {x[s][0], x[s][1], x[s][2], x[s][3], y[s][0], y[s][1], y[s][2], y[s][3]};
    a.f[s] = __builtin_bit_cast(typename Mfma<f16>::frag, v);
  }
  return a;
}

template <typename T>
__device__ __forceinline__ MatFrags<T> swz_cols_frags(const T* M, int t0) {
  MatFrags<T> a;
#pragma unroll
  for (int s = 0; s < kChunk / Mfma<T>::kStep; ++s) a.f[s] = swz_load_cols<T>(M, t0, s * Mfma<T>::kStep);
  return a;
}
// The 16-bit transpose fragments of swz_cols_frags from transpose reads
// (two per fragment instead of eight 16-bit gathers), issued as inline
// assembly so that the compiler does not drain the wave's in-flight LDS-DMA
// before them.  The compiler does not see these reads either, so the
// function waits for them itself (lgkmcnt(0), tied to their registers so
// that nothing reads them earlier); meant for fragments loaded just before a
// barrier, which waits the same way.
template <typename T>
__device__ __forceinline__ MatFrags<T> swz_cols_frags_sync(const T* M, int t0) {
  static_assert(sizeof(T) == 2 && Mfma<T>::kStep == 32 && kChunk == 64, "two 16-bit k-steps");
  typedef Swz<T> TL;
  typedef __attribute__((address_space(3))) const char* lds_ptr;
  const int lane = threadIdx.x & 63, jj = lane & 15;
  const int col = t0 + 4 * (jj & 3);
  const char* b = reinterpret_cast<const char*>(M);
  u16x4 x[2], y[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int row = 32 * s + 8 * (lane >> 4) + (jj >> 2);
    const uint32_t a0 = (uint32_t)(uintptr_t)(lds_ptr)(b + TL::off(row, col));
    const uint32_t a1 = (uint32_t)(uintptr_t)(lds_ptr)(b + TL::off(row + 4, col));
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(x[s]) : "v"(a0));
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(y[s]) : "v"(a1));
  }
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(x[0]), "+v"(y[0]), "+v"(x[1]), "+v"(y[1]));
  MatFrags<T> a;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const u16x8 v = {x[s][0], x[s][1], x[s][2], x[s][3], y[s][0], y[s][1], y[s][2], y[s][3]};
    a.f[s] = __builtin_bit_cast(typename Mfma<T>::frag, v);
  }
  return a;
}
// frag_tr for N fragments (tile-transpose rows r0[n], k = k0[n] ..) issued
// as inline assembly, so that the compiler does not drain the wave's
// in-flight LDS-DMA and stores before them; the function waits for its own
// reads (lgkmcnt(0)) and ties the results to that wait.
template <class TL, typename T, int N>
__device__ __forceinline__ void frags_tr_sync(const void* base, const int (&r0)[N], const int (&k0)[N],
                                              typename Mfma<T>::frag (&f)[N]) {
  static_assert(sizeof(T) == 2 && Mfma<T>::kStep == 32, "16-bit k-steps of 32");
  typedef __attribute__((address_space(3))) const char* lds_ptr;
  const int lane = threadIdx.x & 63, jj = lane & 15;
  const char* b = reinterpret_cast<const char*>(base);
  u16x4 x[N], y[N];
#pragma unroll
  for (int n = 0; n < N; ++n) {
    const int row = k0[n] + 8 * (lane >> 4) + (jj >> 2), col = r0[n] + 4 * (jj & 3);
    const uint32_t a0 = (uint32_t)(uintptr_t)(lds_ptr)(b + TL::off(row, col));
    const uint32_t a1 = (uint32_t)(uintptr_t)(lds_ptr)(b + TL::off(row + 4, col));
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(x[n]) : "v"(a0));
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(y[n]) : "v"(a1));
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int n = 0; n < N; ++n) {
    asm volatile("" : "+v"(x[n]), "+v"(y[n]));
    const u16x8 v = {x[n][0], x[n][1], x[n][2], x[n][3], y[n][0], y[n][1], y[n][2], y[n][3]};
    f[n] = __builtin_bit_cast(typename Mfma<T>::frag, v);
  }
}

// acc += A * B with A from MatFrags and B^T rows b0.. of a 64-token tile
template <typename T, class TB = Swz<T>>
__device__ __forceinline__ void mma_frags(floatx4& acc, const MatFrags<T>& a, const void* B, int b0) {
  typedef Mfma<T> F;
#pragma unroll
  for (int s = 0; s < kChunk / F::kStep; ++s)
    acc = F::mma(a.f[s], TB::template frag<F>(B, b0, s * F::kStep), acc);
}

// acc += A(rows a0.., :K) * B(rows b0.., :K)^T with both operands in tiles
template <typename T, int K, class TA, class TB>
__device__ __forceinline__ void mma_tiles(floatx4& acc, const void* A, int a0, const void* B, int b0) {
  typedef Mfma<T> F;
#pragma unroll
  for (int k0 = 0; k0 < K; k0 += F::kStep)
    acc = F::mma(TA::template frag<F>(A, a0, k0), TB::template frag<F>(B, b0, k0), acc);
}

// acc += A * B(rows b0.., :K)^T with the A fragments in registers (afr[k-step])
template <typename T, int K, class TB>
__device__ __forceinline__ void mma_rega_tile(floatx4& acc, const typename Mfma<T>::frag* afr,
                                              const void* B, int b0) {
  typedef Mfma<T> F;
#pragma unroll
  for (int s = 0; s < K / F::kStep; ++s)
    acc = F::mma(afr[s], TB::template frag<F>(B, b0, s * F::kStep), acc);
}

// Row (inside a 16-row tile) and column of accumulator element r of this lane.
__device__ __forceinline__ int acc_row(int r) { return 4 * ((threadIdx.x & 63) >> 4) + r; }
__device__ __forceinline__ int acc_col() { return threadIdx.x & 15; }

// DPP lane exchange inside a row of 16 lanes.
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL,
                                                                0xF, 0xF, false));
}

// Sum / max over aligned groups of N lanes (N = 2, 4, 8, 16) inside a 16-lane
// row; every lane of a group gets the result.
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  x += dpp<0xB1>(x);                         // quad_perm [1,0,3,2]
  if constexpr (N >= 4) x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
  if constexpr (N >= 8) x += dpp<0x141>(x);  // row_half_mirror
  if constexpr (N >= 16) x += dpp<0x140>(x); // row_mirror
  return x;
}
template <int N>
__device__ __forceinline__ float group_max(float x) {
  x = fmaxf(x, dpp<0xB1>(x));
  if constexpr (N >= 4) x = fmaxf(x, dpp<0x4E>(x));
  if constexpr (N >= 8) x = fmaxf(x, dpp<0x141>(x));
  if constexpr (N >= 16) x = fmaxf(x, dpp<0x140>(x));
  return x;
}

// Power-of-two scale 2^e for a block of values whose largest magnitude has
// the fp32 bit pattern mbits: e = (biased exponent) - 140, so that the largest
// magnitude over 2^e lies in [2^13, 2^14) and the block stored as fp16 keeps
// fp16's full relative precision for its largest entries without overflow.
// e is at least -126; blocks of zeros (or subnormals only) get e = 0.
__device__ __forceinline__ int pow2_scale_exp(uint32_t mbits) {
  const int be = (int)(mbits >> 23);
  return be == 0 ? 0 : max(be - 140, -126);
}
__device__ __forceinline__ float exp2_int(int e) {   // 2^e, -126 <= e <= 127
  return __uint_as_float((uint32_t)(e + 127) << 23);
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, false);
}

// Largest |x| over a 16-lane row, as an fp32 bit pattern (unsigned compares
// of the magnitude bits, which fold into DPP max instructions).
__device__ __forceinline__ uint32_t row16_absmax_bits(float a, float b) {
  uint32_t m = max(__float_as_uint(a) & 0x7FFFFFFFu, __float_as_uint(b) & 0x7FFFFFFFu);
  m = max(m, dpp_u32<0xB1>(m));
  m = max(m, dpp_u32<0x4E>(m));
  m = max(m, dpp_u32<0x141>(m));
  return max(m, dpp_u32<0x140>(m));
}

// Largest |x| over a wave, as an fp32 bit pattern (wave-uniform): the lane's
// own magnitudes m (bits), then over each 16-lane row and the four rows.
__device__ __forceinline__ uint32_t wave_absmax_bits(uint32_t m) {
  m = max(m, dpp_u32<0xB1>(m));
  m = max(m, dpp_u32<0x4E>(m));
  m = max(m, dpp_u32<0x141>(m));
  m = max(m, dpp_u32<0x140>(m));
  return max(max((uint32_t)__builtin_amdgcn_readlane((int)m, 0), (uint32_t)__builtin_amdgcn_readlane((int)m, 16)),
             max((uint32_t)__builtin_amdgcn_readlane((int)m, 32), (uint32_t)__builtin_amdgcn_readlane((int)m, 48)));
}

// Largest of four values per lane over the wave, the four reduced together
// (a transpose-reduce): exchanges with lanes c ^ 1 and c ^ 2 inside each quad
// leave lane c (c = lane % 16) with the quad's largest v[2 (c & 1) + ((c >> 1)
// & 1)], rotations by 8 and 4 inside the 16-lane row and exchanges across
// rows then give every lane that value's wave maximum; lanes 0, 2, 1, 3 hold
// those of v[0], v[1], v[2], v[3].  Unsigned maxima (fp32 magnitude bits):
// exact, so the order does not matter.
__device__ __forceinline__ uint32_t wave_max4_bits(const uint32_t (&v)[4]) {
  const int lane = threadIdx.x & 63;
  const bool b0 = lane & 1, b1 = lane & 2;
  const uint32_t x0 = max(b0 ? v[2] : v[0], dpp_u32<0xB1>(b0 ? v[0] : v[2]));   // quad_perm [1,0,3,2]
  const uint32_t x1 = max(b0 ? v[3] : v[1], dpp_u32<0xB1>(b0 ? v[1] : v[3]));
  uint32_t y = max(b1 ? x1 : x0, dpp_u32<0x4E>(b1 ? x0 : x1));                  // quad_perm [2,3,0,1]
  y = max(y, dpp_u32<0x128>(y));   // row_ror:8
  y = max(y, dpp_u32<0x124>(y));   // row_ror:4
  y = max(y, (uint32_t)__shfl_xor((int)y, 16, 64));
  return max(y, (uint32_t)__shfl_xor((int)y, 32, 64));
}

// 4 x 4 transpose across the lanes of each quad (lanes 4g + i, i = 0..3): lane
// i enters with x[r] = M[i][r] and leaves with x[r] = M[r][i].  Two exchange
// rounds, with lane i ^ 1 for the registers whose index differs from i in bit
// 0, then with lane i ^ 2 for bit 1; each lane sends two values per round.
__device__ __forceinline__ floatx4 quad_transpose(floatx4 x) {
  const int i = threadIdx.x & 3;
  const bool odd = i & 1, hi = i & 2;
  {
    const float r0 = dpp<0xB1>(odd ? x[0] : x[1]);   // quad_perm [1,0,3,2]
    const float r1 = dpp<0xB1>(odd ? x[2] : x[3]);
    x[0] = odd ? r0 : x[0];
    x[1] = odd ? x[1] : r0;
    x[2] = odd ? r1 : x[2];
    x[3] = odd ? x[3] : r1;
  }
  {
    const float r0 = dpp<0x4E>(hi ? x[0] : x[2]);    // quad_perm [2,3,0,1]
    const float r1 = dpp<0x4E>(hi ? x[1] : x[3]);
    x[0] = hi ? r0 : x[0];
    x[1] = hi ? r1 : x[1];
    x[2] = hi ? x[2] : r0;
    x[3] = hi ? x[3] : r1;
  }
  return x;
}

// Largest |x| over the 8 values of two accumulator tiles held by one lane, as
// an fp32 bit pattern (float maxima of absolute values fold into v_max3_f32
// with operand modifiers: one instruction per two values; a NaN is skipped).
__device__ __forceinline__ uint32_t lane_absmax_bits(const floatx4& a, const floatx4& b) {
  float m = fmaxf(fmaxf(fabsf(a[0]), fabsf(a[1])), fabsf(a[2]));
  m = fmaxf(fmaxf(m, fabsf(a[3])), fabsf(b[0]));
  m = fmaxf(fmaxf(m, fabsf(b[1])), fabsf(b[2]));
  return __float_as_uint(fmaxf(m, fabsf(b[3])));
}

// Log-cosh residual r = c tanh(x / c) (c < 0: no bound, r = x; c = 0: r = 0).
__device__ __forceinline__ float resid_tanh(float x, float c) {
  if (c < 0.f) return x;
  if (c == 0.f) return 0.f;
  return c * tanhf(x / c);
}

__device__ __forceinline__ uint32_t cvt_pk_f16(float a, float b) {
  return __builtin_bit_cast(uint32_t, f16x2{to_f16(a), to_f16(b)});
}

// Packs two adjacent 16 x 16 accumulator tiles (a0: columns 0..15, a1:
// columns 16..31 of a 16-row strip), each value times `scale` and rounded to
// fp16, into one 16-byte piece per lane holding 8 consecutive columns of one
// row: on return `row` (0..15) and `col` (0, 8, 16 or 24) say where the piece
// goes.  Three DPP exchanges (lanes c^1 and c^2 inside quads, then c^4 inside
// rows) turn a lane's 4 rows x 1 column of both tiles into 1 row x 8 columns.
__device__ __forceinline__ uint4 pack_strip_f16(const floatx4& a0, const floatx4& a1, float scale,
                                                int& row, int& col) {
  typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
  const int lane = threadIdx.x & 63, c = lane & 15, q = lane >> 4, g = c >> 2;
  const bool odd = c & 1, upper = c & 2, hi4 = g & 1;
  // v_perm byte selectors over {recv:keep}: even lanes (keep, recv), odd (recv, keep)
  const uint32_t selA = odd ? 0x01000504u : 0x05040100u;
  const uint32_t selB = odd ? 0x03020706u : 0x07060302u;
  u32x2 out[2];
#pragma unroll
  for (int jt = 0; jt < 2; ++jt) {
    const floatx4& a = jt ? a1 : a0;
    const uint32_t p01 = cvt_pk_f16(a[0] * scale, a[1] * scale);
    const uint32_t p23 = cvt_pk_f16(a[2] * scale, a[3] * scale);
    // round 1, lanes c and c^1: even lanes end with rows 0, 1 and odd
    // lanes with rows 2, 3, each as a column pair
    const uint32_t keep = odd ? p23 : p01;
    const uint32_t recv = dpp_u32<0xB1>(odd ? p01 : p23);
    const uint32_t x = __builtin_amdgcn_perm(recv, keep, selA);
    const uint32_t y = __builtin_amdgcn_perm(recv, keep, selB);
    // round 2, lanes c and c^2: each lane ends with one row, 4 columns
    const uint32_t recv2 = dpp_u32<0x4E>(upper ? x : y);
    out[jt] = upper ? u32x2{recv2, y} : u32x2{x, recv2};
  }
  // round 3, lanes c and c^4 (column groups g, g^1): the lower lane keeps its
  // tile-0 columns and takes its partner's, the upper lane the same for tile
  // 1 (row_shl:4 / row_shr:4 stay inside the 16-lane row)
  const u32x2 snd = hi4 ? out[0] : out[1];
  const uint32_t fromR0 = dpp_u32<0x104>(snd.x), fromR1 = dpp_u32<0x104>(snd.y);   // lane c + 4
  const uint32_t fromL0 = dpp_u32<0x114>(snd.x), fromL1 = dpp_u32<0x114>(snd.y);   // lane c - 4
  row = 4 * q + (((c & 1) << 1) | ((c >> 1) & 1));
  col = hi4 ? 16 + 4 * (g - 1) : 4 * g;
  return hi4 ? uint4{fromL0, fromL1, out[1].x, out[1].y} : uint4{out[0].x, out[0].y, fromR0, fromR1};
}

// Saves one 32-column block of a state held in MFMA accumulators: tile
// acc[it][jt] holds rows row0 + 16 it + acc_row(r) and columns
// 16 jt + acc_col().  Each 16-row x 32-column tile is divided by one power of
// two (pow2_scale_exp of the tile's largest magnitude) and stored as fp16
// row-major (row stride ld); the scale goes to sc[(row0 / 16 + it) * sc_ld].
// fp16 keeps 11 significant bits for every value within 2^-28 of the tile's
// largest, so one scale per tile loses nothing a per-row scale would keep
// for states whose rows span fewer than ~28 binades.  Each tile leaves in one
// 16-byte store per lane (pack_strip_f16; a wave writes 16 rows x 64 B).
// Largest magnitude of each 16-row x 32-column tile of such a state block
// (wave-uniform fp32 bits): mt[it] for the tile of rows row0 + 16 it.
template <int IT>
__device__ __forceinline__ void state_tile_absmax(const floatx4 (&acc)[IT][2], uint32_t (&mt)[IT]) {
#pragma unroll
  for (int it = 0; it < IT; ++it) mt[it] = wave_absmax_bits(lane_absmax_bits(acc[it][0], acc[it][1]));
}

// save_state_f16 with the tile maxima already known (state_tile_absmax of the
// same values).
template <int IT>
__device__ __forceinline__ void save_state_f16_max(const floatx4 (&acc)[IT][2], const uint32_t (&mt)[IT],
                                                   f16* dst, int64_t ld, float* sc, int64_t sc_ld,
                                                   int row0) {
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int e = pow2_scale_exp(mt[it]);
    int row, col;
    const uint4 v = pack_strip_f16(acc[it][0], acc[it][1], exp2_int(-e), row, col);
    *reinterpret_cast<uint4*>(dst + (int64_t)(row0 + 16 * it + row) * ld + col) = v;
    // every lane stores the (wave-uniform) scale to the same address: a
    // store under a lane condition becomes a branch, after which the
    // compiler can no longer count the wave's outstanding memory operations
    // and drains them all at its next wait
    sc[(int64_t)(row0 / 16 + it) * sc_ld] = exp2_int(e);
  }
}

template <int IT>
__device__ __forceinline__ void save_state_f16(const floatx4 (&acc)[IT][2], f16* dst, int64_t ld,
                                               float* sc, int64_t sc_ld, int row0) {
  uint32_t mt[IT];
  state_tile_absmax<IT>(acc, mt);
  save_state_f16_max<IT>(acc, mt, dst, ld, sc, sc_ld, row0);
}

// Scheduling hint for the enclosing basic block: alternate one LDS read, two
// MFMAs and VALU_PER vector instructions, NMFMA / 2 times.
template <int NMFMA, int VALU_PER>
__device__ __forceinline__ void interleave_mfma_valu() {
#pragma unroll
  for (int i = 0; i < NMFMA / 2; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);        // DS read
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);        // MFMA
    __builtin_amdgcn_sched_group_barrier(0x002, VALU_PER, 0); // VALU
  }
}

// fp32 counterpart of save_state_f16 (no scales): dst[row * ld + col].
template <int IT, int JT>
__device__ __forceinline__ void save_state_f32(const floatx4 (&acc)[IT][JT], float* dst, int64_t ld,
                                               int row0) {
#pragma unroll
  for (int it = 0; it < IT; ++it)
#pragma unroll
    for (int jt = 0; jt < JT; ++jt)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        dst[(int64_t)(row0 + 16 * it + acc_row(r)) * ld + 16 * jt + acc_col()] = acc[it][jt][r];
}

// Stores the 4 accumulator rows of this lane, column-major into LDS as a
// transposed tile: dst[col * ld + row]  (4 consecutive elements).
template <typename T>
__device__ __forceinline__ void store_acc_t(T* dst, int ld, floatx4 v) {
  T* p = dst + acc_col() * ld + acc_row(0);
  if constexpr (sizeof(T) == 2) {   // one 8-byte store (p is 8-byte aligned)
    typedef T T4 __attribute__((ext_vector_type(4)));
    T4 w;
#pragma unroll
    for (int r = 0; r < 4; ++r) w[r] = from_f<T>(v[r]);
    *reinterpret_cast<T4*>(p) = w;
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r) p[r] = from_f<T>(v[r]);
  }
}

// Stores the 4 accumulator rows of this lane transposed into a tile: element
// (row, col) of the accumulator tile goes to tile row r0 + col, column
// c0 + row (4 consecutive elements, one 8- or 16-byte store).
// r0 a multiple of 16, c0 a multiple of 16 elements.
template <class TL>
__device__ __forceinline__ void store_acc_tile(void* base, int r0, int c0, floatx4 v) {
  typedef typename std::remove_pointer<decltype(TL::ptr(nullptr, 0, 0))>::type T;
  T* p = reinterpret_cast<T*>(reinterpret_cast<char*>(base) +
                              TL::off_split(r0, acc_col(), acc_row(0) * (int)sizeof(T), c0 * (int)sizeof(T)));
  typedef T T4 __attribute__((ext_vector_type(4)));
  T4 w;
#pragma unroll
  for (int r = 0; r < 4; ++r) w[r] = from_f<T>(v[r]);
  *reinterpret_cast<T4*>(p) = w;
}

// Inverse of store_acc_tile: the accumulator-layout values of tile rows
// r0 + column, columns c0 + row (one 8- or 16-byte read).
template <class TL>
__device__ __forceinline__ floatx4 load_acc_tile(const void* base, int r0, int c0) {
  typedef typename std::remove_pointer<decltype(TL::ptr(nullptr, 0, 0))>::type T;
  typedef T T4 __attribute__((ext_vector_type(4)));
  const T4 w = *reinterpret_cast<const T4*>(reinterpret_cast<const char*>(base) +
                                            TL::off_split(r0, acc_col(), acc_row(0) * (int)sizeof(T), c0 * (int)sizeof(T)));
  floatx4 v;
#pragma unroll
  for (int r = 0; r < 4; ++r) v[r] = to_f<T>(w[r]);
  return v;
}

// Stores the 4 accumulator rows of this lane into LDS row-major: dst[row * ld + col].
template <typename T>
__device__ __forceinline__ void store_acc(T* dst, int ld, floatx4 v) {
  T* p = dst + acc_row(0) * ld + acc_col();
#pragma unroll
  for (int r = 0; r < 4; ++r) p[r * ld] = from_f<T>(v[r]);
}

// ---------------------------------------------------------------------------
// Sequences and chunks.  Either B dense sequences of length T (dense_T >= 0)
// or a device table built from cu_seqlens.
// ---------------------------------------------------------------------------
struct SeqInfo {     // one per sequence, in the device table
  int64_t start;
  int32_t len;
  int32_t chunk0;    // global index of the sequence's first chunk
};

struct ChunkInfo {   // one per chunk, in the device table
  int64_t tok;       // first token
  int32_t len;       // tokens in the chunk (1..64)
  int32_t seq;
};

struct SeqTable {
  int64_t dense_T;          // >= 0: dense layout with this T; < 0: use tables
  int32_t nseq;             // number of sequences
  int32_t dense_nch;        // chunks per dense sequence
  const SeqInfo* seqs;      // [nseq]            (varlen)
  const ChunkInfo* chunks;  // [max_chunks]      (varlen)
  const int32_t* nchunks;   // total chunks      (varlen)
  const int32_t* order;     // [nseq] sequences, longest first (varlen)
};

__device__ __forceinline__ SeqInfo seq_info(const SeqTable& t, int n) {
  if (t.dense_T >= 0) return SeqInfo{(int64_t)n * t.dense_T, (int32_t)t.dense_T, n * t.dense_nch};
  return t.seqs[n];
}

__device__ __forceinline__ int seq_order(const SeqTable& t, int i) {
  return t.dense_T >= 0 ? i : t.order[i];
}

// Returns false if c is past the last chunk.
__device__ __forceinline__ bool chunk_info(const SeqTable& t, int c, ChunkInfo& out) {
  if (t.dense_T >= 0) {
    if (t.dense_nch == 0) return false;
    const int n = c / t.dense_nch, j = c % t.dense_nch;
    if (n >= t.nseq) return false;
    const int64_t tok = (int64_t)n * t.dense_T + (int64_t)j * kChunk;
    const int64_t rem = t.dense_T - (int64_t)j * kChunk;
    out = ChunkInfo{tok, (int32_t)(rem < kChunk ? rem : kChunk), n};
    return true;
  }
  if (c >= *t.nchunks) return false;
  out = t.chunks[c];
  return true;
}

// Decay logarithm with the documented floor 2^-126 on the decay.
__device__ __forceinline__ float log_decay(float a) { return __logf(fmaxf(a, 1.17549435e-38f)); }

// Gate activations of the pre-activation inputs (Mamba-2 decay, sigmoid
// write strengths): softplus(z) = log(1 + e^z), sigmoid(z) = 1 / (1 + e^-z).
__device__ __forceinline__ float softplus_f(float z) {
  return z > 20.f ? z : log1pf(__expf(z));
}
__device__ __forceinline__ float sigmoid_f(float z) { return 1.f / (1.f + __expf(-z)); }

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ float wave_inclusive_scan(float x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  return x;
}

// Gate block of one (chunk, head), as written by the prep kernel:
//   [0..63] g  : inclusive cumulative log-decay of S inside the chunk
//   [64..]  h  : same for R
//   [128..] beta, [192..] gamma  (0 on padding rows)
constexpr int kGateBlock = 4 * kChunk;

// Matrices of one (chunk, head), as written by the prep kernel, each 64 x 64
// (row = query token t, column = key token s) and lower block-triangular in
// 16 x 16 blocks, stored packed (tri_off):
enum : int {
  kMatTS = 0,   // T^S = (I + A^S)^{-1}                     (RDN only)
  kMatMG = 1,   // e^{g_{t-1} - g_s} (k_t . k_s)       s < t
  kMatMP = 2,   // e^{g_t - g_s}     (q_t . k_s)       s < t
  kMatTR = 3,   // T^R = (I + A^R)^{-1}                     (RDN only)
  kMatMR = 4,   // e^{h_t - h_s}     (q_t . k_s)       s <= t
  kNumMats = 5
};

}  // namespace rla
