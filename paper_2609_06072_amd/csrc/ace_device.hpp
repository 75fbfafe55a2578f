// Device-side building blocks shared by the libace kernels (gfx950, wave64).
//
// Matrix-core fragments.  Every contraction in the library is issued as
// 16x16 output blocks on the CDNA4 MFMA units:
//   bf16: v_mfma_f32_16x16x32_bf16 -- one 16-byte fragment (8 bf16) per lane
//   fp32: v_mfma_f32_16x16x4f32    -- one 16-byte fragment (4 floats) per lane,
//                                     consumed by four MFMAs (element i in step i)
// Lane l = 16*g + c (g = l >> 4 in 0..3, c = l & 15) supplies row/column c of
// its operand; its fragment covers the PER contraction indices PER*g .. PER*g+PER-1
// of a K-block of KB = 4*PER (32 for bf16, 16 for fp32).  The accumulator
// block holds D[4*g + v][c] in element v.  Since a contraction is a sum, any
// assignment of contraction indices to (g, element) works as long as both
// operands use the same one; the kernels use that freedom to feed an
// accumulator straight back in as an operand (see Tr<T>::kmap_acc).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ace {

constexpr int kMaxKeys = 256;
constexpr int kMaxRank = 256;
constexpr int kMaxK = 32;
constexpr int kThreads = 256;  // every kernel runs 4 waves of 64

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

// Per-key ranks and rank offsets, passed by value in the kernel arguments so
// that no host-to-device copy precedes a launch.
struct KeyTable {
  int32_t n_keys;
  int32_t R;
  int32_t rank[kMaxKeys];
  int32_t roff[kMaxKeys + 1];
};

template <typename T>
struct Tr;

template <>
struct Tr<float> {
  using frag = f32x4;
  static constexpr int PER = 4;
  static constexpr int KB = 16;
  __device__ static inline f32x4 mma(frag a, frag b, f32x4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], c, 0, 0, 0);
    return c;
  }
  __device__ static inline frag zero() { return frag{0.f, 0.f, 0.f, 0.f}; }
  __device__ static inline frag load(const float* p) {
    return *reinterpret_cast<const f32x4*>(p);
  }
  using v4 = f32x4;
  __device__ static inline v4 load4raw(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
  // 4 consecutive elements -> 4 floats (p 16-byte aligned)
  __device__ static inline f32x4 load4(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
  __device__ static inline void store4(float* p, f32x4 v) { *reinterpret_cast<f32x4*>(p) = v; }
  // Fragment of the rank-K-block m built from accumulator blocks: block m's
  // element v of lane group g is index 16*m + 4*g + v, which is exactly the
  // natural fragment layout of a K-block of 16.
  static constexpr int ACC_PER_FRAG = 1;
  __device__ static inline frag from_acc(const f32x4* acc, int m, float s) {
    return acc[m] * s;
  }
  __device__ static inline frag from_f32(const float* v) { return frag{v[0], v[1], v[2], v[3]}; }
  __device__ static inline float to_f32(float v) { return v; }
  __device__ static inline float from_float(float v) { return v; }
};

template <>
struct Tr<__bf16> {
  using frag = bf16x8;
  static constexpr int PER = 8;
  static constexpr int KB = 32;
  __device__ static inline f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static inline frag zero() {
    u32x4 z = {0u, 0u, 0u, 0u};
    return __builtin_bit_cast(frag, z);
  }
  __device__ static inline frag load(const __bf16* p) {
    return __builtin_bit_cast(frag, *reinterpret_cast<const u32x4*>(p));
  }
  using v4 = bf16x4;
  __device__ static inline v4 load4raw(const __bf16* p) {
    return __builtin_bit_cast(bf16x4, *reinterpret_cast<const u32x2*>(p));
  }
  __device__ static inline f32x4 load4(const __bf16* p) {
    bf16x4 v = __builtin_bit_cast(bf16x4, *reinterpret_cast<const u32x2*>(p));
    return f32x4{(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
  }
  __device__ static inline void store4(__bf16* p, f32x4 v) {
    bf16x4 b = {(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
    *reinterpret_cast<u32x2*>(p) = __builtin_bit_cast(u32x2, b);
  }
  // A rank K-block of 32 covers accumulator blocks 2m and 2m+1: element i of
  // lane group g is rank index 32*m + 16*(i/4) + 4*g + (i%4).
  static constexpr int ACC_PER_FRAG = 2;
  __device__ static inline frag from_acc(const f32x4* acc, int m, float s) {
    const f32x4 a = acc[2 * m] * s, b = acc[2 * m + 1] * s;
    return frag{(__bf16)a[0], (__bf16)a[1], (__bf16)a[2], (__bf16)a[3],
                (__bf16)b[0], (__bf16)b[1], (__bf16)b[2], (__bf16)b[3]};
  }
  __device__ static inline frag from_f32(const float* v) {
    return frag{(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3],
                (__bf16)v[4], (__bf16)v[5], (__bf16)v[6], (__bf16)v[7]};
  }
  __device__ static inline float to_f32(__bf16 v) { return (float)v; }
  __device__ static inline __bf16 from_float(float v) { return (__bf16)v; }
};

// Rank index held by element i of lane group g in rank K-block m when the
// fragment was built from accumulators (Tr<T>::from_acc).
template <typename T>
__device__ inline int kmap_acc(int m, int g, int i) {
  if constexpr (Tr<T>::PER == 4) {
    return 16 * m + 4 * g + i;
  } else {
    return 32 * m + 16 * (i >> 2) + 4 * g + (i & 3);
  }
}

// Loads the operand fragment of one weight row (base = the row's first
// element, valid columns [0, ncols)) for rank K-block m in the
// accumulator-derived order (kmap_acc).  Columns >= ncols read as zero.
// `aligned4` says the row starts on a multiple of 4 elements.
template <typename T>
__device__ inline typename Tr<T>::frag load_acc_order(const T* base, int ncols, int m, int g,
                                                      bool row_ok, bool aligned4) {
  typename Tr<T>::frag f = Tr<T>::zero();
  if (!row_ok) return f;
  constexpr int CH = Tr<T>::PER / 4;  // 4-element chunks per fragment
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int r0 = kmap_acc<T>(m, g, 4 * c);
    if (aligned4 && r0 + 3 < ncols) {
      const typename Tr<T>::v4 v = Tr<T>::load4raw(base + r0);
#pragma unroll
      for (int i = 0; i < 4; ++i) f[4 * c + i] = v[i];
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = r0 + i;
        f[4 * c + i] = r < ncols ? base[r] : (T)0.f;
      }
    }
  }
  return f;
}

// Exclusive block-wide scan of one int per thread (kThreads threads).
__device__ inline int block_exclusive_scan(int v, int* lds /* kThreads ints */, int* total) {
  const int t = threadIdx.x;
  lds[t] = v;
  __syncthreads();
#pragma unroll
  for (int off = 1; off < kThreads; off <<= 1) {
    const int add = t >= off ? lds[t - off] : 0;
    __syncthreads();
    lds[t] += add;
    __syncthreads();
  }
  const int incl = lds[t];
  *total = lds[kThreads - 1];
  __syncthreads();
  return incl - v;
}

// Tile table of a persistent launch over per-key row segments: tiles of BM
// rows, key-major.  tstart[q] = first tile of key q, tstart[n_keys] = total.
// seg[q] = offsets[q] (first row of key q), seg[n_keys] = U.
__device__ inline void build_tile_table(const int32_t* offsets, int n_keys, int BM, int* seg,
                                        int* tstart, int* scan_lds) {
  const int t = threadIdx.x;
  int tiles = 0;
  for (int i = t; i <= n_keys; i += kThreads) seg[i] = offsets[i];
  __syncthreads();
  if (t < n_keys) tiles = (seg[t + 1] - seg[t] + BM - 1) / BM;
  int total;
  const int ex = block_exclusive_scan(tiles, scan_lds, &total);
  if (t < n_keys) tstart[t] = ex;
  if (t == 0) tstart[n_keys] = total;
  __syncthreads();
}

// Key q with tstart[q] <= tile < tstart[q+1] (binary search; uniform).
__device__ inline int find_key(const int* tstart, int n_keys, int tile) {
  int lo = 0, hi = n_keys;  // invariant: tstart[lo] <= tile < tstart[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (tstart[mid] <= tile) lo = mid; else hi = mid;
  }
  return lo;
}

}  // namespace ace
