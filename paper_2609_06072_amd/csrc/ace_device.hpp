// Device-side building blocks shared by the libace kernels (gfx950, wave64).
//
// Matrix-core fragments.  Every contraction in the library is issued as
// 16x16 output blocks on the CDNA4 MFMA units:
//   bf16: v_mfma_f32_16x16x32_bf16 -- one 16-byte fragment (8 bf16) per lane
//   fp32: v_mfma_f32_16x16x4f32    -- one 16-byte fragment (4 floats) per lane,
//                                     consumed by four MFMAs (element i in step i)
// Lane l = 16*g + c (g = l >> 4 in 0..3, c = l & 15) supplies row/column c of
// its operand; its fragment holds contraction indices PER*g .. PER*g+PER-1 of a
// K-block of KB = 4*PER (32 for bf16, 16 for fp32).  The accumulator block
// holds D[4*g + v][c] in element v.
//
// Rank permutation.  The shrink H^T = A_q X^T puts rank indices on the rows
// of D.  Because the rows of the A operand may be any permutation of A_q's
// rows, the shrink loads row rank_of_row(rb, i) into operand row i of rank
// block rb; then the accumulators of rank blocks (APF*m .. APF*m+APF-1) of
// lane group g hold exactly rank indices KB*m + PER*g .. + PER-1: a natural
// K-block fragment, so H feeds the expand MFMA without any data movement and
// the expand's weight fragments are plain 16-byte loads.
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
  static constexpr int APF = 1;  // accumulator blocks per rank K-block
  __device__ static inline f32x4 mma(frag a, frag b, f32x4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], c, 0, 0, 0);
    return c;
  }
  __device__ static inline frag zero() { return frag{0.f, 0.f, 0.f, 0.f}; }
  __device__ static inline frag load(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
  __device__ static inline void store(float* p, frag v) { *reinterpret_cast<f32x4*>(p) = v; }
  // streaming (non-temporal) variants for data touched once per call
  __device__ static inline frag load_nt(const float* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
  }
  __device__ static inline void store_nt(float* p, frag v) {
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(p));
  }
  __device__ static inline f32x4 lo4(frag f) { return f; }
  __device__ static inline void to_f32(frag f, float* v) {
    v[0] = f[0]; v[1] = f[1]; v[2] = f[2]; v[3] = f[3];
  }
  __device__ static inline frag from_f32(const float* v) { return frag{v[0], v[1], v[2], v[3]}; }
  // fragment of rank K-block m from the accumulators (times s)
  __device__ static inline frag from_acc(const f32x4* acc, int m, float s) { return acc[m] * s; }
};

template <>
struct Tr<__bf16> {
  using frag = bf16x8;
  static constexpr int PER = 8;
  static constexpr int KB = 32;
  static constexpr int APF = 2;
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
  __device__ static inline void store(__bf16* p, frag v) {
    *reinterpret_cast<u32x4*>(p) = __builtin_bit_cast(u32x4, v);
  }
  // streaming (non-temporal) variants for data touched once per call
  __device__ static inline frag load_nt(const __bf16* p) {
    return __builtin_bit_cast(frag, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p)));
  }
  __device__ static inline void store_nt(__bf16* p, frag v) {
    __builtin_nontemporal_store(__builtin_bit_cast(u32x4, v), reinterpret_cast<u32x4*>(p));
  }
  __device__ static inline void to_f32(frag f, float* v) {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = (float)f[i];
  }
  __device__ static inline frag from_f32(const float* v) {
    return frag{(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3],
                (__bf16)v[4], (__bf16)v[5], (__bf16)v[6], (__bf16)v[7]};
  }
  __device__ static inline frag from_acc(const f32x4* acc, int m, float s) {
    const f32x4 a = acc[2 * m] * s, b = acc[2 * m + 1] * s;
    return frag{(__bf16)a[0], (__bf16)a[1], (__bf16)a[2], (__bf16)a[3],
                (__bf16)b[0], (__bf16)b[1], (__bf16)b[2], (__bf16)b[3]};
  }
};

// Rank index loaded into operand row i (0..15) of rank block rb by the
// shrink, so that accumulator element v of lane group g in rank block rb
// holds rank rank_of_row<T>(rb, 4*g + v) and from_acc yields natural order.
template <typename T>
__device__ __host__ inline int rank_of_row(int rb, int i) {
  constexpr int APF = Tr<T>::APF, PER = Tr<T>::PER, KB = Tr<T>::KB;
  return KB * (rb / APF) + PER * (i >> 2) + 4 * (rb % APF) + (i & 3);
}

// PER consecutive elements p[0 .. PER) of which the first nvalid are read
// (the rest are zero); a full fragment uses one 16-byte load when `vec`.
template <typename T>
__device__ inline typename Tr<T>::frag load_frag(const T* p, int nvalid, bool vec) {
  constexpr int PER = Tr<T>::PER;
  if (nvalid >= PER && vec) return Tr<T>::load(p);
  typename Tr<T>::frag f = Tr<T>::zero();
  if (nvalid <= 0) return f;
#pragma unroll
  for (int e = 0; e < PER; ++e)
    if (e < nvalid) f[e] = p[e];
  return f;
}

// Exclusive block-wide scan of one int per thread (kThreads threads): a
// shuffle scan inside each wave, then the wave totals through LDS (two
// barriers).  lds needs kThreads / 64 ints and is free again on return.
__device__ inline int block_exclusive_scan(int v, int* lds, int* total) {
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int o = __shfl_up(incl, off, 64);
    if (lane >= off) incl += o;
  }
  if (lane == 63) lds[w] = incl;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kThreads / 64; ++i) {
    const int s = lds[i];
    if (i < w) base += s;
    tot += s;
  }
  *total = tot;
  __syncthreads();
  return base + incl - v;
}

// Tile table of a launch over per-key row segments: tiles of BM rows,
// key-major.  tstart[q] = first tile of key q, tstart[n_keys] = total.
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

// XCD-aware tile table.  Blocks are dispatched to the XCDs round-robin, so
// block b runs on XCD b % kXcds.  Within a key the rows are sorted by token,
// so the x-th eighth of a key's tiles covers about the x-th eighth of the
// tokens; bucket x collects that eighth of every key and is served by the
// blocks with b % kXcds == x.  Rows that share a token (the same token's rows
// in other groups) then meet in the same XCD's L2.
// bstart[q] = first index of key q's tiles inside the bucket, bfirst[q] = the
// key-local index of that tile, bstart[n_keys] = the bucket's tile count.
constexpr int kXcds = 8;
// With seg_map, the segments are seg_map[offsets[q]] .. seg_map[offsets[q+1]].
__device__ inline void build_bucket_table(const int32_t* offsets, const int32_t* seg_map,
                                          int n_keys, int BM, int bucket, int* seg, int* bstart,
                                          int* bfirst, int* scan_lds) {
  const int t = threadIdx.x;
  for (int i = t; i <= n_keys; i += kThreads) seg[i] = seg_map ? seg_map[offsets[i]] : offsets[i];
  __syncthreads();
  int cnt = 0;
  if (t < n_keys) {
    const int nq = (seg[t + 1] - seg[t] + BM - 1) / BM;
    const int j0 = (bucket * nq + kXcds - 1) / kXcds;
    const int j1 = ((bucket + 1) * nq + kXcds - 1) / kXcds;
    bfirst[t] = j0;
    cnt = j1 - j0;
  }
  int total;
  const int ex = block_exclusive_scan(cnt, scan_lds, &total);
  if (t < n_keys) bstart[t] = ex;
  if (t == 0) bstart[n_keys] = total;
  __syncthreads();
}

// Key q and row range of tile `tile` when every key's rows (segment
// offsets[q] .. offsets[q+1]) are cut into tiles of BM rows, key-major.  Every
// wave computes it on its own: lane l owns keys KPL*l .. KPL*l + KPL - 1, a
// wave-level scan of the per-lane tile counts finds the owning lane, which
// broadcasts the result (no LDS, no barrier).  Returns false (in every lane)
// when the tile is past the last one.
__device__ inline bool locate_tile(const int32_t* offsets, int n_keys, int BM, int tile, int* q_out,
                                   int* u0_out, int* uend_out) {
  constexpr int KPL = kMaxKeys / 64;
  const int lane = threadIdx.x & 63;
  int off[KPL + 1], tl[KPL];
#pragma unroll
  for (int i = 0; i <= KPL; ++i) off[i] = offsets[min(lane * KPL + i, n_keys)];
  int cnt = 0;
#pragma unroll
  for (int i = 0; i < KPL; ++i) {
    tl[i] = (off[i + 1] - off[i] + BM - 1) / BM;  // zero past n_keys (clamped offsets)
    cnt += tl[i];
  }
  int incl = cnt;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(incl, o, 64);
    if (lane >= o) incl += v;
  }
  const int excl = incl - cnt;
  const unsigned long long hit = __ballot(tile >= excl && tile < incl);
  if (hit == 0ull) return false;
  const int owner = __builtin_ctzll(hit);
  int t = tile - excl, q = 0, u0 = 0, ue = 0;
  bool found = false;
#pragma unroll
  for (int i = 0; i < KPL; ++i) {
    if (!found && t < tl[i]) {
      q = lane * KPL + i;
      u0 = off[i] + t * BM;
      ue = off[i + 1];
      found = true;
    }
    if (!found) t -= tl[i];
  }
  *q_out = __shfl(q, owner, 64);
  *u0_out = __shfl(u0, owner, 64);
  *uend_out = __shfl(ue, owner, 64);
  return true;
}

// Largest q in [0, n) with arr[q] <= x, for a non-decreasing arr (uniform).
__device__ inline int upper_index(const int* arr, int n, int x) {
  int lo = 0, hi = n;  // invariant: arr[lo] <= x < arr[hi] (arr[n] treated as +inf)
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (arr[mid] <= x) lo = mid; else hi = mid;
  }
  return lo;
}

// ---- direct global -> LDS copies (gfx950 global_load_lds_dwordx4)

typedef __attribute__((address_space(3))) void lds_void;

__device__ inline uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const lds_void*)p;
}

// 16-byte copy global -> LDS: lane l's bytes land at lds_base + 16 * l
// (lds_base wave-uniform).  Issued as inline assembly so that the compiler does
// not treat every later LDS read as dependent on it; completion is awaited
// explicitly with wait_vmcnt before the barrier that publishes the data.
__device__ inline void dma16(const void* g, uint32_t lds_base) {
  asm volatile("global_load_lds_dwordx4 %1, off" ::"{m0}"(lds_base), "v"(g) : "memory");
}
// The same copy with the non-temporal policy (data read once per call).
__device__ inline void dma16_nt(const void* g, uint32_t lds_base) {
  asm volatile("global_load_lds_dwordx4 %1, off nt" ::"{m0}"(lds_base), "v"(g) : "memory");
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// s_waitcnt vmcnt(n) for a wave-uniform 0 <= n <= N
template <int N>
__device__ inline void wait_vmcnt_upto(int n) {
  if constexpr (N > 0) {
    if (n >= N) {
      wait_vmcnt<N>();
      return;
    }
    wait_vmcnt_upto<N - 1>(n);
  } else {
    (void)n;
    wait_vmcnt<0>();
  }
}

}  // namespace ace
