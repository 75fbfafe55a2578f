// Expand and scatter-add (the second GEMM of Sec. 3.1.3 and the reuse of
// Sec. 3.5): for every row u of key q and every slot j it serves,
//   out[t*k + j][n] += w_tj * sum_r W_q[n][r] * H[u][r]
// where H is the row-major output of the contraction (already scaled by
// alpha / r_q and zero beyond r_q).  W_q = B_q (forward: out = y) or
// W_q = A_q^T (backward with per-pair input: out = dx, w = 1).
//
// Work items are (tile of BM rows of one key) x (chunk of 128 output
// columns), enumerated from the device-side segment offsets; each block takes
// a contiguous range of items, so consecutive items usually share a tile and
// reuse its pair list and H fragments.  Per item:
//   - every thread issues its y loads for the item at once (16-byte pieces,
//     16 consecutive threads per 256-byte row piece), before any math;
//   - each wave multiplies its two 16-column blocks of W against the four
//     16-row blocks of H on the matrix cores and writes C to LDS (in the
//     output precision);
//   - the threads add w * C to their y pieces and store them.
// When the tile changes, wave 0 lists the new tile's (row, slot) pairs in LDS.
#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

constexpr int kBM = 64;                 // rows per tile
constexpr int kChunk = 128;             // output columns per item
constexpr int kPrefetch = 8;            // y pieces per thread issued up front
constexpr int kBPW = kChunk / 16 / 4;   // 16-column blocks per wave

template <typename T, int RB>
__global__ __launch_bounds__(kThreads) void expand_kernel(ExpandArgs a) {
  using F = typename Tr<T>::frag;
  constexpr int PER = Tr<T>::PER, KB = Tr<T>::KB, APF = Tr<T>::APF;
  constexpr int NM = RB / APF;
  constexpr int PPR = kChunk / PER;     // 16-byte pieces per pair per item
  constexpr int CST = kChunk + 16 / (int)sizeof(T);  // LDS row stride of C (elements)
  __shared__ int seg[kMaxKeys + 1];
  __shared__ int tstart[kMaxKeys + 1];
  __shared__ int scan[kThreads];
  __shared__ __attribute__((aligned(16))) T Cs[kBM * CST];
  __shared__ uint16_t plist[kBM * kMaxK];  // (row << 5) | slot
  __shared__ int toks[kBM];
  __shared__ int npairs_s;
  const int n_keys = a.keys.n_keys;
  build_tile_table(a.offsets, n_keys, kBM, seg, tstart, scan);
  const int n_items = tstart[n_keys] * a.nch;
  const int per_block = (n_items + gridDim.x - 1) / gridDim.x;
  const int i_begin = blockIdx.x * per_block;
  const int i_end = min(n_items, i_begin + per_block);
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int c16 = lane & 15, g = lane >> 4;
  const T* H = static_cast<const T*>(a.H);
  const T* W = static_cast<const T*>(a.W);
  T* O = static_cast<T*>(a.out);
  const int k = a.k, n_out = a.n_out, R = a.keys.R;

  int cur_tile = -1, q = 0, u0 = 0, u_end = 0, r_q = 1, roff = 0, nmb = 1, npairs = 0;
  F hf[4][NM];
  for (int item = i_begin; item < i_end; ++item) {
    const int tile = item / a.nch;
    const int n0 = (item % a.nch) * kChunk;
    if (tile != cur_tile) {  // block-uniform
      cur_tile = tile;
      q = upper_index(tstart, n_keys, tile);
      u0 = seg[q] + (tile - tstart[q]) * kBM;
      u_end = seg[q + 1];
      r_q = a.keys.rank[q];
      roff = a.keys.roff[q];
      nmb = (r_q + KB - 1) / KB;
      __syncthreads();  // readers of the previous tile's plist/toks are done
      if (wave == 0) {
        const int u = u0 + lane;
        const int uc = min(u, u_end - 1);  // unconditional loads
        const int tok = a.row_token[uc];
        uint32_t sl = a.row_slots[uc];
        if (u >= u_end) sl = 0u;
        toks[lane] = tok;
        const int cnt = __builtin_popcount(sl);
        int incl = cnt;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const int o = __shfl_up(incl, off, 64);
          if (lane >= off) incl += o;
        }
        int e = incl - cnt;
        for (uint32_t mm = sl; mm; mm &= mm - 1u) plist[e++] = (uint16_t)((lane << 5) | __builtin_ctz(mm));
        if (lane == 63) npairs_s = incl;
      }
      // H fragments of the four row blocks (rows past the segment re-read the
      // last row; nothing is stored for them)
#pragma unroll
      for (int jb = 0; jb < 4; ++jb) {
        const int u = min(u0 + 16 * jb + c16, u_end - 1);
        const T* hr = H + (size_t)u * a.rpad + PER * g;
#pragma unroll
        for (int m = 0; m < NM; ++m) hf[jb][m] = Tr<T>::load(hr + KB * m);
      }
      __syncthreads();
      npairs = npairs_s;
    }
    const int nitems = npairs * PPR;

    // y pieces of this thread, loaded before the math (clamped, unconditional)
    F yv[kPrefetch];
#pragma unroll
    for (int pf = 0; pf < kPrefetch; ++pf) {
      const int it = tid + pf * kThreads;
      const bool ok = it < nitems;
      const int e = ok ? it / PPR : 0;
      const int col = n0 + (it % PPR) * PER;
      const int ent = plist[e];
      const int p = toks[ent >> 5] * k + (ent & 31);
      const bool cok = ok && col < n_out;
      yv[pf] = Tr<T>::load(O + (cok ? (size_t)p * n_out + col : 0));
    }
    // W fragments of this wave's column blocks (rows past n_out re-read the
    // last row; rank columns past r_q meet zeros in H)
    const T* Wq = W + (size_t)a.w_key_mul * roff;
    const int ldw = a.w_stride_is_rank ? r_q : R;
    // 16-byte loads need aligned rows; clamping a fragment that starts past
    // r_q back to r_q - PER only keeps every valid rank in place when r_q is a
    // multiple of PER
    const bool vec = (ldw % PER) == 0 && ((size_t)a.w_key_mul * roff) % PER == 0 && (r_q % PER) == 0;
    F wf[kBPW][NM];
#pragma unroll
    for (int bi = 0; bi < kBPW; ++bi) {
      const int nrow = min(n0 + 16 * (wave * kBPW + bi) + c16, n_out - 1);
      const T* wr = Wq + (size_t)nrow * ldw;
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        const int r0 = KB * m + PER * g;
        if (vec) {
          wf[bi][m] = Tr<T>::load(wr + min(r0, r_q - PER));
        } else {
          wf[bi][m] = (m < nmb && r0 < r_q) ? load_frag<T>(wr + r0, r_q - r0, false) : Tr<T>::zero();
        }
      }
    }
    f32x4 c[kBPW][4];
#pragma unroll
    for (int bi = 0; bi < kBPW; ++bi)
#pragma unroll
      for (int jb = 0; jb < 4; ++jb) {
        c[bi][jb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < NM; ++m)
          if (m < nmb) c[bi][jb] = Tr<T>::mma(wf[bi][m], hf[jb][m], c[bi][jb]);  // C[u][n0+16b+4g+v]
      }
    __syncthreads();  // readers of the previous item's C are done
#pragma unroll
    for (int bi = 0; bi < kBPW; ++bi) {
      const int b = wave * kBPW + bi;
#pragma unroll
      for (int jb = 0; jb < 4; ++jb) {
        T* cp = &Cs[(16 * jb + c16) * CST + 16 * b + 4 * g];
#pragma unroll
        for (int v = 0; v < 4; ++v) cp[v] = (T)c[bi][jb][v];
      }
    }
    __syncthreads();

    for (int base = 0; base < nitems; base += kPrefetch * kThreads) {
#pragma unroll
      for (int pf = 0; pf < kPrefetch; ++pf) {
        const int it = base + tid + pf * kThreads;
        if (it < nitems) {
          const int e = it / PPR, pc = (it % PPR) * PER, col = n0 + pc;
          if (col < n_out) {
            const int ent = plist[e];
            const int row = ent >> 5;
            const int p = toks[row] * k + (ent & 31);
            const float w = a.pair_w ? a.pair_w[p] : 1.f;
            T* op = O + (size_t)p * n_out + col;
            const F old = base == 0 ? yv[pf] : Tr<T>::load(op);
            float o[PER], cv[PER];
            Tr<T>::to_f32(old, o);
            Tr<T>::to_f32(*reinterpret_cast<const F*>(&Cs[row * CST + pc]), cv);
#pragma unroll
            for (int e2 = 0; e2 < PER; ++e2) o[e2] += w * cv[e2];
            Tr<T>::store(op, Tr<T>::from_f32(o));
          }
        }
      }
    }
  }
}

template <typename T, int RB>
hipError_t launch_expand_rb(ExpandArgs a, long P, hipStream_t stream) {
  a.nch = (a.n_out + kChunk - 1) / kChunk;
  const long bound = P > 0 ? ((P + kBM - 1) / kBM + a.keys.n_keys) * a.nch : 0;
  const long cap = 8L * device_cu_count();
  const int grid = (int)(bound < cap ? bound : cap);
  if (grid > 0) expand_kernel<T, RB><<<grid, kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_expand(int dtype, const ExpandArgs& a, int r_max, long P, hipStream_t stream) {
  const int rb = rank_blocks(r_max);
  if (dtype == ACE_BF16) {
    if (rb == 2) return launch_expand_rb<__bf16, 2>(a, P, stream);
    if (rb == 4) return launch_expand_rb<__bf16, 4>(a, P, stream);
    if (rb == 8) return launch_expand_rb<__bf16, 8>(a, P, stream);
    return launch_expand_rb<__bf16, 16>(a, P, stream);
  }
  if (rb == 2) return launch_expand_rb<float, 2>(a, P, stream);
  if (rb == 4) return launch_expand_rb<float, 4>(a, P, stream);
  if (rb == 8) return launch_expand_rb<float, 8>(a, P, stream);
  return launch_expand_rb<float, 16>(a, P, stream);
}

}  // namespace ace
