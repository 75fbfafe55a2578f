// Expand and scatter-add (the second GEMM of Sec. 3.1.3 and the reuse of
// Sec. 3.5): for every row u of key q and every slot j it serves,
//   out[t*k + j][n] += w_tj * sum_r W_q[n][r] * H[u][r]
// where H is the row-major output of the contraction (already scaled by
// alpha / r_q and zero beyond r_q).  W_q = B_q (forward: out = y) or
// W_q = A_q^T (backward with per-pair input: out = dx, w = 1).
//
// One block per work item: (tile of BM rows of one key) x (two chunks of 128
// output columns).  The item is located from the device-side segment
// offsets (a wave-level scan, no host sync); blocks past the last item exit
// at once.  Per item:
//   - wave 0 lists the tile's (row, slot) pairs in LDS;
//   - the threads issue the loads of the pair weights, of H and of W (cache
//     hits), then those of the item's y pieces in both chunks (16-byte
//     pieces, 16 consecutive threads per 256-byte row piece, kSlots per
//     thread and chunk), which are in flight during the matrix work (loads
//     return in order, so the small operands arrive first);
//   - each wave multiplies its two 16-column blocks of W against the four
//     16-row blocks of H on the matrix cores and writes C of the first chunk
//     to LDS in fp32; the threads add w * C to their y pieces of that chunk
//     and store them; then the same for the second chunk (H stays in
//     registers), so y is rounded once per call (items with more pieces take
//     further batches of loads per chunk).
// Two chunks per block halve the per-item set-up (tile lookup, pair list, H)
// per byte of y and double the y bytes in flight per block.
// The y pieces held across the matrix work cost registers and save the
// latency of a round trip to the memory per item.  y is read and written
// once per call, with non-temporal loads and stores, so that it does not
// displace from the caches what the next launches read.
#include <type_traits>

#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

constexpr int kBM = 64;                 // rows per tile
constexpr int kBM48 = 48;               // rows per tile, bf16 rows serving several slots, two chunks
constexpr int kChunk = 128;             // output columns per chunk
constexpr int kBPW = kChunk / 16 / 4;   // 16-column blocks per wave
constexpr int kWideOut = 4096;          // outputs at least this wide take two chunks per item

// NC chunks per item (1 or 2), BM rows per tile (a multiple of 16, <= 64)
template <typename T, int RB, int NC, int BM>
__global__ __launch_bounds__(kThreads, (std::is_same<T, __bf16>::value && RB <= 4) ? 4 : 1) void expand_kernel(ExpandArgs a) {
  using F = typename Tr<T>::frag;
  constexpr int PER = Tr<T>::PER, KB = Tr<T>::KB, APF = Tr<T>::APF;
  constexpr int NM = RB / APF;
  constexpr int kSlots = NC == 2 ? 4 : 6;   // y pieces per thread and chunk in flight
  constexpr int PPR = kChunk / PER;     // 16-byte pieces per pair and chunk
  constexpr int CST = kChunk + 4;       // LDS row stride of C (fp32)
  // bf16 at 64 ranks or more: the tile's H rows are loaded once into LDS and
  // every wave reads its fragments there (rows 16 bytes longer than the ranks,
  // so the 16 rows of a fragment read spread over the banks); H is read into
  // registers before C is written, so both share one buffer
  constexpr bool HLDS = std::is_same<T, __bf16>::value && RB >= 4;
  constexpr int HST = HLDS ? NM * KB + 8 : 8;   // LDS row stride of H (elements)
  constexpr int NJB = BM / 16;          // 16-row blocks per tile
  static_assert(BM % 16 == 0 && BM <= 64, "tile rows");
  static_assert(HST * sizeof(T) <= CST * sizeof(float), "H staging exceeds the C buffer");
  // the second chunk's W fragments are loaded with the first chunk's while
  // they are few; at higher ranks after the first chunk is done
  constexpr bool WB_EARLY = RB <= 2;
  __shared__ __attribute__((aligned(16))) float Cs[BM * CST];
  T* const Hs = reinterpret_cast<T*>(Cs);
  __shared__ uint16_t plist[BM * kMaxK];  // (row << 5) | slot
  __shared__ int toks[BM];
  __shared__ int npairs_s;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int c16 = lane & 15, g = lane >> 4;
  const int tile = blockIdx.x / a.nch;
  const int n0 = (blockIdx.x - tile * a.nch) * (NC * kChunk);
  int q, u0, u_end;
  if (!locate_tile(a.offsets, a.keys.n_keys, BM, tile, &q, &u0, &u_end)) return;  // block-uniform
  const T* H = static_cast<const T*>(a.H);
  const T* W = static_cast<const T*>(a.W);
  T* O = static_cast<T*>(a.out);
  const int k = a.k, n_out = a.n_out, R = a.keys.R;
  const int r_q = a.keys.rank[q], roff = a.keys.roff[q];
  const int nmb = (r_q + KB - 1) / KB;
  const bool has2 = NC == 2 && n0 + kChunk < n_out;   // block-uniform: a second chunk

  if (wave == 0) {
    const int u = u0 + lane;
    const int uc = min(u, u_end - 1);  // unconditional loads
    const int tok = a.row_token[uc];
    uint32_t sl = a.row_slots[uc];
    if (u >= u_end || lane >= BM) sl = 0u;
    if (lane < BM) toks[lane] = tok;
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
  __syncthreads();  // plist, toks published
  const int nitems = npairs_s * PPR;   // pieces per chunk
  if (nitems == 0) return;  // block-uniform (a row serves at least one slot)

  // Slot pf of the batch at base: piece j = base + tid + pf * kThreads of a
  // chunk (pieces past the item re-read the item's last piece, marked -1 in
  // po; the same j in both chunks is the same pair and C position).
  auto locate = [&](int base, int pf, int& po, int& co) {
    const int it = base + tid + pf * kThreads;
    const bool ok = it < nitems;
    const int itc = ok ? it : nitems - 1;
    const int ent = plist[itc / PPR];
    const int p = toks[ent >> 5] * k + (ent & 31);
    po = ok ? p : -1;
    co = (ent >> 5) * CST + (itc % PPR) * PER;
    return p;
  };
  // y piece of slot pf in the chunk at column c0 (pieces past n_out, or
  // marked, read y[0] and are not stored)
  auto y_at = [&](int base, int pf, int po, int c0) {
    const int c = c0 + ((base + tid + pf * kThreads) % PPR) * PER;
    return O + (po >= 0 && c < n_out ? (size_t)po * n_out + c : 0);
  };
  auto finish = [&](int base, int pf, int po, int co, float w, F yv, int c0) {
    const int c = c0 + ((base + tid + pf * kThreads) % PPR) * PER;
    if (po < 0 || c >= n_out) return;
    float o[PER];
    Tr<T>::to_f32(yv, o);
    const float* cp = &Cs[co];
#pragma unroll
    for (int e2 = 0; e2 < PER; e2 += 4) {
      const f32x4 cv = *reinterpret_cast<const f32x4*>(cp + e2);
#pragma unroll
      for (int v = 0; v < 4; ++v) o[e2 + v] += w * cv[v];
    }
    Tr<T>::store_nt(O + (size_t)po * n_out + c, Tr<T>::from_f32(o));
  };
  // later batches of one chunk (items with many pairs): loads then finish,
  // in the given slot arrays
  auto more_batches = [&](int c0, F (&yv)[kSlots], int (&po)[kSlots], int (&co)[kSlots],
                          float (&wv)[kSlots]) {
    for (int base = kSlots * kThreads; base < nitems; base += kSlots * kThreads) {
#pragma unroll
      for (int pf = 0; pf < kSlots; ++pf) {
        if (base + pf * kThreads < nitems) {  // block-uniform
          const int p = locate(base, pf, po[pf], co[pf]);
          yv[pf] = Tr<T>::load_nt(y_at(base, pf, po[pf], c0));
          wv[pf] = a.pair_w ? a.pair_w[p] : 1.f;
        }
      }
#pragma unroll
      for (int pf = 0; pf < kSlots; ++pf)
        if (base + pf * kThreads < nitems) finish(base, pf, po[pf], co[pf], wv[pf], yv[pf], c0);
    }
  };

  // First batch of both chunks.  Loads return in order, so the small
  // operands (pair weights, H, W: cache hits) are issued before the y pieces
  // (HBM): the matrix work then runs while the y pieces are in flight.  Every
  // load of this batch is unconditional, so that the waits for H and W count
  // exactly the y loads behind them.
  int po0[kSlots], co0[kSlots];
  float wv0[kSlots];
  {
    int pp[kSlots];
#pragma unroll
    for (int pf = 0; pf < kSlots; ++pf) pp[pf] = locate(0, pf, po0[pf], co0[pf]);
    if (a.pair_w) {  // block-uniform, before H and W
#pragma unroll
      for (int pf = 0; pf < kSlots; ++pf) wv0[pf] = a.pair_w[pp[pf]];
    } else {
#pragma unroll
      for (int pf = 0; pf < kSlots; ++pf) wv0[pf] = 1.f;
    }
  }
  constexpr int PPRH = NM * KB / PER;   // 16-byte pieces per H row
  constexpr int HN = HLDS ? (BM * PPRH + kThreads - 1) / kThreads : 1;
  F hv[HN];
  F hf[NJB][NM];
  if constexpr (HLDS) {
    // BM rows x NM*KB ranks in 16-byte pieces (rows past the segment re-read
    // the last row; pieces past the tile re-read its last piece and are not
    // stored)
#pragma unroll
    for (int i = 0; i < HN; ++i) {
      const int j = min(tid + i * kThreads, BM * PPRH - 1);
      const int u = min(u0 + j / PPRH, u_end - 1);
      hv[i] = Tr<T>::load(H + (size_t)u * a.rpad + (j % PPRH) * PER);
    }
  } else {
    // H fragments of the four row blocks (rows past the segment re-read the
    // last row; nothing is stored for them)
#pragma unroll
    for (int jb = 0; jb < NJB; ++jb) {
      const int u = min(u0 + 16 * jb + c16, u_end - 1);
      const T* hr = H + (size_t)u * a.rpad + PER * g;
#pragma unroll
      for (int m = 0; m < NM; ++m) hf[jb][m] = Tr<T>::load(hr + KB * m);
    }
  }
  // W fragments of this wave's column blocks of the chunk at c0 (rows past
  // n_out re-read the last row; rank columns past r_q meet zeros in H)
  const T* Wq = W + (size_t)a.w_key_mul * roff;
  const int ldw = a.w_stride_is_rank ? r_q : R;
  // 16-byte loads need aligned rows; clamping a fragment that starts past
  // r_q back to r_q - PER only keeps every valid rank in place when r_q is a
  // multiple of PER
  const bool vec = (ldw % PER) == 0 && ((size_t)a.w_key_mul * roff) % PER == 0 && (r_q % PER) == 0;
  auto load_w = [&](int c0, F (&wf)[kBPW][NM]) {
#pragma unroll
    for (int bi = 0; bi < kBPW; ++bi) {
      const int nrow = min(c0 + 16 * (wave * kBPW + bi) + c16, n_out - 1);
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
  };
  // C = H W^T of the chunk into LDS (fp32)
  auto c_tile = [&](const F (&wf)[kBPW][NM]) {
#pragma unroll
    for (int bi = 0; bi < kBPW; ++bi) {
      const int b = wave * kBPW + bi;
#pragma unroll
      for (int jb = 0; jb < NJB; ++jb) {
        f32x4 c = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < NM; ++m)
          if (m < nmb) c = Tr<T>::mma(wf[bi][m], hf[jb][m], c);  // C[u][c0+16b+4g+v]
        *reinterpret_cast<f32x4*>(&Cs[(16 * jb + c16) * CST + 16 * b + 4 * g]) = c;
      }
    }
  };
  F wf0[kBPW][NM], wf1[kBPW][NM];
  load_w(n0, wf0);
  if constexpr (NC == 2 && WB_EARLY) load_w(n0 + kChunk, wf1);
  F y0[kSlots], y1[kSlots];
#pragma unroll
  for (int pf = 0; pf < kSlots; ++pf) y0[pf] = Tr<T>::load_nt(y_at(0, pf, po0[pf], n0));
  if constexpr (NC == 2) {
#pragma unroll
    for (int pf = 0; pf < kSlots; ++pf) y1[pf] = Tr<T>::load_nt(y_at(0, pf, po0[pf], n0 + kChunk));
  }

  if constexpr (HLDS) {
#pragma unroll
    for (int i = 0; i < HN; ++i) {
      const int j = tid + i * kThreads;
      if (j < BM * PPRH) Tr<T>::store(&Hs[(j / PPRH) * HST + (j % PPRH) * PER], hv[i]);
    }
    __syncthreads();
#pragma unroll
    for (int jb = 0; jb < NJB; ++jb)
#pragma unroll
      for (int m = 0; m < NM; ++m) hf[jb][m] = Tr<T>::load(&Hs[(16 * jb + c16) * HST + KB * m + PER * g]);
    __syncthreads();  // every wave holds its H fragments; C reuses the buffer
  }
  c_tile(wf0);
  __syncthreads();  // C of the first chunk is published
#pragma unroll
  for (int pf = 0; pf < kSlots; ++pf) finish(0, pf, po0[pf], co0[pf], wv0[pf], y0[pf], n0);
  if constexpr (NC == 1) {
    more_batches(n0, y0, po0, co0, wv0);   // the first batch's slots are free
  } else {
    // the first batch's pair slots still serve the second chunk
    int po1[kSlots], co1[kSlots];
    float wv1[kSlots];
    more_batches(n0, y0, po1, co1, wv1);
    if (!has2) return;  // block-uniform
    if constexpr (!WB_EARLY) load_w(n0 + kChunk, wf1);
    __syncthreads();  // every wave is done with the first chunk's C
    c_tile(wf1);
    __syncthreads();  // C of the second chunk is published
#pragma unroll
    for (int pf = 0; pf < kSlots; ++pf) finish(0, pf, po0[pf], co0[pf], wv0[pf], y1[pf], n0 + kChunk);
    more_batches(n0 + kChunk, y1, po1, co1, wv1);
  }
}

template <typename T, int RB>
hipError_t launch_expand_rb(ExpandArgs a, long P, hipStream_t stream) {
  // two chunks per item at ranks up to 32 and for wide outputs; at higher
  // ranks with few chunks per tile the second chunk's W load, issued after
  // the first chunk is done, costs more than the shared set-up saves
  const int nc = (RB <= 2 || a.n_out >= kWideOut) ? 2 : 1;
  a.nch = (a.n_out + nc * kChunk - 1) / (nc * kChunk);   // items per tile
  // bf16 with two chunks: four y pieces per thread and chunk cover 64 pairs,
  // so where rows serve several slots, tiles of 48 rows keep most tiles within
  // one batch of loads (a second batch costs a round trip to the memory)
  const int bm = (std::is_same<T, __bf16>::value && a.multi_slot && nc == 2) ? kBM48 : kBM;
  // tiles are bounded by P / bm plus one ragged tile per key; U itself stays
  // on the device
  const long grid = P > 0 ? ((P + bm - 1) / bm + a.keys.n_keys) * a.nch : 0;
  if (grid > 0x7fffffffL) return hipErrorInvalidConfiguration;
  if (grid > 0) {
    if constexpr (std::is_same<T, __bf16>::value) {
      if (bm == kBM48) {
        expand_kernel<T, RB, 2, kBM48><<<(int)grid, kThreads, 0, stream>>>(a);
        return hipGetLastError();
      }
    }
    if (nc == 2) expand_kernel<T, RB, 2, kBM><<<(int)grid, kThreads, 0, stream>>>(a);
    else expand_kernel<T, RB, 1, kBM><<<(int)grid, kThreads, 0, stream>>>(a);
  }
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
