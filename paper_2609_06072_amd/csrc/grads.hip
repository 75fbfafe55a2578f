// Reductions of the backward over the rows of the permutation and over the
// ranks (Sec. 3.1.2 / 3.4: a shared adapter collects every routed pair of its
// group):
//   dB_q[n][r] = sum_u G_u[n] Hs_u[r]          (G_u = sum_{j in slots(u)} w_j dY[t*k+j])
//   dA_q[r][c] = sum_u dH_u[r] x_u[c]
//   dx[t][c]  += sum_K dHdense[t][K] A^T[c][K mod R]   (shared input only)
//
// grad_w_kernel  -- one item = (key, chunk of <= 1024 rows, block of 128
//   gradient columns, dB or dA).  Items are enumerated from the device-side
//   segment offsets, so a skewed key is split over several blocks.  The
//   chunk's row metadata goes to LDS first; then 128-row stages of the large
//   operand (G or x, 16-byte loads issued one stage ahead into registers) are
//   written transposed into LDS and multiplied on the matrix cores against the
//   small operand (Hs or dH, stored per key as [r][u]).  A key of one chunk
//   writes its gradient directly; otherwise every chunk writes a partial.
// grad_reduce_kernel -- sums the partials of a (key, column block) in chunk
//   order (deterministic) and writes the gradient.
// dx_gemm_kernel -- dense GEMM dx += dHdense A on 128x128 output tiles, the
//   tile staged through LDS for a coalesced read-modify-write of dx.
#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

constexpr int kColBlk = 128;     // gradient columns per item
constexpr int kSplitRows = 1024; // rows per item (split-K chunk)

// Item table of the weight-gradient pass: key q has ns_q = max(1, ceil(U_q /
// kSplitRows)) chunks times nb column blocks.  istart[q] = first item of q.
__device__ inline void build_item_table(const int32_t* offsets, int n_keys, int nb, int* seg,
                                        int* istart, int* scan_lds) {
  const int t = threadIdx.x;
  for (int i = t; i <= n_keys; i += kThreads) seg[i] = offsets[i];
  __syncthreads();
  int items = 0;
  if (t < n_keys) {
    const int cnt = seg[t + 1] - seg[t];
    items = max(1, (cnt + kSplitRows - 1) / kSplitRows) * nb;
  }
  int total;
  const int ex = block_exclusive_scan(items, scan_lds, &total);
  if (t < n_keys) istart[t] = ex;
  if (t == 0) istart[n_keys] = total;
  __syncthreads();
}

// Writes one accumulator fragment of an item's gradient block: element v of
// lane (g, c16) of column block cbi of wave w and rank block rb.
__device__ inline void store_grad(const GradArgs& a, bool isB, int q, int col0, int w, int cbi,
                                  int rb, int lane, f32x4 val) {
  const int c16 = lane & 15, g = lane >> 4;
  const int r_q = a.keys.rank[q], roff = a.keys.roff[q];
  if (isB) {  // D[n][r]
    const int r = 16 * rb + c16;
    if (r >= r_q) return;
    float* dst = a.dB + (size_t)a.d_out * roff;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int n = col0 + 32 * w + 16 * cbi + 4 * g + v;
      if (n < a.d_out) dst[(size_t)n * r_q + r] = val[v];
    }
  } else {    // D[r][c]
    const int c = col0 + 32 * w + 16 * cbi + c16;
    if (c >= a.d_in) return;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = 16 * rb + 4 * g + v;
      if (r < r_q) a.dA[(size_t)(roff + r) * a.d_in + c] = val[v];
    }
  }
}

// PER consecutive elements at p (one 16-byte load, always in bounds of the
// workspace) with the ones from index nvalid on set to zero.
template <typename T>
__device__ inline typename Tr<T>::frag load_masked(const T* p, int nvalid) {
  typename Tr<T>::frag f = Tr<T>::load(p);
#pragma unroll
  for (int e = 0; e < Tr<T>::PER; ++e)
    if (e >= nvalid) f[e] = (T)0.f;
  return f;
}

// Transpose of a PER x PER block held as PER row fragments: out[e] holds
// element e of every row.
template <typename T>
__device__ inline void transpose_block(const typename Tr<T>::frag (&in)[Tr<T>::PER],
                                       typename Tr<T>::frag (&out)[Tr<T>::PER]);

template <>
__device__ inline void transpose_block<float>(const f32x4 (&in)[4], f32x4 (&out)[4]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = f32x4{in[0][e], in[1][e], in[2][e], in[3][e]};
}

template <>
__device__ inline void transpose_block<__bf16>(const bf16x8 (&in)[8], bf16x8 (&out)[8]) {
  // word m of row r holds columns 2m (low half) and 2m+1 (high half); word m2
  // of column e holds rows 2m2 (low half) and 2m2+1 (high half)
  u32x4 w[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) w[r] = __builtin_bit_cast(u32x4, in[r]);
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    u32x4 ev, od;
#pragma unroll
    for (int m2 = 0; m2 < 4; ++m2) {
      const uint32_t a = w[2 * m2][m], b = w[2 * m2 + 1][m];
      ev[m2] = (a & 0xffffu) | (b << 16);
      od[m2] = (a >> 16) | (b & 0xffff0000u);
    }
    out[2 * m] = __builtin_bit_cast(bf16x8, ev);
    out[2 * m + 1] = __builtin_bit_cast(bf16x8, od);
  }
}

// Stage geometry of the weight-gradient kernel.
template <typename T>
struct GradGeo {
  static constexpr int PER = Tr<T>::PER, KB = Tr<T>::KB;
  static constexpr int NKB = 4;                      // K-blocks per stage
  static constexpr int RPS = NKB * KB;               // rows per stage (128 bf16, 64 f32)
  static constexpr int NI = RPS / PER;               // row groups of PER rows per stage
  static constexpr int NJ = kColBlk / PER;           // 16-byte column pieces per row
  static constexpr int NBLK = NI * NJ / kThreads;    // PER x PER blocks per thread (1 bf16, 2 f32)
  static constexpr int TI = NI / 8;                  // 8 x 8 block tiles along the rows
  static constexpr int SLD = RPS + PER;              // LDS stride of a transposed column (elements)
  static constexpr int MPT = kSplitRows / kThreads;
  static_assert(NBLK >= 1 && NI % 8 == 0, "stage shape");
};

template <typename T>
struct GradSmem {
  int seg[kMaxKeys + 1];
  int istart[kMaxKeys + 1];
  __attribute__((aligned(16))) T S[kColBlk * GradGeo<T>::SLD];
  // per row of the chunk: source row of the first slot (pair for dB, x row
  // for dA); dB only: pair of the second slot (the first again if none, bit 31
  // set when there are more) and the weights of the two slots
  int m0[kSplitRows];
  int m1[kSplitRows];
  float mw0[kSplitRows];
  float mw1[kSplitRows];
};

// One item: rows r0 .. r0+nrows of key q against gradient columns col0 ..
// col0+128 of dB_q (ISB) or dA_q.  TWO: rows may serve several slots.
template <typename T, int RB, bool ISB, bool TWO>
__device__ __forceinline__ void grad_item(const GradArgs& a, GradSmem<T>& sm, int item, int q, int s,
                                          int cb, const int (&bi)[GradGeo<T>::NBLK],
                                          const int (&bj)[GradGeo<T>::NBLK]) {
  using G = GradGeo<T>;
  using F = typename Tr<T>::frag;
  constexpr int PER = G::PER, KB = G::KB, NKB = G::NKB, RPS = G::RPS, NBLK = G::NBLK;
  constexpr int SLD = G::SLD, MPT = G::MPT;
  constexpr bool PF = RB <= 2;  // small-operand fragments prefetched a stage ahead
  constexpr int NKP = PF ? NKB : 1;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int c16 = lane & 15, g = lane >> 4;
  const int k = a.k;
  const int lo = sm.seg[q], hi = sm.seg[q + 1];
  const int ns = max(1, (hi - lo + kSplitRows - 1) / kSplitRows);
  const int r0 = lo + s * kSplitRows;
  const int nrows = max(0, min(hi, r0 + kSplitRows) - r0);
  const int ncol = ISB ? a.d_out : a.d_in;
  const int col0 = cb * kColBlk;
  const int r_q = a.keys.rank[q], roff = a.keys.roff[q];
  const int nrb = (r_q + 15) >> 4;
  const T* small = static_cast<const T*>(ISB ? a.Ht : a.dHt);
  const T* src = static_cast<const T*>(ISB ? a.dy : a.x);
  const T* DY = static_cast<const T*>(a.dy);
  const int lds_src = ISB ? a.d_out : a.d_in;
  const long hcol0 = (long)(r0 - lo);   // column of the chunk's first row in Ht/dHt
  const long hmax = a.ldh - PER;

  __syncthreads();  // the previous item's readers of the metadata and S are done
  if (nrows > 0) {
    int tv[MPT];
    uint32_t sv[MPT];
#pragma unroll
    for (int i = 0; i < MPT; ++i) {
      const int u = r0 + min(tid + i * kThreads, nrows - 1);
      tv[i] = a.row_token[u];
      sv[i] = a.row_slots[u];
    }
    int p0[MPT], p1[MPT];
#pragma unroll
    for (int i = 0; i < MPT; ++i) {
      const uint32_t sl = sv[i] | (sv[i] == 0u ? 1u : 0u);  // rows always serve a slot
      const uint32_t rest = sl & (sl - 1u);
      p0[i] = tv[i] * k + __builtin_ctz(sl);
      p1[i] = tv[i] * k + __builtin_ctz(rest ? rest : sl);
      sm.m0[tid + i * kThreads] = ISB ? p0[i] : (a.per_pair ? p0[i] : tv[i]);
      if (ISB) sm.m1[tid + i * kThreads] = p1[i] | ((rest & (rest - 1u)) ? (int)0x80000000 : 0);
    }
    if (ISB) {
      if (a.pair_w) {
        float w0[MPT], w1[MPT];
#pragma unroll
        for (int i = 0; i < MPT; ++i) {
          w0[i] = a.pair_w[p0[i]];
          w1[i] = a.pair_w[p1[i]];
        }
#pragma unroll
        for (int i = 0; i < MPT; ++i) {
          sm.mw0[tid + i * kThreads] = w0[i];
          sm.mw1[tid + i * kThreads] = w1[i];
        }
      } else {
#pragma unroll
        for (int i = 0; i < MPT; ++i) {
          sm.mw0[tid + i * kThreads] = 1.f;
          sm.mw1[tid + i * kThreads] = 1.f;
        }
      }
    }
  }
  __syncthreads();

  f32x4 acc[2][RB];
#pragma unroll
  for (int cbi = 0; cbi < 2; ++cbi)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc[cbi][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nst = (nrows + RPS - 1) / RPS;
  F v[NBLK][PER];
  F v2[TWO ? NBLK : 1][PER];
  F tf[NKP][RB];
  auto load_small = [&](int st, int kb, F* dst) {
    const int ul = st * RPS + kb * KB + PER * g;
    const long hc = min(hcol0 + ul, hmax);   // a clamped fragment is fully masked
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      if (rb < nrb) {
        // rank rows past r_q repeat row r_q - 1; nothing is stored for them
        const int rr = min(16 * rb + c16, r_q - 1);
        dst[rb] = load_masked<T>(small + (size_t)(roff + rr) * a.ldh + hc, nrows - ul);
      }
    }
  };
  auto load_stage = [&](int st) {
#pragma unroll
    for (int x = 0; x < NBLK; ++x) {
      const int cc = min(col0 + PER * bj[x], ncol - PER);
#pragma unroll
      for (int r = 0; r < PER; ++r) {
        const int row = min(st * RPS + PER * bi[x] + r, nrows - 1);
        v[x][r] = Tr<T>::load(src + (size_t)sm.m0[row] * lds_src + cc);
      }
      if (TWO) {
#pragma unroll
        for (int r = 0; r < PER; ++r) {
          const int row = min(st * RPS + PER * bi[x] + r, nrows - 1);
          v2[TWO ? x : 0][r] = Tr<T>::load(DY + (size_t)(sm.m1[row] & 0x7fffffff) * a.d_out + cc);
        }
      }
    }
    if (PF) {
#pragma unroll
      for (int kb = 0; kb < NKP; ++kb) load_small(st, kb, tf[kb]);
    }
  };
  auto write_stage = [&](int st) {
#pragma unroll
    for (int x = 0; x < NBLK; ++x) {
      const bool cok = col0 + PER * bj[x] < ncol;
      if (ISB) {  // G rows: weighted sum of the row's slots, rounded to T
#pragma unroll
        for (int r = 0; r < PER; ++r) {
          const int row = st * RPS + PER * bi[x] + r;
          const int rowc = min(row, nrows - 1);
          float f[PER];
          Tr<T>::to_f32(v[x][r], f);
          const float w0 = sm.mw0[rowc];
#pragma unroll
          for (int e = 0; e < PER; ++e) f[e] *= w0;
          if (TWO) {
            const int p1 = sm.m1[rowc];
            const float w1 = (p1 & 0x7fffffff) != sm.m0[rowc] ? sm.mw1[rowc] : 0.f;
            float f2[PER];
            Tr<T>::to_f32(v2[TWO ? x : 0][r], f2);
#pragma unroll
            for (int e = 0; e < PER; ++e) f[e] += w1 * f2[e];
            if (p1 < 0 && row < nrows) {  // third and further slots (rare)
              const int u = r0 + row;
              const int tok = a.row_token[u];
              uint32_t mm = a.row_slots[u];
              mm &= mm - 1u;
              mm &= mm - 1u;
              const int cc = min(col0 + PER * bj[x], ncol - PER);
              for (; mm; mm &= mm - 1u) {
                const int p2 = tok * k + __builtin_ctz(mm);
                const float w = a.pair_w ? a.pair_w[p2] : 1.f;
                float f3[PER];
                Tr<T>::to_f32(Tr<T>::load(DY + (size_t)p2 * a.d_out + cc), f3);
#pragma unroll
                for (int e = 0; e < PER; ++e) f[e] += w * f3[e];
              }
            }
          }
          v[x][r] = Tr<T>::from_f32(f);
        }
      }
      // rows past the chunk and columns past the matrix are zero
#pragma unroll
      for (int r = 0; r < PER; ++r)
        if (!(cok && st * RPS + PER * bi[x] + r < nrows)) v[x][r] = Tr<T>::zero();
      F o[PER];
      transpose_block<T>(v[x], o);
#pragma unroll
      for (int e = 0; e < PER; ++e)
        *reinterpret_cast<F*>(&sm.S[(PER * bj[x] + e) * SLD + PER * bi[x]]) = o[e];
    }
  };
  if (nst > 0) load_stage(0);
  for (int st = 0; st < nst; ++st) {
    write_stage(st);
    F cur[NKP][RB];
    if (PF) {
#pragma unroll
      for (int kb = 0; kb < NKP; ++kb)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) cur[kb][rb] = tf[kb][rb];
    }
    __syncthreads();
    if (st + 1 < nst) load_stage(st + 1);
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
      const int ul = st * RPS + kb * KB;  // first row of the K-block (chunk-local)
      if (ul >= nrows) break;
      F tl[RB];
      if (!PF) load_small(st, kb, tl);
#pragma unroll
      for (int cbi = 0; cbi < 2; ++cbi) {
        const F sf = *reinterpret_cast<const F*>(&sm.S[(32 * wave + 16 * cbi + c16) * SLD + kb * KB + PER * g]);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          if (rb < nrb) {
            const F t = PF ? cur[PF ? kb : 0][rb] : tl[rb];
            if (ISB) acc[cbi][rb] = Tr<T>::mma(sf, t, acc[cbi][rb]);   // D[n][r]
            else acc[cbi][rb] = Tr<T>::mma(t, sf, acc[cbi][rb]);       // D[r][c]
          }
        }
      }
    }
    __syncthreads();  // the next stage overwrites S
  }

  if (ns == 1) {
#pragma unroll
    for (int cbi = 0; cbi < 2; ++cbi)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        if (rb < nrb) store_grad(a, ISB, q, col0, wave, cbi, rb, lane, acc[cbi][rb]);
  } else {
    f32x4* part = reinterpret_cast<f32x4*>(a.part) + (size_t)item * (4 * 2 * RB * 64);
#pragma unroll
    for (int cbi = 0; cbi < 2; ++cbi)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) part[((wave * 2 + cbi) * RB + rb) * 64 + lane] = acc[cbi][rb];
  }
}

template <typename T, int RB, bool MULTI>
__global__ __launch_bounds__(kThreads) void grad_w_kernel(GradArgs a) {
  using G = GradGeo<T>;
  __shared__ GradSmem<T> sm;
  const int n_keys = a.keys.n_keys;
  const int nb = a.nbB + a.nbA;
  build_item_table(a.offsets, n_keys, nb, sm.seg, sm.istart, reinterpret_cast<int*>(sm.S));
  const int total = sm.istart[n_keys];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // Staging: thread block x covers rows PER*bi .. +PER and columns PER*bj ..
  // +PER of a stage.  Eight consecutive lanes take eight consecutive row
  // groups of one column piece, so a load instruction reads whole 128-byte
  // lines and the transposed 16-byte LDS writes of eight lanes are contiguous.
  int bi[G::NBLK], bj[G::NBLK];
#pragma unroll
  for (int x = 0; x < G::NBLK; ++x) {
    const int tile = wave + 4 * x;
    bi[x] = (tile % G::TI) * 8 + (lane & 7);
    bj[x] = (tile / G::TI) * 8 + (lane >> 3);
  }
  for (int item = blockIdx.x; item < total; item += gridDim.x) {
    const int q = upper_index(sm.istart, n_keys, item);
    const int local = item - sm.istart[q];
    const int s = local / nb, rem = local % nb;
    if (rem < a.nbB) grad_item<T, RB, true, MULTI>(a, sm, item, q, s, rem, bi, bj);
    else grad_item<T, RB, false, false>(a, sm, item, q, s, rem - a.nbB, bi, bj);
  }
}

// One block per (key, column block, dB|dA): sums the chunk partials in order.
template <int RB>
__global__ __launch_bounds__(kThreads) void grad_reduce_kernel(GradArgs a) {
  __shared__ int seg[kMaxKeys + 1];
  __shared__ int istart[kMaxKeys + 1];
  __shared__ int scan[kThreads];
  const int n_keys = a.keys.n_keys;
  const int nb = a.nbB + a.nbA;
  build_item_table(a.offsets, n_keys, nb, seg, istart, scan);
  const int q = blockIdx.x / nb, rem = blockIdx.x % nb;
  const int ns = max(1, (seg[q + 1] - seg[q] + kSplitRows - 1) / kSplitRows);
  if (ns == 1) return;  // written directly by grad_w_kernel
  const bool isB = rem < a.nbB;
  const int cb = isB ? rem : rem - a.nbB;
  const int nrb = (a.keys.rank[q] + 15) >> 4;
  const f32x4* part = reinterpret_cast<const f32x4*>(a.part);
  constexpr int PER_ITEM = 4 * 2 * RB * 64;
  for (int e = threadIdx.x; e < PER_ITEM; e += kThreads) {
    const int lane = e & 63;
    const int rb = (e >> 6) % RB;
    const int wc = (e >> 6) / RB;  // wave * 2 + cbi
    if (rb >= nrb) continue;
    f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < ns; ++c) s += part[(size_t)(istart[q] + c * nb + rem) * PER_ITEM + e];
    store_grad(a, isB, q, cb * kColBlk, wc >> 1, wc & 1, rb, lane, s);
  }
}

// dx[t][c] += sum_K dHf[t][K] At[c][K mod R] on a 128 x 128 tile; wave
// (wy, wx) owns tokens 64*wy.. and columns 64*wx.. as 4 x 4 MFMA blocks.
constexpr int kDxTile = 128;

template <typename T>
__global__ __launch_bounds__(kThreads) void dx_gemm_kernel(DxArgs a) {
  using F = typename Tr<T>::frag;
  constexpr int PER = Tr<T>::PER, KB = Tr<T>::KB;
  constexpr int CST = kDxTile + 16 / (int)sizeof(T);
  __shared__ __attribute__((aligned(16))) T Cs[kDxTile * CST];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int c16 = lane & 15, g = lane >> 4;
  const int wy = wave >> 1, wx = wave & 1;
  const int ntc = (a.d_in + kDxTile - 1) / kDxTile;
  const int t0 = (blockIdx.x / ntc) * kDxTile, c0 = (blockIdx.x % ntc) * kDxTile;
  const T* At = static_cast<const T*>(a.At);
  const T* Hf = static_cast<const T*>(a.dHf);
  T* DX = static_cast<T*>(a.dx);
  const int R = a.R, KR = a.KR;
  const bool vec = (R % PER) == 0;
  const T* arow[4];
  const T* hrow[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    arow[b] = At + (size_t)min(c0 + 64 * wx + 16 * b + c16, a.d_in - 1) * R;
    hrow[b] = Hf + (size_t)min(t0 + 64 * wy + 16 * b + c16, a.T - 1) * KR;
  }
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  struct Stage {
    F w[4], h[4];
  };
  // full K-blocks: 16-byte loads (a fragment never straddles a multiple of R
  // when R % PER == 0)
  auto load_fast = [&](int kk, Stage& st) {
    const int kof = kk + PER * g;
    const int km = kof % R;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      st.w[b] = Tr<T>::load(arow[b] + km);
      st.h[b] = Tr<T>::load(hrow[b] + kof);
    }
  };
  auto load_slow = [&](int kk, Stage& st) {
    const int kof = kk + PER * g;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      st.w[b] = Tr<T>::zero();
      st.h[b] = load_frag<T>(hrow[b] + kof, KR - kof, false);
#pragma unroll
      for (int e = 0; e < PER; ++e)
        if (kof + e < KR) st.w[b][e] = arow[b][(kof + e) % R];
    }
  };
  auto mma = [&](const Stage& st) {
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) acc[cb][tb] = Tr<T>::mma(st.w[cb], st.h[tb], acc[cb][tb]);  // D[c][t]
  };
  const int nkb = (KR + KB - 1) / KB;
  const int nfull = vec ? KR / KB : 0;
  {
    Stage SA, SB;
    if (nfull > 0) load_fast(0, SA);
    int i = 0;
    for (; i + 1 < nfull; i += 2) {
      load_fast((i + 1) * KB, SB);
      mma(SA);
      if (i + 2 < nfull) load_fast((i + 2) * KB, SA);
      mma(SB);
    }
    if (i < nfull) mma(SA);
    for (i = nfull; i < nkb; ++i) {
      load_slow(i * KB, SA);
      mma(SA);
    }
  }
  // tile -> LDS as [t][c], then a coalesced read-modify-write of dx
#pragma unroll
  for (int cb = 0; cb < 4; ++cb)
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      T* cp = &Cs[(64 * wy + 16 * tb + c16) * CST + 64 * wx + 16 * cb + 4 * g];
#pragma unroll
      for (int v = 0; v < 4; ++v) cp[v] = (T)acc[cb][tb][v];
    }
  __syncthreads();
  constexpr int PPR = kDxTile / PER;
  constexpr int NP = kDxTile * PPR / kThreads;
  F old[NP];
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int it = tid + i * kThreads;
    const int tr = it / PPR, pc = (it % PPR) * PER;
    const int t = min(t0 + tr, a.T - 1), c = min(c0 + pc, a.d_in - PER);
    old[i] = Tr<T>::load(DX + (size_t)t * a.d_in + c);
  }
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int it = tid + i * kThreads;
    const int tr = it / PPR, pc = (it % PPR) * PER;
    if (t0 + tr < a.T && c0 + pc < a.d_in) {
      float o[PER], cv[PER];
      Tr<T>::to_f32(old[i], o);
      Tr<T>::to_f32(*reinterpret_cast<const F*>(&Cs[tr * CST + pc]), cv);
#pragma unroll
      for (int e = 0; e < PER; ++e) o[e] += cv[e];
      Tr<T>::store(DX + (size_t)(t0 + tr) * a.d_in + c0 + pc, Tr<T>::from_f32(o));
    }
  }
}

template <typename T, int RB>
hipError_t launch_grads_rb(const GradArgs& g, long P, hipStream_t stream) {
  const int nb = g.nbB + g.nbA;
  const long items = ((P + kSplitRows - 1) / kSplitRows + g.keys.n_keys) * nb;
  const long cap = 8L * device_cu_count();
  const int grid = (int)(items < cap ? items : cap);
  if (grid > 0) {
    if (g.multi) grad_w_kernel<T, RB, true><<<grid, kThreads, 0, stream>>>(g);
    else grad_w_kernel<T, RB, false><<<grid, kThreads, 0, stream>>>(g);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (P > kSplitRows) grad_reduce_kernel<RB><<<g.keys.n_keys * nb, kThreads, 0, stream>>>(g);
  return hipGetLastError();
}

}  // namespace

size_t grads_part_bytes(int T, int k, int d_in, int d_out, int n_keys, int r_max) {
  const long P = (long)T * k;
  const long nb = (d_out + kColBlk - 1) / kColBlk + (d_in + kColBlk - 1) / kColBlk;
  const long items = ((P + kSplitRows - 1) / kSplitRows + n_keys) * nb;
  return (size_t)items * 4 * 2 * rank_blocks(r_max) * 64 * sizeof(f32x4);
}

hipError_t launch_grads(int dtype, GradArgs g, int r_max, long P, hipStream_t stream) {
  g.nbB = (g.d_out + kColBlk - 1) / kColBlk;
  g.nbA = (g.d_in + kColBlk - 1) / kColBlk;
  const int rb = rank_blocks(r_max);
  if (dtype == ACE_BF16) {
    if (rb == 2) return launch_grads_rb<__bf16, 2>(g, P, stream);
    if (rb == 4) return launch_grads_rb<__bf16, 4>(g, P, stream);
    if (rb == 8) return launch_grads_rb<__bf16, 8>(g, P, stream);
    return launch_grads_rb<__bf16, 16>(g, P, stream);
  }
  if (rb == 2) return launch_grads_rb<float, 2>(g, P, stream);
  if (rb == 4) return launch_grads_rb<float, 4>(g, P, stream);
  if (rb == 8) return launch_grads_rb<float, 8>(g, P, stream);
  return launch_grads_rb<float, 16>(g, P, stream);
}

hipError_t launch_dx_gemm(int dtype, const DxArgs& d, hipStream_t stream) {
  const int tiles = ((d.T + kDxTile - 1) / kDxTile) * ((d.d_in + kDxTile - 1) / kDxTile);
  if (tiles <= 0) return hipSuccess;
  if (dtype == ACE_BF16) dx_gemm_kernel<__bf16><<<tiles, kThreads, 0, stream>>>(d);
  else dx_gemm_kernel<float><<<tiles, kThreads, 0, stream>>>(d);
  return hipGetLastError();
}

}  // namespace ace
