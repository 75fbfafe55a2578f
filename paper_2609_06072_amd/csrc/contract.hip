// Rank contraction over the rows of the permutation: for every row u of key q
//   out[u][r] = s_q * sum_c W_q[r][c] * src_u[c],   r < r_q,  s_q = alpha / r_q
// with either
//   src_u = x[row_token[u]]            (shared input; Sec. 3.5: once per row,
//                                       i.e. once per (token, active group))
//   src_u = S[t*k + j]                 (the row's single pair: per-pair input of
//                                       the down projection, or dY)
//   src_u = S[plist[u]]                (u a pair position: dY of that pair)
// and W = A (the shrink h = A_q x of Sec. 3.1.3) or W = B^T (dH = B_q^T dY).
// With out_w, the result of a single-pair row is multiplied by the pair's
// weight.
//
// A block takes a tile of BM rows of one key.  The four waves split the
// contraction (wave w takes K-blocks w, w+4, ...), so each source row and each
// weight row is read once per tile, and the partial sums meet in LDS in a
// fixed order (deterministic).  Results go to any of three layouts:
//   row-major  [U][rpad]      operand of the expand kernel (zero beyond r_q)
//   per key    [R][ldh]       column u - offsets[q]: operand of the column pass
//   dense      [T*kslots][R]  per-token rows: operand of the dense dx GEMM
#include <type_traits>

#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

// Writes row u's result h (scaled, zero past r_q) to the requested outputs.
template <typename T, int RB>
__device__ inline void contract_store(const ContractArgs& a, int q, int lo, int u, f32x4 (&h)[RB]) {
  constexpr int KB = Tr<T>::KB, APF = Tr<T>::APF;
  const int k = a.k, R = a.keys.R;
  const int r_q = a.keys.rank[q], roff = a.keys.roff[q];
  const int nrb = ((r_q + KB - 1) / KB) * APF;
  const int g = (threadIdx.x & 63) >> 4;
  int tok = 0;
  uint32_t slots = 1u;
  if (a.src_mode != kSrcPairList) {
    tok = a.row_token[u];
    slots = a.row_slots[u];
  }
  if (a.out_w && a.pair_w) {  // single-pair rows: times the pair's weight
    const float w = a.pair_w[tok * k + (__builtin_ctz(slots | 0x80000000u) & 31)];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) h[rb] *= w;
  }
  if (a.out_row) {
    T* dst = static_cast<T*>(a.out_row) + (size_t)u * a.rpad;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int r0 = rank_of_row<T>(rb, 4 * g);  // 4 consecutive ranks
      if (r0 < a.rpad) {
#pragma unroll
        for (int v = 0; v < 4; ++v) dst[r0 + v] = (T)h[rb][v];
      }
    }
  }
  if (a.out_t && !a.out_t_pairs) {
    T* dst = static_cast<T*>(a.out_t);
    const long col = u - lo;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
      if (rb < nrb) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int r = rank_of_row<T>(rb, 4 * g + v);
          if (r < r_q) dst[(size_t)(roff + r) * a.ldh + col] = (T)h[rb][v];
        }
      }
  }
  if (a.out_t && a.out_t_pairs) {  // one column per pair served, times its weight
    T* dst = static_cast<T*>(a.out_t);
    long col = a.ppos ? (long)a.ppos[u] - a.ppos[lo] : (long)(u - lo);
    for (uint32_t mm = slots; mm; mm &= mm - 1u, ++col) {
      const float w = a.pair_w ? a.pair_w[tok * k + __builtin_ctz(mm)] : 1.f;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        if (rb < nrb) {
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int r = rank_of_row<T>(rb, 4 * g + v);
            if (r < r_q) dst[(size_t)(roff + r) * a.ldh + col] = (T)(h[rb][v] * w);
          }
        }
    }
  }
  if (a.out_dense) {
    const int j0 = __builtin_ctz(slots | 0x80000000u) & 31;
    const size_t drow = (size_t)tok * a.kslots + (a.kslots > 1 ? j0 : 0);
    T* dst = static_cast<T*>(a.out_dense) + drow * R + roff;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
      if (rb < nrb) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int r = rank_of_row<T>(rb, 4 * g + v);
          if (r < r_q) dst[r] = (T)h[rb][v];
        }
      }
  }
}

template <int RB>
struct CGeo {
  static constexpr int NRB = RB <= 4 ? 4 : (RB == 8 ? 2 : 1);
  static constexpr int UNROLL = RB <= 8 ? 2 : 1;
};

template <typename T, int RB>
__global__ __launch_bounds__(kThreads) void contract_kernel(ContractArgs a) {
  using F = typename Tr<T>::frag;
  constexpr int PER = Tr<T>::PER, KB = Tr<T>::KB, APF = Tr<T>::APF;
  constexpr int NRB = CGeo<RB>::NRB, U = CGeo<RB>::UNROLL;
  constexpr int BM = 16 * NRB;
  __shared__ int seg[kMaxKeys + 1];
  __shared__ int bstart[kMaxKeys + 1];
  __shared__ int bfirst[kMaxKeys];
  __shared__ int scan[kThreads];
  __shared__ f32x4 red[4][NRB][RB][64];
  const int n_keys = a.keys.n_keys;
  const int bucket = blockIdx.x % kXcds;
  build_bucket_table(a.offsets, a.src_mode == kSrcPairList ? a.ppos : nullptr, n_keys, BM, bucket,
                     seg, bstart, bfirst, scan);
  const int total = bstart[n_keys];
  const int stride = gridDim.x / kXcds;  // the grid is a multiple of kXcds
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c16 = lane & 15, g = lane >> 4;
  const T* S = static_cast<const T*>(a.src);
  const T* W = static_cast<const T*>(a.W);
  const int K = a.K, k = a.k;
  const int nks = (K + KB - 1) / KB, nks_full = K / KB;

  for (int idx = blockIdx.x / kXcds; idx < total; idx += stride) {
    const int q = upper_index(bstart, n_keys, idx);
    const int lo = seg[q];
    const int u0 = lo + (bfirst[q] + idx - bstart[q]) * BM;
    const int u_end = seg[q + 1];
    const int r_q = a.keys.rank[q], roff = a.keys.roff[q];
    const int nmb = (r_q + KB - 1) / KB;
    const int nrb = nmb * APF;  // rank blocks spanned by rank_of_row for r < r_q

    // Source rows.  Rows past the segment re-read the last row (never
    // stored); weight rows past r_q re-read row r_q - 1 (zeroed before any
    // store), so every load is unconditional and a wave keeps all of them in
    // flight.
    const T* srow[NRB];
    int sv[NRB];
    uint32_t slv[NRB];
#pragma unroll
    for (int ib = 0; ib < NRB; ++ib) {  // unconditional loads: one round trip
      const int uc = min(u0 + 16 * ib + c16, u_end - 1);
      if (a.src_mode == kSrcPairList) {
        sv[ib] = a.plist[uc];
        slv[ib] = 1u;
      } else {
        sv[ib] = a.row_token[uc];
        slv[ib] = a.row_slots[uc];
      }
    }
#pragma unroll
    for (int ib = 0; ib < NRB; ++ib) {
      const int j0 = __builtin_ctz(slv[ib] | 0x80000000u) & 31;
      const int sr = a.src_mode == kSrcPerPair ? sv[ib] * k + j0 : sv[ib];
      srow[ib] = S + (size_t)sr * K;
    }
    const T* wrow[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int r = rank_of_row<T>(rb, c16);
      wrow[rb] = W + (size_t)(roff + (r < r_q ? r : r_q - 1)) * a.ldw;
    }

    f32x4 acc[NRB][RB];
#pragma unroll
    for (int ib = 0; ib < NRB; ++ib)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) acc[ib][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
    // Main loop over this wave's full stages (U K-blocks each), register
    // double-buffered: the next stage's loads are in flight while the
    // matrix cores work on the current one.
    struct Stage {
      F sf[U][NRB];
      F wf[U][RB];
    };
    auto load_stage = [&](int ks0, Stage& st) {
#pragma unroll
      for (int s = 0; s < U; ++s) {
        const int kof = (ks0 + 4 * s) * KB + PER * g;
#pragma unroll
        for (int ib = 0; ib < NRB; ++ib) st.sf[s][ib] = Tr<T>::load(srow[ib] + kof);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) st.wf[s][rb] = Tr<T>::load(wrow[rb] + kof);
      }
    };
    auto mma_stage = [&](const Stage& st) {
#pragma unroll
      for (int s = 0; s < U; ++s)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          if (rb < nrb) {
#pragma unroll
            for (int ib = 0; ib < NRB; ++ib) acc[ib][rb] = Tr<T>::mma(st.wf[s][rb], st.sf[s][ib], acc[ib][rb]);
          }
    };
    // stages of this wave: ks0 = wave + 4*U*i with ks0 + 4*(U-1) < nks_full
    const int n_main = nks_full > wave + 4 * (U - 1) ? (nks_full - wave - 4 * (U - 1) + 4 * U - 1) / (4 * U) : 0;
    {
      Stage SA, SB;
      if (n_main > 0) load_stage(wave, SA);
      int i = 0;
      for (; i + 1 < n_main; i += 2) {
        load_stage(wave + 4 * U * (i + 1), SB);
        mma_stage(SA);
        if (i + 2 < n_main) load_stage(wave + 4 * U * (i + 2), SA);
        mma_stage(SB);
      }
      if (i < n_main) mma_stage(SA);
    }
    int ks0 = wave + 4 * U * n_main;
    for (; ks0 < nks; ks0 += 4) {  // leftover K-blocks of this wave (masked tail)
      const int kof = ks0 * KB + PER * g;
      const int nv = K - kof;
      const int kc = nv > 0 ? kof : 0;
      F sf[NRB], wf[RB];
#pragma unroll
      for (int ib = 0; ib < NRB; ++ib) sf[ib] = nv > 0 ? load_frag<T>(srow[ib] + kc, nv, true) : Tr<T>::zero();
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) wf[rb] = load_frag<T>(wrow[rb] + kc, nv, true);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        if (rb < nrb) {
#pragma unroll
          for (int ib = 0; ib < NRB; ++ib) acc[ib][rb] = Tr<T>::mma(wf[rb], sf[ib], acc[ib][rb]);
        }
    }

    // ---- partial sums meet in LDS; wave w finishes row block w % NRB
    __syncthreads();
#pragma unroll
    for (int ib = 0; ib < NRB; ++ib)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) red[wave][ib][rb][lane] = acc[ib][rb];
    __syncthreads();
    const int ib = wave % NRB;
    if (wave >= NRB) continue;  // the other waves' row blocks are done by waves < NRB
    const int u = u0 + 16 * ib + c16;
    if (u0 + 16 * ib >= u_end) continue;  // wave-uniform
    const bool valid = u < u_end;
    const float s = a.alpha / (float)r_q;
    f32x4 h[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      h[rb] = (((red[0][ib][rb][lane] + red[1][ib][rb][lane]) + red[2][ib][rb][lane]) +
               red[3][ib][rb][lane]) * s;
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (rank_of_row<T>(rb, 4 * g + v) >= r_q) h[rb][v] = 0.f;
    }
    if (!valid) continue;
    contract_store<T, RB>(a, q, lo, u, h);
  }
}

// ------------------------------------------------------------- bf16 path
//
// A block takes a tile of 64 rows of one key; wave w owns rows 16w .. 16w+15
// for every rank over the whole contraction, so no cross-wave reduction is
// needed.  Stages of KC contraction indices of the 64 source rows and of the
// key's weight rows are copied global -> LDS (global_load_lds_dwordx4, row
// pieces with 16-byte chunks XOR-swizzled by row), NBUF stages in flight;
// MFMA fragments are plain 16-byte LDS reads.  Only the weight rows below r_q
// (rounded up to a copy) are copied.
//
// Row sums (row_sum, pair-position sources): a row serves up to k pairs, at
// consecutive positions.  A tile then takes the rows whose first pair lies in
// a window of 65 - k positions, so their pairs (at most 64) are all in the
// tile; the per-pair results times the pair weights go to LDS in fp32 and
// every row's sum (pairs in position order) is stored once.
template <int RB, int NWV>
struct CDma {
  // contraction indices per stage and stages in LDS: ranks up to 32 take
  // 128-column stages two deep (three blocks per CU); larger ranks, whose
  // weight rows double the bytes of a stage, 64-column stages three deep
  static constexpr int KC = RB <= 2 ? 128 : 64;
  static constexpr int NBUF = RB <= 2 ? 2 : 3;  // at most 4 (see the waits)
  static constexpr int THREADS = 64 * NWV;       // NWV waves of 16 tile rows each
  static constexpr int ROWS = 16 * NWV;          // tile rows
  static constexpr int CPR = KC / 8;             // 16-byte chunks per row piece
  static constexpr int RPI = 64 / CPR;           // row pieces per copy instruction
  static constexpr int SBYTES = ROWS * KC * 2;   // tile source rows x KC bf16
  static constexpr int WROWS = 16 * RB;
  static constexpr int WBYTES = WROWS * KC * 2;  // weight rows x KC bf16
  static constexpr int NS = 16 / RPI;            // source copies per wave per stage
  static constexpr int NW = (WROWS / RPI + NWV - 1) / NWV;   // weight copies per wave per stage (at most)
  static constexpr int LDS = NBUF * (SBYTES + WBYTES);
  // LDS per CU is 160 KiB; the tile tables take about 4 KiB more per block
  static constexpr int BLOCKS_PER_CU = (160 * 1024) / (LDS + 4 * 1024 + 512) < 1 ? 1 : (160 * 1024) / (LDS + 4 * 1024 + 512);
  // row sums: per-pair results [ROWS][RPS] fp32 over the stage buffers
  static constexpr int RPS = 16 * RB + 4;   // 16-byte skew between positions
  static_assert(ROWS * RPS * 4 <= LDS, "per-pair results exceed the stage buffers");
  static_assert(WROWS / RPI <= NWV * NW, "weight copies");
};

// Chunk swizzle of weight row w (CPR 16-byte chunks per staged row).  A
// fragment read touches the rows rank_of_row(rb, i), i = 0..15: w & 3 = i & 3,
// bit 2 of w = rb & 1 and bits 3.. = i >> 2, so w & (CPR - 1) alone would give
// only four distinct chunk positions among the first eight lanes at 8 chunks
// per row (two-way bank conflicts); folding bit 3 into bit 2 spreads them
// over eight (and the 16 rows over 16 positions at 16 chunks per row).
template <int CPR>
__device__ inline int w_swz(int w) { return (w ^ ((w >> 3) << 2)) & (CPR - 1); }

// Tile size in pair positions when rows are summed (every row's pairs lie in
// the tile) or rows otherwise, for tiles of `rows` rows.
inline __host__ __device__ int contract_tile(int row_sum, int k, int rows) {
  return row_sum ? rows + 1 - k : rows;
}

// Row sums of a tile whose pair positions p0 .. p1 - 1 hold rows ua .. ub - 1
// (rstart = first position of this lane's row ua + 64 (wave / 4) + lane, rend
// the next row's, rtok its token): the per-pair results, scaled and times the
// pair weights, go to LDS (fp32); then lane l of wave w sums row ua + 64 (w /
// 4) + l over its pairs in position order for the rank chunks 8 (w % 4),
// 8 (w % 4) + 32, ... and stores the bf16 sum per key (column u - rfirst)
// and/or per token.
template <int RB, int NWV>
__device__ inline void row_sum_store(const ContractArgs& a, int q, const f32x4 (&acc)[RB], float s,
                                     float pw, int ua, int ub, int p0, int rfirst, int rstart,
                                     int rend, int rtok, float* hp) {
  constexpr int RPS = CDma<RB, NWV>::RPS;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c16 = lane & 15, g = lane >> 4;
  const int r_q = a.keys.rank[q], roff = a.keys.roff[q], R = a.keys.R;
  __syncthreads();   // every wave is done reading the staging buffers
  {
    float* dst = hp + (16 * wave + c16) * RPS;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int r0 = rank_of_row<__bf16>(rb, 4 * g);   // 4 consecutive ranks
      f32x4 h = (acc[rb] * s) * pw;
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (r0 + v >= r_q) h[v] = 0.f;
      *reinterpret_cast<f32x4*>(dst + r0) = h;
    }
  }
  __syncthreads();
  const int u = ua + 64 * (wave / 4) + lane;
  if (u >= ub) return;
  const int b0 = rstart - p0, b1 = rend - p0;
  __bf16* dt = static_cast<__bf16*>(a.out_t);
  const long col = u - rfirst;
  __bf16* df = a.out_dense ? static_cast<__bf16*>(a.out_dense) + (size_t)rtok * R + roff : nullptr;
  for (int r0 = 8 * (wave % 4); r0 < r_q; r0 += 32) {
    const float* src = hp + b0 * RPS + r0;
    f32x4 lo = *reinterpret_cast<const f32x4*>(src), hi = *reinterpret_cast<const f32x4*>(src + 4);
    for (int pos = b0 + 1; pos < b1; ++pos) {
      src += RPS;
      lo += *reinterpret_cast<const f32x4*>(src);
      hi += *reinterpret_cast<const f32x4*>(src + 4);
    }
    const bf16x8 v = {(__bf16)lo[0], (__bf16)lo[1], (__bf16)lo[2], (__bf16)lo[3],
                      (__bf16)hi[0], (__bf16)hi[1], (__bf16)hi[2], (__bf16)hi[3]};
    if (dt) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (r0 + e < r_q) dt[(size_t)(roff + r0 + e) * a.ldh + col] = v[e];
    }
    if (df) {
      if (r0 + 8 <= r_q && ((roff + r0) & 7) == 0) {
        Tr<__bf16>::store(df + r0, v);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (r0 + e < r_q) df[r0 + e] = v[e];
      }
    }
  }
}

template <int RB, int NWV>
__global__ __launch_bounds__(64 * NWV, RB == 8 ? 2 : 1) void contract_dma_kernel(ContractArgs a) {
  using G = CDma<RB, NWV>;
  constexpr int KC = G::KC, NBUF = G::NBUF, KB = Tr<__bf16>::KB;
  constexpr int CPR = G::CPR, RPI = G::RPI;
  // stage buffers: NBUF source stages, then NBUF weight stages; the row sums
  // reuse the whole area for the per-pair results
  __shared__ __attribute__((aligned(16))) char smem[G::LDS];
  char (*Sb)[G::SBYTES] = reinterpret_cast<char (*)[G::SBYTES]>(smem);
  char (*Wb)[G::WBYTES] = reinterpret_cast<char (*)[G::WBYTES]>(smem + NBUF * G::SBYTES);
  __shared__ int seg[kMaxKeys + 1];
  __shared__ int bstart[kMaxKeys + 1];
  __shared__ int bfirst[kMaxKeys];
  __shared__ int scan[kThreads];   // block_exclusive_scan reads the first kThreads / 64
  static_assert(G::THREADS >= kMaxKeys, "one thread per key in the tile tables");
  const int n_keys = a.keys.n_keys;
  const int bucket = blockIdx.x % kXcds;
  const int K = a.K, k = a.k;
  const bool rsum = a.row_sum != 0;   // implies kSrcPairList
  const int TS = contract_tile(a.row_sum, k, G::ROWS);
  build_bucket_table(a.offsets, a.src_mode == kSrcPairList ? a.ppos : nullptr, n_keys, TS, bucket,
                     seg, bstart, bfirst, scan);
  const int total = bstart[n_keys];
  const int stride = gridDim.x / kXcds;  // the grid is a multiple of kXcds
  // wave-uniform values kept in scalar registers (uniform branches, no exec masks)
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c16 = lane & 15, g = lane >> 4;
  const __bf16* S = static_cast<const __bf16*>(a.src);
  const __bf16* W = static_cast<const __bf16*>(a.W);
  const int cpos = lane & (CPR - 1), crow = lane / CPR;   // 16-byte position / row inside a copy

  for (int idx = blockIdx.x / kXcds; idx < total; idx += stride) {
    const int q = upper_index(bstart, n_keys, idx);
    const int lo = seg[q];
    int u0 = lo + (bfirst[q] + idx - bstart[q]) * TS;
    const int nst = (K + KC - 1) / KC;
    int u_end = seg[q + 1];
    const int r_q = a.keys.rank[q], roff = a.keys.roff[q];
    // row sums: rows ua .. ub - 1 start inside the window [u0, u0 + TS); their
    // pairs are positions ppos[ua] .. ppos[ub] - 1, which become u0 .. u_end
    int ua = 0, ub = 0, rfirst = 0, rtok = 0, rstart = 0, rend = 0;
    float pw = 1.f;
    if (rsum) {
      const int y = (lane & 1) ? min(u0 + TS, u_end) : u0;
      int row, pos;
      if (y < u_end) {   // first row starting at or after position y
        const int r0 = a.pair_row[a.plist[y]];
        const int s0 = a.ppos[r0], s1 = a.ppos[r0 + 1];
        row = s0 == y ? r0 : r0 + 1;
        pos = s0 == y ? s0 : s1;
      } else {
        row = a.offsets[q + 1];
        pos = u_end;
      }
      ua = __shfl(row, 0);
      ub = __shfl(row, 1);
      u0 = __shfl(pos, 0);
      u_end = __shfl(pos, 1);
      if (ua >= ub) continue;   // block-uniform: no row starts in this window
      rfirst = a.offsets[q];
      const int er = ua + 64 * (wave / 4) + lane;   // this lane's row in the epilogue
      if (er < ub) {
        rstart = a.ppos[er];
        rend = er + 1 < ub ? a.ppos[er + 1] : u_end;
        rtok = a.row_token[er];
      }
      if (a.pair_w) pw = a.pair_w[a.plist[min(u0 + 16 * wave + c16, u_end - 1)]];
    }
    // weight copies this wave issues per stage (rows below r_q only)
    const int wcopies = (r_q + RPI - 1) / RPI;
    const int nw = min(G::NW, max(0, wcopies - wave * G::NW));

    // source rows this lane copies (rows past the segment re-read the last
    // one) and the chunk of the row piece it copies
    const __bf16* sptr[G::NS];
    int scol[G::NS];
#pragma unroll
    for (int i = 0; i < G::NS; ++i) {
      const int uc = min(u0 + 16 * wave + RPI * i + crow, u_end - 1);
      int sr;
      if (a.src_mode == kSrcPairList) {
        sr = a.plist[uc];
      } else {
        const int tok = a.row_token[uc];
        sr = a.src_mode == kSrcPerPair ? tok * k + (__builtin_ctz(a.row_slots[uc] | 0x80000000u) & 31) : tok;
      }
      sptr[i] = S + (size_t)sr * K;
      scol[i] = 8 * (cpos ^ ((16 * wave + RPI * i + crow) & (CPR - 1)));
    }
    const __bf16* wptr[G::NW];
    int wcol[G::NW];
#pragma unroll
    for (int i = 0; i < G::NW; ++i) {
      const int rl = RPI * (wave * G::NW + i) + crow;  // weight row of the tile (rank)
      wptr[i] = W + (size_t)(roff + min(rl, r_q - 1)) * a.ldw;
      wcol[i] = 8 * (cpos ^ w_swz<CPR>(rl));
    }
    // copies of stage st (columns past K are clamped; masked at the reads)
    auto issue = [&](int st) {
      const int b = st % NBUF;
      const int k0 = st * KC;
#pragma unroll
      for (int i = 0; i < G::NS; ++i)
        dma16(sptr[i] + min(k0 + scol[i], K - 8),
              __builtin_amdgcn_readfirstlane(lds_addr(&Sb[b][(16 * wave + RPI * i) * KC * 2])));
#pragma unroll
      for (int i = 0; i < G::NW; ++i)
        if (i < nw)
          dma16(wptr[i] + min(k0 + wcol[i], K - 8),
                __builtin_amdgcn_readfirstlane(lds_addr(&Wb[b][RPI * (wave * G::NW + i) * KC * 2])));
    };
    const int per_stage = G::NS + nw;   // copies per stage of this wave

    __syncthreads();  // the previous tile is done with the buffers
    f32x4 acc[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p < NBUF - 1; ++p)
      if (p < nst) issue(p);
    // this wave's copies of stage st are done once at most those of the
    // stages issued after it are outstanding; the barrier publishes them
    auto begin_stage = [&](int st) {
      wait_vmcnt_upto<(NBUF - 2) * (G::NS + G::NW)>(min(NBUF - 2, nst - 1 - st) * per_stage);
      __syncthreads();
      if (st + NBUF - 1 < nst) issue(st + NBUF - 1);
    };
    // K-block kb of stage st; the ragged form masks the indices past the
    // block's range
    auto kblock = [&](int st, int kb, bool ragged) {
      const int b = st % NBUF;
      const int kk = st * KC + kb * KB;
      const int chunk = kb * 4 + g;
      const int rl = 16 * wave + c16;
      bf16x8 sf = *reinterpret_cast<const bf16x8*>(&Sb[b][rl * KC * 2 + ((chunk ^ (rl & (CPR - 1))) << 4)]);
      if (ragged) {
        const int nv = K - (kk + 8 * g);
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (e >= nv) sf[e] = (__bf16)0.f;
      }
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        // weight rows at or past r_q were not copied: their results are zeroed below
        const int wr = rank_of_row<__bf16>(rb, c16);
        const bf16x8 wf = *reinterpret_cast<const bf16x8*>(&Wb[b][wr * KC * 2 + ((chunk ^ w_swz<CPR>(wr)) << 4)]);
        acc[rb] = Tr<__bf16>::mma(wf, sf, acc[rb]);   // D[rank][row]
      }
    };
    // full stages: a loop with no branch around the matrix work (a branch
    // there made the compiler copy the accumulators every stage)
    const int nst_full = K / KC;
    for (int st = 0; st < nst_full; ++st) {
      begin_stage(st);
#pragma unroll
      for (int kb = 0; kb < KC / KB; ++kb) kblock(st, kb, false);
    }
    if (nst_full < nst) {   // block-uniform: the last, partial stage
      const int st = nst_full;
      begin_stage(st);
#pragma unroll
      for (int kb = 0; kb < KC / KB; ++kb) {
        const int kk = st * KC + kb * KB;
        if (kk < K) kblock(st, kb, kk + KB > K);
      }
    }

    const float s = a.alpha / (float)r_q;
    if (rsum) {
      row_sum_store<RB, NWV>(a, q, acc, s, pw, ua, ub, u0, rfirst, rstart, rend, rtok,
                             reinterpret_cast<float*>(smem));
      continue;
    }
    const int u = u0 + 16 * wave + c16;
    if (u0 + 16 * wave >= u_end || u >= u_end) continue;
    f32x4 h[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      h[rb] = acc[rb] * s;
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (rank_of_row<__bf16>(rb, 4 * g + v) >= r_q) h[rb][v] = 0.f;
    }
    contract_store<__bf16, RB>(a, q, lo, u, h);
  }
}

template <int RB, int NWV>
hipError_t launch_contract_dma(const ContractArgs& a, long P, hipStream_t stream) {
  using G = CDma<RB, NWV>;
  const int TS = contract_tile(a.row_sum, a.k, G::ROWS);
  // tiles per bucket <= (all tiles) / kXcds + n_keys
  const long pb = P > 0 ? ((P + TS - 1) / TS + a.keys.n_keys) / kXcds + a.keys.n_keys : 0;
  const long cap = (long)G::BLOCKS_PER_CU * device_cu_count() / kXcds;
  const int grid = (int)(pb < cap ? pb : cap) * kXcds;
  if (grid > 0) contract_dma_kernel<RB, NWV><<<grid, G::THREADS, 0, stream>>>(a);
  return hipGetLastError();
}

template <typename T, int RB>
hipError_t launch_contract_rb(const ContractArgs& a, long P, hipStream_t stream) {
  constexpr int BM = 16 * CGeo<RB>::NRB;
  // tiles per bucket <= (all tiles) / kXcds + n_keys
  const long per_bucket = P > 0 ? ((P + BM - 1) / BM + a.keys.n_keys) / kXcds + a.keys.n_keys : 0;
  if constexpr (std::is_same<T, __bf16>::value) {
    return launch_contract_dma<RB, 4>(a, P, stream);
  }
  const long cap = 6L * device_cu_count() / kXcds;
  const int grid = (int)(per_bucket < cap ? per_bucket : cap) * kXcds;
  if (grid > 0) contract_kernel<T, RB><<<grid, kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace

int rank_blocks(int r_max) {
  const int rb = (r_max + 15) / 16;
  return rb <= 2 ? 2 : rb <= 4 ? 4 : rb <= 8 ? 8 : 16;
}

int rank_pad(int dtype, int r_max) {
  // KB * (RB / APF) = 16 * RB for both element types
  (void)dtype;
  return 16 * rank_blocks(r_max);
}

hipError_t launch_contract(int dtype, const ContractArgs& a, int r_max, long P,
                           hipStream_t stream) {
  if (a.row_sum && (dtype != ACE_BF16 || a.src_mode != kSrcPairList)) return hipErrorInvalidValue;
  const int rb = rank_blocks(r_max);
  if (dtype == ACE_BF16) {
    if (rb == 2) return launch_contract_rb<__bf16, 2>(a, P, stream);
    if (rb == 4) return launch_contract_rb<__bf16, 4>(a, P, stream);
    if (rb == 8) return launch_contract_rb<__bf16, 8>(a, P, stream);
    return launch_contract_rb<__bf16, 16>(a, P, stream);
  }
  if (rb == 2) return launch_contract_rb<float, 2>(a, P, stream);
  if (rb == 4) return launch_contract_rb<float, 4>(a, P, stream);
  if (rb == 8) return launch_contract_rb<float, 8>(a, P, stream);
  return launch_contract_rb<float, 16>(a, P, stream);
}

}  // namespace ace
