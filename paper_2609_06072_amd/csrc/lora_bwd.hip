// Grouped LoRA backward: gradients of L = <dY, Y_out> (Sec. 3.1.2 and 3.4 --
// a shared adapter collects the gradient of every routed pair of its group).
//
// With G_u = sum_{j in slots(u)} w_j dY[t*k+j] (the row's output gradient),
// s_q = alpha / r_q, Hs_u = s_q A_q x_u and dH_u = s_q B_q^T G_u:
//   dB_q  = sum_u G_u Hs_u^T                    (per key, K = rows of q)
//   dA_q  = sum_u dH_u x_u^T                    (per key, K = rows of q)
//   dx    += sum over the rows that read x of A_q^T dH_u
//
// Launches, all deterministic (each output is reduced in a fixed order):
//   prep      -- A^T and B_q^T into the workspace (so every MFMA operand is
//                contiguous along its contraction index); zeroes the dense
//                per-token dH buffer used for dx; when the forward's h is
//                passed in, builds Hw (below) from it in the same launch.
//   contract  -- without the forward's h: Hs per row (x against A), stored
//                per key and per pair served as [r][pair position], times the
//                pair's weight (Hw).
//   contract  -- dH per row (gathered G against B^T), stored per key as
//                [r][u] and either as dense per-token rows (shared input) or
//                row-major for the expand below (per-pair input).  Rows that
//                serve several pairs are contracted per pair and summed per
//                row: in the contraction's epilogue (bf16) or by a combine
//                launch (fp32).
//   expand    -- per-pair input only: dx[t*k+j] += A_q^T dH_u (each row owns
//                its input row).
//   grads     -- dB_q over each key's pairs and dA_q over its rows (split into
//                chunks for skewed keys, partials summed in order).
//   dx GEMM   -- shared input only: dx += dHdense A over K = R (token-major).
#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

constexpr int kTile = 64;   // transpose tile / column block
constexpr int kMaxJobs = kMaxKeys + 3;

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

struct WsLayout {
  size_t At, Bt, Ht, dHt, dHf, dHrow, part, dHp, total;
};

// Ranks up to 16 take the backward in which the dB pass also contracts dY
// against B^T (bf16): its fp32 partials per column block use this rank stride.
constexpr int kFusedDhMaxRank = 16;
int dh_stride(int r_max) { return r_max <= 8 ? 8 : 16; }
// With shared input the dB pass forms the dH partials only for outputs of at
// least this many columns: below it the second read of dY is cheap and the
// dA items overlap best with the dB items in one launch.
constexpr int kSharedDhMinOut = 1280;
// Ranks 33..64 (bf16, shared input, outputs of at least kSharedDhMinOut
// columns): dB items of kWideCols columns form the dH partials (a
// contraction over all of d_out, re-reading dY, otherwise).
bool wide_dh(int r_max, int d_out) { return rank_blocks(r_max) == 4 && d_out >= kSharedDhMinOut; }
// outputs below this many columns take dB items of 512 pairs on the wide path
constexpr int kWideLongOut = 4096;
constexpr int kWideSplitB = 4096;   // dB chunk of the wide items from kWideLongOut columns

// Workspace regions for element size es: At [d_in][R], Bt [R][d_out],
// Ht/dHt [R][ldh] (column = row index inside the key's segment), dense dH
// [T*kslots][R] (kslots <= k), row-major dH [P][rpad], split partials of the
// weight gradients; 256 bytes of slack at the end, since the gradient pass
// reads whole 16-byte fragments of Ht/dHt rows past a segment's end (and
// masks them).
WsLayout ws_layout(int T, int k, int d_in, int d_out, int n_keys, int R, int r_max, size_t es) {
  const int rpad = rank_pad(ACE_F32, r_max);
  const size_t P = (size_t)T * k;
  const size_t ldh = (P + 7) & ~(size_t)7;
  const size_t nbB = (d_out + kGradColBlk - 1) / kGradColBlk;
  WsLayout w{};
  size_t o = 0;
  w.At = o;    o += align256(es * d_in * R);
  w.Bt = o;    o += align256(es * (size_t)R * d_out);
  w.Ht = o;    o += align256(es * (size_t)R * ldh);
  w.dHt = o;   o += align256(es * (size_t)R * ldh);
  w.dHf = o;   o += align256(es * P * R);
  w.dHrow = o; o += align256(es * P * rpad);
  w.part = o;  o += align256(grads_part_bytes(T, k, d_in, d_out, n_keys, r_max));
  const size_t nbW = (d_out + kWideCols - 1) / kWideCols;
  w.dHp = o;   o += r_max <= kFusedDhMaxRank ? align256(sizeof(float) * nbB * P * dh_stride(r_max))
                    : wide_dh(r_max, d_out) ? align256(sizeof(float) * nbW * P * 64) : 0;
  w.total = o + 256;
  return w;
}

// Sum over the pairs of a row: dH_u = sum_i w_{p_i} dHp[ppos[u] + i]
// (dHp = s B^T dY per pair position, row-major [P][rpad]); written per key as
// [r][u - offsets[q]] for the weight gradient and/or as dense per-token rows
// for the dx GEMM (either output may be null).  The pre-combined mode uses
// the same sum for h_u = sum_i w_{p_i} h_{p_i}.
struct CombineArgs {
  const int32_t* offsets;
  const int32_t* row_token;
  const int32_t* ppos;
  const int32_t* plist;
  const float* pair_w;
  const void* dHp;
  int32_t rpad;
  void* dHt;
  long ldh;
  void* dHf;
  KeyTable keys;
};

// A block takes 64 consecutive rows; lane l of wave w handles row 64b + l and
// the rank chunks w, w + 4, ... (PER ranks each), so the transposed stores of
// a wave cover 64 consecutive columns.  The first two pairs of a row are
// loaded unconditionally (a missing second pair gets weight 0); further pairs
// (rare) are added in a loop.
template <typename T>
__global__ __launch_bounds__(kThreads) void combine_kernel(CombineArgs a) {
  constexpr int PER = Tr<T>::PER;
  __shared__ int seg[kMaxKeys + 1];
  const int n_keys = a.keys.n_keys;
  for (int i = threadIdx.x; i <= n_keys; i += kThreads) seg[i] = a.offsets[i];
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int U = seg[n_keys];
  const int u = blockIdx.x * 64 + lane;
  if (u >= U) return;
  const int q = upper_index(seg, n_keys, u);
  const int r_q = a.keys.rank[q], roff = a.keys.roff[q], R = a.keys.R;
  const long col = u - seg[q];
  const int tok = a.row_token[u];
  const int p0 = a.ppos[u], p1 = a.ppos[u + 1];
  const int pb = min(p0 + 1, p1 - 1);
  float w0 = 1.f, w1 = p1 - p0 > 1 ? 1.f : 0.f;
  if (a.pair_w) {
    const float x0 = a.pair_w[a.plist[p0]], x1 = a.pair_w[a.plist[pb]];
    w0 = x0;
    w1 = p1 - p0 > 1 ? x1 : 0.f;
  }
  const T* src = static_cast<const T*>(a.dHp);
  T* dt = static_cast<T*>(a.dHt);
  T* df = a.dHf ? static_cast<T*>(a.dHf) + (size_t)tok * R + roff : nullptr;
  for (int r0 = PER * wave; r0 < r_q; r0 += 4 * PER) {
    float f0[PER], f1[PER];
    Tr<T>::to_f32(Tr<T>::load(src + (size_t)p0 * a.rpad + r0), f0);
    Tr<T>::to_f32(Tr<T>::load(src + (size_t)pb * a.rpad + r0), f1);
    float acc[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] = w0 * f0[e] + w1 * f1[e];
    for (int pos = p0 + 2; pos < p1; ++pos) {
      const float w = a.pair_w ? a.pair_w[a.plist[pos]] : 1.f;
      float f[PER];
      Tr<T>::to_f32(Tr<T>::load(src + (size_t)pos * a.rpad + r0), f);
#pragma unroll
      for (int e = 0; e < PER; ++e) acc[e] += w * f[e];
    }
#pragma unroll
    for (int e = 0; e < PER; ++e)
      if (r0 + e < r_q) {
        const T v = (T)acc[e];
        if (dt) dt[(size_t)(roff + r0 + e) * a.ldh + col] = v;
        if (df) df[r0 + e] = v;
      }
  }
}

// Hw from the forward's h (h_u = s_q A_q x_u per row, row-major [U][rpad]):
// Hw[roff + r][pair position - first pair of the key] = w_p h_u[r] for every
// pair p the row serves -- what the Hs contract below would store.  Runs as
// blocks of the prep launch: lane l of wave w handles row 64 blk + l and the
// rank chunks w, w + 4, ...
struct HwJob {
  const int32_t* offsets;
  const int32_t* row_token;
  const uint32_t* row_slots;
  const int32_t* ppos;   // first pair position of each row, or null (one pair per row)
  const float* pair_w;
  const void* h;
  int32_t rpad;
  int32_t k;
  void* Hw;
  long ldh;
};

template <typename T>
__device__ inline void hw_rows(const HwJob& a, const KeyTable& keys, int blk, int* seg) {
  constexpr int PER = Tr<T>::PER;
  const int n_keys = keys.n_keys;
  for (int i = threadIdx.x; i <= n_keys; i += kThreads) seg[i] = a.offsets[i];
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int u = blk * 64 + lane;
  if (u >= seg[n_keys]) return;
  const int q = upper_index(seg, n_keys, u);
  const int r_q = keys.rank[q], roff = keys.roff[q];
  const int tok = a.row_token[u];
  const uint32_t slots = a.row_slots[u];
  const long col0 = a.ppos ? (long)a.ppos[u] - a.ppos[seg[q]] : (long)(u - seg[q]);
  const T* src = static_cast<const T*>(a.h) + (size_t)u * a.rpad;
  T* dst = static_cast<T*>(a.Hw);
  for (int r0 = PER * wave; r0 < r_q; r0 += 4 * PER) {
    float f[PER];
    Tr<T>::to_f32(Tr<T>::load(src + r0), f);
    long col = col0;
    for (uint32_t mm = slots; mm; mm &= mm - 1u, ++col) {
      const float w = a.pair_w ? a.pair_w[tok * a.k + __builtin_ctz(mm)] : 1.f;
#pragma unroll
      for (int e = 0; e < PER; ++e)
        if (r0 + e < r_q) dst[(size_t)(roff + r0 + e) * a.ldh + col] = (T)(f[e] * w);
    }
  }
}

// ------------------------------------------------------------------ prep

struct PrepArgs {
  const void* A;
  const void* B;
  void* At;
  void* Bt;
  void* dHf;
  int32_t d_in, d_out, R;
  long dHf_vecs;                    // 16-byte vectors to zero
  int32_t n_jobs;
  int32_t job_start[kMaxJobs + 1];  // block ranges: job 0 = A, 1..n_keys = B_q, n_keys + 1 =
                                    //   zero, n_keys + 2 = Hw rows
  int32_t job_cols_tiles[kMaxJobs];
  HwJob hw;
  KeyTable keys;
};

template <typename T>
__global__ __launch_bounds__(kThreads) void bwd_prep_kernel(PrepArgs a) {
  __shared__ T tile[kTile][kTile + 1];
  __shared__ int seg[kMaxKeys + 1];
  const int b = blockIdx.x;
  const int job = upper_index(a.job_start, a.n_jobs, b);
  const int tb = b - a.job_start[job];
  const int n_keys = a.keys.n_keys;
  if (job == n_keys + 2) {  // Hw from the forward's h
    hw_rows<T>(a.hw, a.keys, tb, seg);
    return;
  }
  if (job == n_keys + 1) {  // zero the dense dH buffer
    u32x4* d = static_cast<u32x4*>(a.dHf);
    const long base = (long)tb * kThreads * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const long e = base + i * kThreads + threadIdx.x;
      if (e < a.dHf_vecs) d[e] = u32x4{0u, 0u, 0u, 0u};
    }
    return;
  }
  // transpose src [rows][cols] (row stride lds) -> dst [cols][rows] (row stride ldd)
  const T* src;
  T* dst;
  int rows, cols, lds, ldd;
  if (job == 0) {
    src = static_cast<const T*>(a.A);
    dst = static_cast<T*>(a.At);
    rows = a.R; cols = a.d_in; lds = a.d_in; ldd = a.R;
  } else {
    const int q = job - 1;
    const int r_q = a.keys.rank[q], roff = a.keys.roff[q];
    src = static_cast<const T*>(a.B) + (size_t)a.d_out * roff;   // B_q [d_out][r_q]
    dst = static_cast<T*>(a.Bt) + (size_t)roff * a.d_out;        // Bt rows roff.. [r_q][d_out]
    rows = a.d_out; cols = r_q; lds = r_q; ldd = a.d_out;
  }
  using F = typename Tr<T>::frag;
  constexpr int PER = Tr<T>::PER;
  constexpr int PPR = kTile / PER;            // 16-byte pieces per tile row
  constexpr int NP = kTile * PPR / kThreads;  // pieces per thread
  const int ct = a.job_cols_tiles[job];
  const int r0 = (tb / ct) * kTile, c0 = (tb % ct) * kTile;
  // 16-byte pieces when rows are aligned; then a piece is either wholly
  // inside the matrix or wholly outside (cols and rows are multiples of PER)
  const bool vs = (lds % PER) == 0 && (cols % PER) == 0;
  const bool vd = (ldd % PER) == 0 && (rows % PER) == 0;
  if (vs) {
    F v[NP];
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const int pc = threadIdx.x + i * kThreads;
      const int rr = pc / PPR, cc = (pc % PPR) * PER;
      v[i] = Tr<T>::load(src + (size_t)min(r0 + rr, rows - 1) * lds + min(c0 + cc, cols - PER));
    }
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const int pc = threadIdx.x + i * kThreads;
      const int rr = pc / PPR, cc = (pc % PPR) * PER;
#pragma unroll
      for (int e = 0; e < PER; ++e) tile[rr][cc + e] = v[i][e];
    }
  } else {
    for (int i = threadIdx.x; i < kTile * kTile; i += kThreads) {
      const int rr = i / kTile, cc = i % kTile;
      if (r0 + rr < rows && c0 + cc < cols) tile[rr][cc] = src[(size_t)(r0 + rr) * lds + c0 + cc];
    }
  }
  __syncthreads();
  if (vd) {
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const int pc = threadIdx.x + i * kThreads;
      const int cc = pc / PPR, rr = (pc % PPR) * PER;
      F o;
#pragma unroll
      for (int e = 0; e < PER; ++e) o[e] = tile[rr + e][cc];
      if (c0 + cc < cols && r0 + rr < rows) Tr<T>::store(dst + (size_t)(c0 + cc) * ldd + r0 + rr, o);
    }
  } else {
    for (int i = threadIdx.x; i < kTile * kTile; i += kThreads) {
      const int cc = i / kTile, rr = i % kTile;
      if (r0 + rr < rows && c0 + cc < cols) dst[(size_t)(c0 + cc) * ldd + r0 + rr] = tile[rr][cc];
    }
  }
}

template <typename T>
hipError_t launch_prep_t(const Problem& p, void* At, void* Bt, void* zero, long zero_bytes,
                         const HwJob* hw, hipStream_t stream) {
  const int R = p.keys.R;
  const int n_keys = p.keys.n_keys;
  PrepArgs pa{};
  pa.A = p.A;
  pa.B = p.B;
  pa.At = At;
  pa.Bt = Bt;
  pa.dHf = zero;
  pa.d_in = p.d_in;
  pa.d_out = p.d_out;
  pa.R = R;
  pa.dHf_vecs = (zero_bytes + 15) / 16;   // the region is 256-byte padded
  pa.keys = p.keys;
  pa.n_jobs = n_keys + 3;
  long nb = 0;
  auto tiles = [](long x) { return (x + kTile - 1) / kTile; };
  pa.job_start[0] = 0;
  pa.job_cols_tiles[0] = (int)tiles(p.d_in);
  nb += At ? tiles(R) * tiles(p.d_in) : 0;
  for (int q = 0; q < n_keys; ++q) {
    pa.job_start[q + 1] = (int)nb;
    pa.job_cols_tiles[q + 1] = (int)tiles(p.keys.rank[q]);
    nb += Bt ? tiles(p.d_out) * tiles(p.keys.rank[q]) : 0;
  }
  pa.job_start[n_keys + 1] = (int)nb;
  pa.job_cols_tiles[n_keys + 1] = 1;
  nb += (pa.dHf_vecs + 4 * kThreads - 1) / (4 * kThreads);
  pa.job_start[n_keys + 2] = (int)nb;
  pa.job_cols_tiles[n_keys + 2] = 1;
  if (hw) {
    pa.hw = *hw;
    nb += ((long)p.T * p.k + 63) / 64;
  }
  pa.job_start[n_keys + 3] = (int)nb;
  if (nb > 0) bwd_prep_kernel<T><<<(int)nb, kThreads, 0, stream>>>(pa);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_combine_t(const Problem& p, const void* hp, int rpad, void* Ht, long ldh,
                            void* Hd, hipStream_t stream) {
  CombineArgs cb{};
  cb.offsets = p.rt->offsets;
  cb.row_token = p.rt->row_token;
  cb.ppos = p.rt->row_pair;
  cb.plist = p.rt->pair_list;
  cb.pair_w = p.pair_w;
  cb.dHp = hp;
  cb.rpad = rpad;
  cb.dHt = Ht;
  cb.ldh = ldh;
  cb.dHf = Hd;
  cb.keys = p.keys;
  const long P = (long)p.T * p.k;
  const int blocks = (int)((P + 63) / 64);
  if (blocks > 0) combine_kernel<T><<<blocks, kThreads, 0, stream>>>(cb);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_bwd_t(const Problem& p, const void* dy, void* dx, float* dA, float* dB,
                        void* ws, hipStream_t stream) {
  const int R = p.keys.R;
  const int n_keys = p.keys.n_keys;
  const int rpad = rank_pad(p.dtype, p.r_max);
  const WsLayout L = ws_layout(p.T, p.k, p.d_in, p.d_out, n_keys, R, p.r_max, sizeof(T));
  char* base = static_cast<char*>(ws);
  const long P = (long)p.T * p.k;
  const long ldh = (long)((((size_t)P) + 7) & ~(size_t)7);
  // kslots: rows of the dense dH buffer per token (1 when (token, key) is unique)
  const int kslots = (!p.per_pair && p.rt->mode == ACE_ROWS_GROUP_PAIRS) ? p.k : 1;

  const long dHf_bytes = p.per_pair ? 0 : (long)p.T * kslots * R * (long)sizeof(T);
  // A^T feeds the per-pair dx expand and the register dx GEMM; the bf16 dx
  // GEMM reads A itself when the dense dH rows are 16-byte aligned
  const bool need_At = p.per_pair || p.dtype != ACE_BF16 || (kslots * R) % 8 != 0;
  // pair positions of rows that serve several slots (from the permutation)
  const bool multi = p.rt->mode == ACE_ROWS_GROUP_DEDUP;
  const int32_t* ppos = multi ? p.rt->row_pair : nullptr;
  const int32_t* plist = multi ? p.rt->pair_list : nullptr;
  // Hw = w s A x, per key and pair [r][pair position]: from the forward's h
  // (blocks of the prep launch) when the caller kept it, else recomputed
  HwJob hw{};
  if (p.h_fwd) {
    hw.offsets = p.rt->offsets;
    hw.row_token = p.rt->row_token;
    hw.row_slots = p.rt->row_slots;
    hw.ppos = ppos;
    hw.pair_w = p.pair_w;
    hw.h = p.h_fwd;
    hw.rpad = rpad;
    hw.k = p.k;
    hw.Hw = base + L.Ht;
    hw.ldh = ldh;
  }
  hipError_t e = launch_prep_t<T>(p, need_At ? base + L.At : nullptr, base + L.Bt, base + L.dHf,
                                  dHf_bytes, p.h_fwd ? &hw : nullptr, stream);
  if (e != hipSuccess) return e;

  ContractArgs c{};
  c.k = p.k;
  c.alpha = p.alpha;
  c.offsets = p.rt->offsets;
  c.row_token = p.rt->row_token;
  c.row_slots = p.rt->row_slots;
  c.rpad = rpad;
  c.ldh = ldh;
  c.kslots = kslots;
  c.keys = p.keys;
  c.pair_w = p.pair_w;
  if (!p.h_fwd) {
    c.src = p.x;
    c.W = p.A;
    c.ldw = p.d_in;
    c.K = p.d_in;
    c.src_mode = p.per_pair ? kSrcPerPair : kSrcShared;
    c.out_t = base + L.Ht;
    c.out_t_pairs = 1;
    c.ppos = ppos;
    e = launch_contract(p.dtype, c, p.r_max, P, stream);
    if (e != hipSuccess) return e;
  }
  GradArgs gr{};
  gr.x = p.x;
  gr.dy = dy;
  gr.Hw = base + L.Ht;
  gr.dHt = base + L.dHt;
  gr.ppos = ppos;
  gr.plist = plist;
  gr.ldh = ldh;
  gr.dA = dA;
  gr.dB = dB;
  gr.part = base + L.part;
  gr.offsets = p.rt->offsets;
  gr.row_token = p.rt->row_token;
  gr.row_slots = p.rt->row_slots;
  gr.k = p.k;
  gr.d_in = p.d_in;
  gr.d_out = p.d_out;
  gr.per_pair = p.per_pair;
  gr.keys = p.keys;
  // shared input at ranks up to 32 with long keys (bf16, at least 1024 pairs
  // per key on average): 2048 contraction indices per item, so that most keys
  // need no split reduction; otherwise 1024 (shorter keys balance better over
  // more items, and higher ranks and the per-pair passes have more work per
  // item)
  const bool long_keys = (long)p.T * p.k >= 1024L * n_keys;
  gr.split = (p.dtype == ACE_BF16 && !p.per_pair && rank_blocks(p.r_max) <= 2 && long_keys) ? 2048
                                                                                            : 1024;
  // Shared input at ranks above 32 with many gradient column blocks (wide
  // projections): the split partials grow with the rank and the number of
  // chunks, so take chunks of 2048 when that still leaves at least four items
  // per CU (three blocks per CU are resident; 4096 left the last round of
  // items a third full and measured slower)
  if (p.dtype == ACE_BF16 && !p.per_pair && rank_blocks(p.r_max) == 4) {
    const long nb = (p.d_out + kGradColBlk - 1) / kGradColBlk + (p.d_in + kGradColBlk - 1) / kGradColBlk;
    if ((long)p.T * p.k / 2048 * nb >= 4L * device_cu_count()) gr.split = 2048;
  }
  // Ranks up to 16 (bf16) with per-pair input, or with shared input and
  // outputs of at least kSharedDhMinOut columns: the dB pass reads dY once and
  // also contracts it against B^T per 128-column block (fp32 partials); dH per
  // row is their sum, then the dA pass.  Ranks 33..64 with shared input and
  // wide outputs: the same with dB items of kWideCols columns (partials of 64
  // ranks per 512 columns).  Otherwise dH by a contraction over all of d_out
  // before the weight gradients: per-block partials of more ranks would cost
  // more than the second read of dY, and for narrow outputs the dA items (x
  // rows from the caches) run best mixed with the dB items in one launch.
  const bool wide = p.dtype == ACE_BF16 && !p.per_pair && wide_dh(p.r_max, p.d_out);
  // narrow outputs give the 512-column items few column blocks: the shortest
  // pair chunks (512 or 768) that still leave at most one item per CU keep
  // more CUs busy (one block per CU; the dA items keep their chunks)
  if (wide && p.d_out < kWideLongOut) {
    const long nbW = (p.d_out + kWideCols - 1) / kWideCols;
    for (int sb = 512; sb <= 768; sb += 256)
      if (((long)p.T * p.k / sb + n_keys) * nbW <= device_cu_count()) {
        gr.split_b = sb;
        break;
      }
  } else if (wide) {
    // wide outputs: chunks of up to 4096 pairs halve the dB partials against
    // 2048; the items' critical path is the same, since at 2048 most blocks
    // take two items (Mixtral-like: 224 items of 4096 pairs, one per CU,
    // against 448 of 2048)
    gr.split_b = kWideSplitB;
  }
  if ((p.dtype == ACE_BF16 && (p.per_pair || p.d_out >= kSharedDhMinOut) && p.r_max <= kFusedDhMaxRank) ||
      wide) {
    gr.phase = 1;
    gr.dHp = reinterpret_cast<float*>(base + L.dHp);
    gr.npos = P;
    gr.dhs = wide ? 64 : dh_stride(p.r_max);
    gr.Bt = base + L.Bt;
    e = wide ? launch_grads_wide(gr, P, stream) : launch_grads(p.dtype, gr, p.r_max, P, stream);
    if (e != hipSuccess) return e;
    DhReduceArgs d{};
    d.dHp = gr.dHp;
    d.npos = P;
    d.dhs = gr.dhs;
    d.pos_major = wide ? 1 : 0;
    d.nbB = wide ? (p.d_out + kWideCols - 1) / kWideCols : (p.d_out + kGradColBlk - 1) / kGradColBlk;
    d.offsets = p.rt->offsets;
    d.row_token = p.rt->row_token;
    d.row_slots = p.rt->row_slots;
    d.ppos = ppos;
    d.plist = plist;
    d.pair_w = p.pair_w;
    d.k = p.k;
    d.alpha = p.alpha;
    d.dHt = base + L.dHt;
    d.ldh = ldh;
    d.dHrow = p.per_pair ? base + L.dHrow : nullptr;
    d.rpad = rpad;
    d.dHf = p.per_pair ? nullptr : base + L.dHf;
    d.kslots = kslots;
    d.keys = p.keys;
    e = launch_dh_reduce(d, P, stream);
    if (e != hipSuccess) return e;
    gr.phase = 2;
    e = launch_grads(p.dtype, gr, p.r_max, P, stream);
    if (e != hipSuccess) return e;
  } else {
    // dH = s B^T G
    c.W = base + L.Bt;
    c.ldw = p.d_out;
    c.K = p.d_out;
    c.src = dy;
    c.out_t_pairs = 0;
    c.ppos = nullptr;
    if (multi && p.dtype == ACE_BF16) {
      // per pair position (single dY rows), summed per row in the epilogue
      c.src_mode = kSrcPairList;
      c.plist = plist;
      c.ppos = ppos;
      c.pair_row = p.rt->pair_row;
      c.row_sum = 1;
      c.out_w = 0;
      c.out_t = base + L.dHt;
      c.out_dense = base + L.dHf;
      c.out_row = nullptr;
      e = launch_contract(p.dtype, c, p.r_max, P, stream);
    } else if (multi) {
      // per pair position (single dY rows), then summed per row
      c.src_mode = kSrcPairList;
      c.plist = plist;
      c.ppos = ppos;
      c.out_w = 0;
      c.out_t = nullptr;
      c.out_dense = nullptr;
      c.out_row = base + L.dHrow;
      e = launch_contract(p.dtype, c, p.r_max, P, stream);
      if (e != hipSuccess) return e;
      e = launch_combine_t<T>(p, base + L.dHrow, rpad, base + L.dHt, ldh, base + L.dHf, stream);
    } else {
      c.src_mode = kSrcPerPair;
      c.out_w = 1;
      c.out_t = base + L.dHt;
      c.out_dense = p.per_pair ? nullptr : base + L.dHf;
      c.out_row = p.per_pair ? base + L.dHrow : nullptr;
      e = launch_contract(p.dtype, c, p.r_max, P, stream);
    }
    if (e != hipSuccess) return e;
    e = launch_grads(p.dtype, gr, p.r_max, P, stream);
    if (e != hipSuccess) return e;
  }
  if (p.per_pair) {
    // dx = A^T dH per pair, after the weight gradients: they read dY again,
    // which the contraction has just pulled through the caches, and dx's
    // read-modify-write in between would push it out
    ExpandArgs x{};
    x.H = base + L.dHrow;
    x.rpad = rpad;
    x.W = base + L.At;
    x.w_key_mul = 1;
    x.w_stride_is_rank = 0;
    x.offsets = p.rt->offsets;
    x.row_token = p.rt->row_token;
    x.row_slots = p.rt->row_slots;
    x.k = p.k;
    x.n_out = p.d_in;
    x.out = dx;
    x.pair_w = nullptr;
    x.keys = p.keys;
    x.multi_slot = p.rt->mode == ACE_ROWS_GROUP_DEDUP;
    return launch_expand(p.dtype, x, p.r_max, P, stream);
  }

  DxArgs d{};
  d.dHf = base + L.dHf;
  d.At = base + L.At;
  d.A = p.A;
  d.dx = dx;
  d.T = p.T;
  d.d_in = p.d_in;
  d.R = R;
  d.KR = kslots * R;
  return launch_dx_gemm(p.dtype, d, stream);
}

}  // namespace

size_t bwd_ws_bytes(int T, int k, int d_in, int d_out, int n_keys, int R, int r_max) {
  return ws_layout(T, k, d_in, d_out, n_keys, R, r_max, sizeof(float)).total;
}

hipError_t launch_prep(const Problem& p, void* At, void* Bt, void* zero, long zero_bytes,
                       hipStream_t stream) {
  if (p.dtype == ACE_BF16) return launch_prep_t<__bf16>(p, At, Bt, zero, zero_bytes, nullptr, stream);
  return launch_prep_t<float>(p, At, Bt, zero, zero_bytes, nullptr, stream);
}

hipError_t launch_combine(const Problem& p, const void* hp, int rpad, void* Ht, long ldh,
                          void* Hd, hipStream_t stream) {
  if (p.dtype == ACE_BF16) return launch_combine_t<__bf16>(p, hp, rpad, Ht, ldh, Hd, stream);
  return launch_combine_t<float>(p, hp, rpad, Ht, ldh, Hd, stream);
}

hipError_t launch_bwd(const Problem& p, const void* dy, void* dx, float* dA, float* dB, void* ws,
                      hipStream_t stream) {
  if (p.dtype == ACE_BF16) return launch_bwd_t<__bf16>(p, dy, dx, dA, dB, ws, stream);
  return launch_bwd_t<float>(p, dy, dx, dA, dB, ws, stream);
}

}  // namespace ace
