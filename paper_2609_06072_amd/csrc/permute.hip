// Route expansion and permutation (Sec. 3.5: the active group set A(x) of each
// token, one row per (token, active group); or one row per routed pair for the
// expert-wise and "shared adapter, per-pair" modes).
//
// A stable counting sort of the emitted rows by key, in two or three launches:
//   count   -- each block owns a chunk of whole tokens (<= 256 pairs).  The
//              block's keys go to LDS; each emitted row sets the bit of its
//              local pair index in a per-key bitmap (LDS, ds_or_b64), and the
//              per-(key, block) population counts are written key-major.
//   scan    -- one block: exclusive scan of the key-major counts gives each
//              (key, block) its first row; counts/offsets/n_dropped written.
//              Only for large cell tables: otherwise every scatter block
//              derives the bases of its own cells from the count table
//              (per-key totals and prefixes, exact integer sums) and block 0
//              writes counts/offsets/n_dropped.
//   scatter -- rebuilds the bitmap; a row's rank inside its (key, block) cell
//              is the popcount of the lower bits, so rows come out sorted by
//              (key, token, slot) with no atomics on rows and no sort.
// Pair positions (the routed pairs in (key, token, slot) order) follow the
// same scheme: in ACE_ROWS_GROUP_DEDUP mode a second bitmap marks every pair
// of a key and second cell table is scanned; in the other modes a row is a
// pair and its position is its row.
#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

constexpr int kPairsPerBlock = 256;
constexpr int kWordsPerKey = kPairsPerBlock / 64;

struct PermArgs {
  const int32_t* ids;
  const int32_t* e2g;  // null in expert mode
  int32_t T, k, E, G, mode, n_keys;
  int32_t tokens_per_block, nblk;
  int32_t fold;        // the scatter derives the cell bases itself (no scan launch)
  int32_t* cell;       // [n_keys * nblk] counts, then (scan) first rows
  int32_t* pcell;      // [n_keys * nblk] pair counts, then first pair positions (dedup)
  int32_t* drops;      // [nblk]
  int32_t* counts;
  int32_t* offsets;
  int32_t* row_token;
  uint32_t* row_slots;
  int32_t* pair_row;
  int32_t* n_dropped;
  int32_t* row_pair;
  int32_t* pair_list;
};

// Stage the block's pair keys (-1 = dropped) and mark emitted rows in the
// per-key bitmaps.  Returns the number of dropped pairs seen by this thread.
// In ACE_ROWS_GROUP_DEDUP mode pbits (right after bits) also marks every pair.
__device__ int stage_and_mark(const PermArgs& a, int p0, int np, int* keys, uint32_t* masks,
                              unsigned long long* bits) {
  const int t = threadIdx.x;
  int drops = 0;
  const bool dedup = a.mode == ACE_ROWS_GROUP_DEDUP;
  unsigned long long* pbits = bits + a.n_keys * kWordsPerKey;
  for (int i = t; i < a.n_keys * kWordsPerKey * (dedup ? 2 : 1); i += kThreads) bits[i] = 0ull;
  for (int lp = t; lp < np; lp += kThreads) {
    const int e = a.ids[p0 + lp];
    int q = -1;
    if (e >= 0 && e < a.E) {
      if (a.mode == ACE_ROWS_EXPERT) {
        q = e;
      } else {
        const int g = a.e2g[e];
        q = (g >= 0 && g < a.G) ? g : -1;
      }
    }
    drops += q < 0;
    keys[lp] = q;
  }
  __syncthreads();
  const int k = a.k;
  for (int lp = t; lp < np; lp += kThreads) {
    const int q = keys[lp];
    if (q < 0) { masks[lp] = 0u; continue; }
    uint32_t m = 1u << (lp % k);
    bool emit = true;
    if (a.mode == ACE_ROWS_GROUP_DEDUP) {
      // leader = first slot of the token with this group; mask = all of them
      const int j = lp % k, tb = lp - j;
      for (int jj = 0; jj < k; ++jj) {
        if (keys[tb + jj] != q) continue;
        if (jj < j) { emit = false; break; }
        m |= 1u << jj;
      }
    }
    masks[lp] = emit ? m : 0u;
    if (emit) atomicOr(&bits[q * kWordsPerKey + (lp >> 6)], 1ull << (lp & 63));
    if (dedup) atomicOr(&pbits[q * kWordsPerKey + (lp >> 6)], 1ull << (lp & 63));
  }
  __syncthreads();
  return drops;
}

__global__ __launch_bounds__(kThreads) void permute_count_kernel(PermArgs a) {
  extern __shared__ unsigned long long bits[];  // [n_keys * kWordsPerKey]
  __shared__ int keys[kPairsPerBlock];
  __shared__ uint32_t masks[kPairsPerBlock];
  __shared__ int red[kThreads];
  const int b = blockIdx.x;
  const int p0 = b * a.tokens_per_block * a.k;
  const int np = min(a.tokens_per_block * a.k, a.T * a.k - p0);
  const int d = stage_and_mark(a, p0, np, keys, masks, bits);
  const bool dedup = a.mode == ACE_ROWS_GROUP_DEDUP;
  for (int q = threadIdx.x; q < a.n_keys; q += kThreads) {
    int c = 0, pc = 0;
#pragma unroll
    for (int w = 0; w < kWordsPerKey; ++w) {
      c += __popcll(bits[q * kWordsPerKey + w]);
      if (dedup) pc += __popcll(bits[(a.n_keys + q) * kWordsPerKey + w]);
    }
    a.cell[q * a.nblk + b] = c;
    if (dedup) a.pcell[q * a.nblk + b] = pc;
  }
  int total;
  block_exclusive_scan(d, red, &total);
  if (threadIdx.x == 0) a.drops[b] = total;
}

// Inclusive scan of one int per lane across a wave of 64.
__device__ inline int wave_inclusive_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int o = __shfl_up(v, off, 64);
    if (lane >= off) v += o;
  }
  return v;
}

// Exclusive scans in place of v[0 .. N) and w[0 .. N) (w may be null) by one
// block of 1024 threads (16 waves); returns the totals.
__device__ int2 scan_cells(int32_t* v, int32_t* w, int N, int2* part) {
  constexpr int MAXPER = 16;   // cells per thread held in registers (N <= 16384)
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int per = (N + 1023) / 1024;
  const int lo = min(N, t * per), hi = min(N, lo + per);
  int sv = 0, sw = 0;
  int rv_[MAXPER], rw_[MAXPER];
  const bool regs = per <= MAXPER;
  if (regs) {
    // unconditional clamped loads, all in flight at once
#pragma unroll
    for (int i = 0; i < MAXPER; ++i) {
      const int idx = min(lo + i, max(N - 1, 0));
      rv_[i] = N > 0 ? v[idx] : 0;
      rw_[i] = (N > 0 && w) ? w[idx] : 0;
    }
#pragma unroll
    for (int i = 0; i < MAXPER; ++i) {
      if (lo + i < hi) {
        sv += rv_[i];
        sw += rw_[i];
      }
    }
  } else {
    for (int i = lo; i < hi; ++i) {
      sv += v[i];
      if (w) sw += w[i];
    }
  }
  const int iv = wave_inclusive_scan(sv), iw = wave_inclusive_scan(sw);
  if (lane == 63) part[wv] = make_int2(iv, iw);
  __syncthreads();
  if (t < 64) {
    int2 x = t < 16 ? part[t] : make_int2(0, 0);
    const int a = wave_inclusive_scan(x.x), b = wave_inclusive_scan(x.y);
    if (t < 16) part[16 + t] = make_int2(a, b);   // inclusive per-wave prefixes
  }
  __syncthreads();
  const int2 before = wv > 0 ? part[16 + wv - 1] : make_int2(0, 0);
  int rv = before.x + iv - sv, rw = before.y + iw - sw;   // exclusive prefixes of this thread
  if (regs) {
#pragma unroll
    for (int i = 0; i < MAXPER; ++i) {
      if (lo + i < hi) {
        v[lo + i] = rv;
        rv += rv_[i];
        if (w) {
          w[lo + i] = rw;
          rw += rw_[i];
        }
      }
    }
  } else {
    for (int i = lo; i < hi; ++i) {
      const int c = v[i];
      v[i] = rv;
      rv += c;
      if (w) {
        const int d = w[i];
        w[i] = rw;
        rw += d;
      }
    }
  }
  const int2 total = part[16 + 15];
  __syncthreads();
  return total;
}

// One block of 1024 threads: exclusive scans over the n_keys * nblk cells.
__global__ __launch_bounds__(1024) void permute_scan_kernel(PermArgs a) {
  __shared__ int2 part[32];
  __shared__ int dsum[16];
  const int t = threadIdx.x;
  const int N = a.n_keys * a.nblk;
  const bool dedup = a.mode == ACE_ROWS_GROUP_DEDUP;
  const int2 tot = scan_cells(a.cell, dedup ? a.pcell : nullptr, N, part);
  const int U = tot.x;
  const int npairs = dedup ? tot.y : U;
  for (int q = t; q < a.n_keys; q += 1024) {
    const int first = a.nblk > 0 ? a.cell[q * a.nblk] : 0;
    const int next = (q + 1 < a.n_keys && a.nblk > 0) ? a.cell[(q + 1) * a.nblk] : U;
    a.offsets[q] = first;
    a.counts[q] = next - first;
  }
  int d = 0;
  for (int b = t; b < a.nblk; b += 1024) d += a.drops[b];
  d = wave_inclusive_scan(d);
  if ((t & 63) == 63) dsum[t >> 6] = d;
  __syncthreads();
  if (t == 0) {
    int dt = 0;
    for (int i = 0; i < 16; ++i) dt += dsum[i];
    *a.n_dropped = dt;
    a.offsets[a.n_keys] = U;
    a.row_pair[U] = npairs;
  }
}

constexpr int kFoldCells = 16384;   // largest cell table the scatter scans itself

__global__ __launch_bounds__(kThreads) void permute_scatter_kernel(PermArgs a) {
  extern __shared__ unsigned long long bits[];
  __shared__ int keys[kPairsPerBlock];
  __shared__ uint32_t masks[kPairsPerBlock];
  __shared__ int tot[kMaxKeys], pre[kMaxKeys], ptot[kMaxKeys], ppre[kMaxKeys];
  __shared__ int cbase[kMaxKeys], pbase[kMaxKeys];
  __shared__ int red[kThreads];
  const int b = blockIdx.x;
  const int k = a.k;
  const int p0 = b * a.tokens_per_block * k;
  const int np = min(a.tokens_per_block * k, a.T * k - p0);
  const bool dedup = a.mode == ACE_ROWS_GROUP_DEDUP;
  if (a.fold) {
    // per-key totals over all blocks and prefixes over the blocks before this one
    const int t = threadIdx.x;
    for (int q = t; q < a.n_keys; q += kThreads) tot[q] = pre[q] = ptot[q] = ppre[q] = 0;
    __syncthreads();
    // each thread sums a contiguous range of the key-major table (at most a
    // few keys), then adds its per-key sums with one LDS atomic per key
    const int N = a.n_keys * a.nblk;
    const int per = (N + kThreads - 1) / kThreads;
    const int lo = min(N, t * per), hi = min(N, lo + per);
    int cq = lo < hi ? lo / a.nblk : 0;
    int st = 0, sp = 0, pt = 0, pp = 0;
    auto flush = [&]() {
      if (st | sp | pt | pp) {
        atomicAdd(&tot[cq], st);
        atomicAdd(&pre[cq], sp);
        atomicAdd(&ptot[cq], pt);
        atomicAdd(&ppre[cq], pp);
      }
      st = sp = pt = pp = 0;
    };
    for (int i0 = lo; i0 < hi; i0 += 8) {
      int cv[8], pv[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {   // unconditional clamped loads, all in flight
        const int i = min(i0 + j, N - 1);
        cv[j] = a.cell[i];
        pv[j] = dedup ? a.pcell[i] : 0;
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int i = i0 + j;
        if (i < hi) {
          const int q = i / a.nblk, bb = i - q * a.nblk;
          if (q != cq) {
            flush();
            cq = q;
          }
          st += cv[j];
          pt += pv[j];
          if (bb < b) {
            sp += cv[j];
            pp += pv[j];
          }
        }
      }
    }
    flush();
    __syncthreads();
    const int q = t;   // n_keys <= kThreads
    int U, npairs;
    const int ks = block_exclusive_scan(q < a.n_keys ? tot[q] : 0, red, &U);
    const int pks = block_exclusive_scan(q < a.n_keys && dedup ? ptot[q] : 0, red, &npairs);
    if (q < a.n_keys) {
      cbase[q] = ks + pre[q];
      pbase[q] = pks + ppre[q];
      if (b == 0) {
        a.offsets[q] = ks;
        a.counts[q] = tot[q];
      }
    }
    if (b == 0) {
      int d = 0;
      for (int bb = t; bb < a.nblk; bb += kThreads) d += a.drops[bb];
      int dt;
      block_exclusive_scan(d, red, &dt);
      if (t == 0) {
        a.offsets[a.n_keys] = U;
        a.row_pair[U] = dedup ? npairs : U;
        *a.n_dropped = dt;
      }
    }
    __syncthreads();
  }
  stage_and_mark(a, p0, np, keys, masks, bits);
  for (int lp = threadIdx.x; lp < np; lp += kThreads) {
    const int q = keys[lp];
    if (q < 0) {
      a.pair_row[p0 + lp] = -1;
      continue;
    }
    const uint32_t m = masks[lp];
    if (m == 0u) continue;  // served by its token's leader slot
    const unsigned long long* kb = bits + q * kWordsPerKey;
    const int w = lp >> 6;
    int rank = __popcll(kb[w] & ((1ull << (lp & 63)) - 1ull));
    for (int i = 0; i < w; ++i) rank += __popcll(kb[i]);
    const int row = (a.fold ? cbase[q] : a.cell[q * a.nblk + b]) + rank;
    const int tok = (p0 + lp) / k;
    a.row_token[row] = tok;
    a.row_slots[row] = m;
    int pos = row;
    if (a.mode == ACE_ROWS_GROUP_DEDUP) {  // the row's first pair among the key's pairs
      const unsigned long long* pb = bits + (a.n_keys + q) * kWordsPerKey;
      int prank = __popcll(pb[w] & ((1ull << (lp & 63)) - 1ull));
      for (int i = 0; i < w; ++i) prank += __popcll(pb[i]);
      pos = (a.fold ? pbase[q] : a.pcell[q * a.nblk + b]) + prank;
    }
    a.row_pair[row] = pos;
    for (uint32_t mm = m; mm; mm &= mm - 1u) {
      const int p = tok * k + __builtin_ctz(mm);
      a.pair_row[p] = row;
      a.pair_list[pos++] = p;
    }
  }
}

}  // namespace

size_t permute_ws_bytes(int T, int k, int n_keys) {
  const int tpb = permute_tokens_per_block(k);
  const long nblk = T > 0 ? (T + tpb - 1) / tpb : 0;
  return (size_t)(2 * nblk * n_keys + nblk) * sizeof(int32_t);
}

int permute_tokens_per_block(int k) { return k > 0 ? kPairsPerBlock / k : 1; }

hipError_t launch_permute(const int32_t* ids, int T, int k, int E, const int32_t* e2g, int G,
                          int mode, int n_keys, const ace_routing* rt, void* ws,
                          hipStream_t stream) {
  PermArgs a{};
  a.ids = ids;
  a.e2g = e2g;
  a.T = T;
  a.k = k;
  a.E = E;
  a.G = G;
  a.mode = mode;
  a.n_keys = n_keys;
  a.tokens_per_block = permute_tokens_per_block(k);
  a.nblk = T > 0 ? (T + a.tokens_per_block - 1) / a.tokens_per_block : 0;
  a.cell = static_cast<int32_t*>(ws);
  a.pcell = a.cell + (size_t)a.nblk * n_keys;
  a.drops = a.pcell + (size_t)a.nblk * n_keys;
  a.counts = rt->counts;
  a.offsets = rt->offsets;
  a.row_token = rt->row_token;
  a.row_slots = rt->row_slots;
  a.pair_row = rt->pair_row;
  a.n_dropped = rt->n_dropped;
  a.row_pair = rt->row_pair;
  a.pair_list = rt->pair_list;
  const size_t lds = (size_t)n_keys * kWordsPerKey * sizeof(unsigned long long) *
                     (mode == ACE_ROWS_GROUP_DEDUP ? 2 : 1);
  a.fold = a.nblk > 0 && (long)a.nblk * n_keys <= kFoldCells;
  if (a.nblk > 0) {
    permute_count_kernel<<<a.nblk, kThreads, lds, stream>>>(a);
  }
  if (!a.fold) permute_scan_kernel<<<1, 1024, 0, stream>>>(a);
  if (a.nblk > 0) {
    permute_scatter_kernel<<<a.nblk, kThreads, lds, stream>>>(a);
  }
  return hipGetLastError();
}

}  // namespace ace
