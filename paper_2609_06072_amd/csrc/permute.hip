// Route expansion and permutation (Sec. 3.5: the active group set A(x) of each
// token, one row per (token, active group); or one row per routed pair for the
// expert-wise and "shared adapter, per-pair" modes).
//
// A stable counting sort of the emitted rows by key, in two or three launches:
//   count   -- each block owns a chunk of whole tokens (<= 256 pairs).  The
//              block's keys go to LDS; each emitted row sets the bit of its
//              local pair index in a per-key bitmap (LDS, ds_or_b64), and the
//              per-(key, block) population counts are written key-major.
//   scan    -- one block per routing: exclusive scan of the key-major counts
//              gives each (key, block) its first row; counts/offsets/n_dropped
//              written.  Only for large cell tables: otherwise every scatter
//              block derives the bases of its own cells from the count table
//              (per-key totals and prefixes, exact integer sums) and block 0
//              writes counts/offsets/n_dropped.
//   scatter -- rebuilds the bitmap; a row's rank inside its (key, block) cell
//              is the popcount of the lower bits, so rows come out sorted by
//              (key, token, slot) with no atomics on rows and no sort.
// Pair positions (the routed pairs in (key, token, slot) order) follow the
// same scheme: in ACE_ROWS_GROUP_DEDUP mode a second bitmap marks every pair
// of a key and second cell table is scanned; in the other modes a row is a
// pair and its position is its row.
//
// One launch sequence can write two routings of the same top-k ids (a
// group-keyed one and the expert-keyed one, as a layer with grouped gate/up
// and expert-wise down projections needs): each routing is a pass with
// bitmaps and cell tables of its own, and the blocks of both passes run side
// by side in each launch (block i serves pass i / nblk, token chunk
// i % nblk).
#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

constexpr int kPairsPerBlock = 256;   // == kThreads: one pair per thread
constexpr int kWordsPerKey = kPairsPerBlock / 64;
// Largest cell tables (counts, plus pair counts in ACE_ROWS_GROUP_DEDUP mode)
// the scatter folds itself: 32 KiB of LDS as 16-bit counts.
constexpr int kFoldCells = 16384;

struct PermPass {
  int32_t mode, n_keys;
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

struct PermArgs {
  const int32_t* ids;
  const int32_t* e2g;  // null unless a pass is group-keyed
  int32_t T, k, E, G;
  int32_t tokens_per_block, nblk, npass;
  int32_t nwords;      // 64-bit words of bitmaps (the largest pass's)
  PermPass pass[kMaxPermPasses];
};

__host__ __device__ inline int pass_words(int mode, int n_keys) {
  return n_keys * kWordsPerKey * (mode == ACE_ROWS_GROUP_DEDUP ? 2 : 1);
}

// Pass i with a constant index for each branch (no dynamic indexing of the
// kernel argument block).
__device__ inline const PermPass& pass_of(const PermArgs& a, int i) {
  return i == 0 ? a.pass[0] : a.pass[kMaxPermPasses - 1];
}

// The block's expert ids (one pair per thread; -1 when out of [0, E)) and the
// map e -> g(e) (-1 when out of [0, G)), loaded together, plus cleared bitmaps.
struct Staged {
  int e, g;
};

__device__ inline Staged issue_ids(const PermArgs& a, int p0, int np) {
  const int t = threadIdx.x;
  Staged s;
  s.e = t < np ? a.ids[p0 + t] : -1;
  s.g = (a.e2g && t < a.E) ? a.e2g[t] : -1;
  return s;
}

__device__ inline void store_ids(const PermArgs& a, Staged s, int* eid, int* gmap,
                                 unsigned long long* bits) {
  const int t = threadIdx.x;
  for (int i = t; i < a.nwords; i += kThreads) bits[i] = 0ull;
  eid[t] = (s.e >= 0 && s.e < a.E) ? s.e : -1;
  gmap[t] = (s.g >= 0 && s.g < a.G) ? s.g : -1;
  __syncthreads();
}

// Keys of the block's pairs for pass P (-1 = dropped) and the emitted rows
// marked in the pass's per-key bitmaps (in ACE_ROWS_GROUP_DEDUP mode a second
// bitmap right after the first marks every pair).  Returns 1 when this
// thread's pair is dropped.
__device__ inline int mark_pass(const PermArgs& a, const PermPass& P, int np, const int* eid,
                                const int* gmap, int* keys, uint32_t* masks,
                                unsigned long long* bits) {
  const int t = threadIdx.x;
  const bool dedup = P.mode == ACE_ROWS_GROUP_DEDUP;
  int q = -1;
  if (t < np) {
    const int e = eid[t];
    q = e < 0 ? -1 : (P.mode == ACE_ROWS_EXPERT ? e : gmap[e]);
    // the routed experts of a token form a set: an id already listed at a
    // lower slot of the same token drops this pair
    const int j = t % a.k, tb = t - j;
    for (int jj = 0; jj < j; ++jj)
      if (eid[tb + jj] == e) q = -1;
    keys[t] = q;
  }
  __syncthreads();
  if (t < np) {
    if (q < 0) {
      masks[t] = 0u;
    } else {
      const int k = a.k;
      uint32_t m = 1u << (t % k);
      bool emit = true;
      if (dedup) {
        // leader = first slot of the token with this group; mask = all of them
        const int j = t % k, tb = t - j;
        for (int jj = 0; jj < k; ++jj) {
          if (keys[tb + jj] != q) continue;
          if (jj < j) { emit = false; break; }
          m |= 1u << jj;
        }
      }
      masks[t] = emit ? m : 0u;
      if (emit) atomicOr(&bits[q * kWordsPerKey + (t >> 6)], 1ull << (t & 63));
      if (dedup) atomicOr(&bits[(P.n_keys + q) * kWordsPerKey + (t >> 6)], 1ull << (t & 63));
    }
  }
  __syncthreads();
  return (t < np && q < 0) ? 1 : 0;
}

__global__ __launch_bounds__(kThreads) void permute_count_kernel(PermArgs a) {
  extern __shared__ unsigned long long bits[];  // the pass's bitmaps
  __shared__ int eid[kPairsPerBlock];
  __shared__ int gmap[kMaxKeys];
  __shared__ int keys[kPairsPerBlock];
  __shared__ uint32_t masks[kPairsPerBlock];
  __shared__ int red[kThreads];
  const int ps = blockIdx.x / a.nblk, b = blockIdx.x % a.nblk;
  const PermPass& P = pass_of(a, ps);
  const int p0 = b * a.tokens_per_block * a.k;
  const int np = min(a.tokens_per_block * a.k, a.T * a.k - p0);
  store_ids(a, issue_ids(a, p0, np), eid, gmap, bits);
  const int d = mark_pass(a, P, np, eid, gmap, keys, masks, bits);
  const bool dedup = P.mode == ACE_ROWS_GROUP_DEDUP;
  for (int q = threadIdx.x; q < P.n_keys; q += kThreads) {
    int c = 0, pc = 0;
#pragma unroll
    for (int w = 0; w < kWordsPerKey; ++w) {
      c += __popcll(bits[q * kWordsPerKey + w]);
      if (dedup) pc += __popcll(bits[(P.n_keys + q) * kWordsPerKey + w]);
    }
    P.cell[q * a.nblk + b] = c;
    if (dedup) P.pcell[q * a.nblk + b] = pc;
  }
  int total;
  block_exclusive_scan(d, red, &total);
  if (threadIdx.x == 0) P.drops[b] = total;
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

// One block of 1024 threads per pass without a fold: exclusive scans over the
// pass's n_keys * nblk cells.
__global__ __launch_bounds__(1024) void permute_scan_kernel(PermArgs a) {
  __shared__ int2 part[32];
  __shared__ int dsum[16];
  const PermPass& P = pass_of(a, blockIdx.x);
  if (P.fold) return;
  const int t = threadIdx.x;
  const int N = P.n_keys * a.nblk;
  const bool dedup = P.mode == ACE_ROWS_GROUP_DEDUP;
  const int2 tot = scan_cells(P.cell, dedup ? P.pcell : nullptr, N, part);
  const int U = tot.x;
  const int npairs = dedup ? tot.y : U;
  for (int q = t; q < P.n_keys; q += 1024) {
    const int first = a.nblk > 0 ? P.cell[q * a.nblk] : 0;
    const int next = (q + 1 < P.n_keys && a.nblk > 0) ? P.cell[(q + 1) * a.nblk] : U;
    P.offsets[q] = first;
    P.counts[q] = next - first;
  }
  int d = 0;
  for (int b = t; b < a.nblk; b += 1024) d += P.drops[b];
  d = wave_inclusive_scan(d);
  if ((t & 63) == 63) dsum[t >> 6] = d;
  __syncthreads();
  if (t == 0) {
    int dt = 0;
    for (int i = 0; i < 16; ++i) dt += dsum[i];
    *P.n_dropped = dt;
    P.offsets[P.n_keys] = U;
    P.row_pair[U] = npairs;
  }
}

// Fold of pass P by scatter block b: per-key totals over all blocks and
// prefixes over the blocks before b, summed from the key-major count tables
// (exact integer sums); cbase/pbase = first row / pair position of b's cells.
// Block 0 also writes counts, offsets, n_dropped and row_pair[U].
// The tables are staged in LDS as 16-bit counts (a cell counts at most
// kPairsPerBlock rows) by coalesced loads, all in flight at once; then
// key q is summed by tpk threads of one wave (strided over the blocks) and a
// butterfly over those lanes.
__device__ inline void stage_counts(const int32_t* src, int N, uint16_t* dst) {
  constexpr int B = 32;
  const int t = threadIdx.x;
  for (int i0 = 0; i0 < N; i0 += B * kThreads) {
    int v[B];
#pragma unroll
    for (int j = 0; j < B; ++j)   // block-uniform guard; the last row clamped
      if (i0 + j * kThreads < N) v[j] = src[min(i0 + j * kThreads + t, N - 1)];
#pragma unroll
    for (int j = 0; j < B; ++j) {
      const int i = i0 + j * kThreads + t;
      if (i0 + j * kThreads < N && i < N) dst[i] = (uint16_t)v[j];
    }
  }
}

__device__ void fold_pass(const PermArgs& a, const PermPass& P, int b, uint16_t* tab,
                          int* tot, int* pre, int* ptot, int* ppre, int* cbase, int* pbase,
                          int* red) {
  const int t = threadIdx.x;
  const bool dedup = P.mode == ACE_ROWS_GROUP_DEDUP;
  const int nblk = a.nblk, n_keys = P.n_keys;
  const int N = n_keys * nblk;
  uint16_t* ptab = tab + N;
  // block 0 sums the dropped counts: loads issued with the table's
  int d = 0;
  if (b == 0)
    for (int bb = t; bb < nblk; bb += kThreads) d += P.drops[bb];
  stage_counts(P.cell, N, tab);
  if (dedup) stage_counts(P.pcell, N, ptab);
  __syncthreads();
  int tpk = 1;   // threads per key: a power of two, at most a wave
  while (tpk < 64 && 2 * tpk * n_keys <= kThreads) tpk *= 2;
  const int q = t / tpk, sub = t % tpk;
  int st = 0, sp = 0, pt = 0, pp = 0;
  if (q < n_keys) {
    for (int bb = sub; bb < nblk; bb += tpk) {
      const int c = tab[q * nblk + bb];
      const int pc = dedup ? ptab[q * nblk + bb] : 0;
      st += c;
      pt += pc;
      if (bb < b) {
        sp += c;
        pp += pc;
      }
    }
  }
  for (int o = tpk >> 1; o > 0; o >>= 1) {
    st += __shfl_xor(st, o, 64);
    sp += __shfl_xor(sp, o, 64);
    pt += __shfl_xor(pt, o, 64);
    pp += __shfl_xor(pp, o, 64);
  }
  if (sub == 0 && q < n_keys) {
    tot[q] = st;
    pre[q] = sp;
    ptot[q] = pt;
    ppre[q] = pp;
  }
  __syncthreads();
  const int kq = t;   // n_keys <= kThreads
  int U, npairs;
  const int ks = block_exclusive_scan(kq < n_keys ? tot[kq] : 0, red, &U);
  const int pks = block_exclusive_scan(kq < n_keys && dedup ? ptot[kq] : 0, red, &npairs);
  if (kq < n_keys) {
    cbase[kq] = ks + pre[kq];
    pbase[kq] = pks + ppre[kq];
    if (b == 0) {
      P.offsets[kq] = ks;
      P.counts[kq] = tot[kq];
    }
  }
  if (b == 0) {
    int dt;
    block_exclusive_scan(d, red, &dt);
    if (t == 0) {
      P.offsets[n_keys] = U;
      P.row_pair[U] = dedup ? npairs : U;
      *P.n_dropped = dt;
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(kThreads) void permute_scatter_kernel(PermArgs a) {
  extern __shared__ unsigned long long bits[];   // the pass's bitmaps, then its count tables
  __shared__ int eid[kPairsPerBlock];
  __shared__ int gmap[kMaxKeys];
  __shared__ int keys[kPairsPerBlock];
  __shared__ uint32_t masks[kPairsPerBlock];
  __shared__ int tot[kMaxKeys], pre[kMaxKeys], ptot[kMaxKeys], ppre[kMaxKeys];
  __shared__ int cbase[kMaxKeys], pbase[kMaxKeys];
  __shared__ int red[kThreads];
  const int ps = blockIdx.x / a.nblk, b = blockIdx.x % a.nblk;
  const PermPass& P = pass_of(a, ps);
  const int k = a.k;
  const int p0 = b * a.tokens_per_block * k;
  const int np = min(a.tokens_per_block * k, a.T * k - p0);
  // the ids are in flight while the cell tables are staged
  const Staged ids = issue_ids(a, p0, np);
  if (P.fold)
    fold_pass(a, P, b, reinterpret_cast<uint16_t*>(bits + a.nwords), tot, pre, ptot, ppre, cbase,
              pbase, red);
  store_ids(a, ids, eid, gmap, bits);
  mark_pass(a, P, np, eid, gmap, keys, masks, bits);
  const int lp = threadIdx.x;
  if (lp >= np) return;
  const int q = keys[lp];
  if (q < 0) {
    P.pair_row[p0 + lp] = -1;
    return;
  }
  const uint32_t m = masks[lp];
  if (m == 0u) return;  // served by its token's leader slot
  const unsigned long long* kb = bits + q * kWordsPerKey;
  const int w = lp >> 6;
  int rank = __popcll(kb[w] & ((1ull << (lp & 63)) - 1ull));
  for (int i = 0; i < w; ++i) rank += __popcll(kb[i]);
  const int row = (P.fold ? cbase[q] : P.cell[q * a.nblk + b]) + rank;
  const int tok = (p0 + lp) / k;
  P.row_token[row] = tok;
  P.row_slots[row] = m;
  int pos = row;
  if (P.mode == ACE_ROWS_GROUP_DEDUP) {  // the row's first pair among the key's pairs
    const unsigned long long* pb = bits + (P.n_keys + q) * kWordsPerKey;
    int prank = __popcll(pb[w] & ((1ull << (lp & 63)) - 1ull));
    for (int i = 0; i < w; ++i) prank += __popcll(pb[i]);
    pos = (P.fold ? pbase[q] : P.pcell[q * a.nblk + b]) + prank;
  }
  P.row_pair[row] = pos;
  for (uint32_t mm = m; mm; mm &= mm - 1u) {
    const int p = tok * k + __builtin_ctz(mm);
    P.pair_row[p] = row;
    P.pair_list[pos++] = p;
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
                          int npass, const PermuteOut* outs, hipStream_t stream) {
  if (npass < 1 || npass > kMaxPermPasses) return hipErrorInvalidValue;
  PermArgs a{};
  a.ids = ids;
  a.e2g = e2g;
  a.T = T;
  a.k = k;
  a.E = E;
  a.G = G;
  a.tokens_per_block = permute_tokens_per_block(k);
  a.nblk = T > 0 ? (T + a.tokens_per_block - 1) / a.tokens_per_block : 0;
  a.npass = npass;
  bool scan = false;
  int words = 0;          // the largest pass's bitmaps
  size_t tab_bytes = 0;   // the largest staged count tables of a folding pass
  for (int i = 0; i < npass; ++i) {
    const PermuteOut& o = outs[i];
    PermPass& P = a.pass[i];
    P.mode = o.mode;
    P.n_keys = o.n_keys;
    words = pass_words(o.mode, o.n_keys) > words ? pass_words(o.mode, o.n_keys) : words;
    P.cell = static_cast<int32_t*>(o.ws);
    P.pcell = P.cell + (size_t)a.nblk * o.n_keys;
    P.drops = P.pcell + (size_t)a.nblk * o.n_keys;
    P.counts = o.rt->counts;
    P.offsets = o.rt->offsets;
    P.row_token = o.rt->row_token;
    P.row_slots = o.rt->row_slots;
    P.pair_row = o.rt->pair_row;
    P.n_dropped = o.rt->n_dropped;
    P.row_pair = o.rt->row_pair;
    P.pair_list = o.rt->pair_list;
    P.fold = a.nblk > 0 &&
             (long)a.nblk * o.n_keys * (o.mode == ACE_ROWS_GROUP_DEDUP ? 2 : 1) <= kFoldCells;
    scan = scan || !P.fold;
    if (P.fold) {
      const size_t tb = (size_t)a.nblk * o.n_keys * sizeof(uint16_t) *
                        (o.mode == ACE_ROWS_GROUP_DEDUP ? 2 : 1);
      tab_bytes = tb > tab_bytes ? tb : tab_bytes;
    }
  }
  a.nwords = words;
  const size_t lds = (size_t)words * sizeof(unsigned long long);
  if (a.nblk > 0) permute_count_kernel<<<a.nblk * npass, kThreads, lds, stream>>>(a);
  if (scan) permute_scan_kernel<<<npass, 1024, 0, stream>>>(a);
  if (a.nblk > 0) permute_scatter_kernel<<<a.nblk * npass, kThreads, lds + tab_bytes, stream>>>(a);
  return hipGetLastError();
}

}  // namespace ace
