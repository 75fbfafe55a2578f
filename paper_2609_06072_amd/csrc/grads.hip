// Reductions of the backward over the rows of the permutation and over the
// ranks (Sec. 3.1.2 / 3.4: a shared adapter collects every routed pair of its
// group):
//   dB_q[n][r] = sum_p dY[p][n] Hw_p[r]    over the pairs p of key q, where
//                Hw_p = w_p s_q A_q xin(p) (the contraction of the row serving
//                p, times the pair's weight)
//   dA_q[r][c] = sum_u dH_u[r] x_u[c]      over the rows u of key q
//   dx[t][c]  += sum_K dHdense[t][K] A^T[c][K mod R]   (shared input only)
// In the pre-combined mode (per-pair input, output combined per token) the
// roles swap: dB_q = sum_u dY[t_u] h_u^T over the rows (h_u = the row's
// combined h) and dA_q = sum_p (w_p dH_{u(p)}) x_p^T over the pairs.
// Both weight gradients are gathered-row GEMMs: a list of rows of a large
// row-major operand L (dY or x) against a small operand S that is contiguous
// along the contraction index (Hw or dH, stored per key as [r][position]).
//
// Items are (key, chunk of <= 1024 contraction indices, 128 gradient columns,
// dB or dA), enumerated on the device from the segment offsets, so a skewed key
// is split over several blocks (chunks of one key about equally long); a key of one chunk writes its gradient
// directly, otherwise every chunk writes a partial and grad_reduce_kernel sums
// them in chunk order (deterministic).
//
// bf16 (grad_dma_kernel): every stage of 64 L rows x 128 columns and the
// matching S slice are copied global -> LDS with global_load_lds_dwordx4 (no
// register staging), two stages in LDS; the L row indices are fetched one
// stage ahead into registers (no row-index table in LDS).  L is
// kept row-major in LDS (16-byte chunks XOR-swizzled by row) and read as MFMA
// fragments along the contraction index with ds_read_b64_tr_b16: within each
// 16-lane group, lane i receives element (i & 3) of the 8-byte reads of lanes
// 4j + (i >> 2), j = 0..3.
// fp32 (grad_reg_kernel): each thread loads a 4 x 4 block of L, transposes it
// in registers and writes 16-byte vectors to LDS.
#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

constexpr int kColBlk = kGradColBlk;   // gradient columns per item
// Contraction indices per item (split-K chunk): GradArgs::split, kSplitRows
// (which bounds the item count and the partials) or kMaxSplit (the fp32
// path's LDS row-index table).
constexpr int kSplitRows = 1024;
constexpr int kMaxSplit = 2048;
constexpr int kMinSplit = 512;    // dB items of the wide single read at narrow outputs
constexpr int kMaxSplitB = 4096;  // dB items of the wide single read at wide outputs

// Item table shared by the gradient kernels.  For key q the dB contraction
// runs over bseg[q] .. bseg[q+1] and the dA contraction over aseg[q] ..
// aseg[q+1]: pairs (positions in pair order; = rows when every row serves one
// pair) and rows respectively, swapped in the pre-combined mode.  Items of q:
// nsB(q) * nbB dB items, then nsA(q) * nbA dA items,
// ns = max(1, ceil(count / split)) (split_b for the dB items).
struct GradTable {
  int bseg[kMaxKeys + 1];
  int aseg[kMaxKeys + 1];
  int istart[kMaxKeys + 1];
  int pstart[kMaxKeys + 1];   // first item of each key among the phase's items (phases 1, 2)
};

__device__ inline int n_split(int cnt, int split) { return max(1, (cnt + split - 1) / split); }

// Indices per chunk when a key's cnt indices form ns chunks: shared evenly,
// in whole 64-index stages, so that no chunk is much shorter than the others
// (at most split, so the last chunk is never empty).
__device__ inline int chunk_len(int cnt, int ns, int split) {
  return min(split, ((cnt + ns - 1) / ns + 63) & ~63);
}

// Item table for the reduce: [0, n_keys] first item of each key, then at
// kItabStride the dB chunk counts, at 2 kItabStride the dA chunk counts.
constexpr int kItabStride = kMaxKeys + 1;
constexpr int kItabInts = 3 * kItabStride;

__device__ inline void build_grad_table(const GradArgs& a, GradTable& tb, int* scan_lds) {
  const int t = threadIdx.x;
  const int n_keys = a.keys.n_keys;
  for (int i = t; i <= n_keys; i += kThreads) {
    const int o = a.offsets[i];
    const int po = a.ppos ? a.ppos[o] : o;
    tb.bseg[i] = a.combined ? o : po;
    tb.aseg[i] = a.combined ? po : o;
  }
  __syncthreads();
  int items = 0, pitems = 0;
  if (t < n_keys) {
    const int ib = n_split(tb.bseg[t + 1] - tb.bseg[t], a.split_b) * a.nbB;
    const int ia = n_split(tb.aseg[t + 1] - tb.aseg[t], a.split) * a.nbA;
    items = ib + ia;
    pitems = a.phase == 1 ? ib : ia;
  }
  int total, ptotal;
  const int ex = block_exclusive_scan(items, scan_lds, &total);
  const int pex = block_exclusive_scan(pitems, scan_lds, &ptotal);
  if (t < n_keys) {
    tb.istart[t] = ex;
    tb.pstart[t] = pex;
  }
  if (t == 0) {
    tb.istart[n_keys] = total;
    tb.pstart[n_keys] = ptotal;
  }
  if (blockIdx.x == 0 && t < n_keys) {   // for the reduce launch
    a.itab[t] = ex;
    a.itab[kItabStride + t] = n_split(tb.bseg[t + 1] - tb.bseg[t], a.split_b);
    a.itab[2 * kItabStride + t] = n_split(tb.aseg[t + 1] - tb.aseg[t], a.split);
  }
  __syncthreads();
}

struct Item {
  int q, s, cb, ns;
  bool isB;
  int kbase;   // first contraction index of the key (pair position or row)
  int k0;      // first index of the chunk, relative to kbase
  int nk;      // indices in the chunk
};

__device__ inline Item decode_item(const GradArgs& a, const GradTable& tb, int item) {
  Item it;
  const int n_keys = a.keys.n_keys;
  it.q = upper_index(tb.istart, n_keys, item);
  int local = item - tb.istart[it.q];
  const int npB = tb.bseg[it.q + 1] - tb.bseg[it.q];
  const int nsB = n_split(npB, a.split_b);
  it.isB = local < nsB * a.nbB;
  int cnt;
  if (it.isB) {
    it.s = local / a.nbB;
    it.cb = local % a.nbB;
    it.ns = nsB;
    it.kbase = tb.bseg[it.q];
    cnt = npB;
  } else {
    local -= nsB * a.nbB;
    it.s = local / a.nbA;
    it.cb = local % a.nbA;
    cnt = tb.aseg[it.q + 1] - tb.aseg[it.q];
    it.ns = n_split(cnt, a.split);
    it.kbase = tb.aseg[it.q];
  }
  const int clen = chunk_len(cnt, it.ns, it.isB ? a.split_b : a.split);
  it.k0 = it.s * clen;
  it.nk = max(0, min(cnt - it.k0, clen));
  return it;
}

// Global index of the i-th item of phase 1 (the dB items of every key) or
// phase 2 (the dA items).
__device__ inline int phase_item(const GradArgs& a, const GradTable& tb, int i) {
  const int q = upper_index(tb.pstart, a.keys.n_keys, i);
  const int local = i - tb.pstart[q];
  if (a.phase == 1) return tb.istart[q] + local;
  return tb.istart[q] + n_split(tb.bseg[q + 1] - tb.bseg[q], a.split_b) * a.nbB + local;
}

// Row of the large operand for contraction index kabs of an item.
__device__ inline int l_row(const GradArgs& a, bool isB, int kabs) {
  if (a.combined) return isB ? a.row_token[kabs] : a.plist[kabs];
  if (isB) {
    if (a.plist) return a.plist[kabs];
    return a.row_token[kabs] * a.k + (__builtin_ctz(a.row_slots[kabs] | 0x80000000u) & 31);
  }
  const int tok = a.row_token[kabs];
  return a.per_pair ? tok * a.k + (__builtin_ctz(a.row_slots[kabs] | 0x80000000u) & 31) : tok;
}

// Loads the chunk's L row indices into idx[0 .. split) (clamped to the
// chunk's last index; unused when the chunk is empty).
template <int MPT>
__device__ inline void load_chunk_rows_n(const GradArgs& a, const Item& it, int* idx) {
  int v[MPT];
#pragma unroll
  for (int i = 0; i < MPT; ++i) {
    const int kabs = it.kbase + it.k0 + min((int)threadIdx.x + i * kThreads, it.nk - 1);
    v[i] = l_row(a, it.isB, kabs);
  }
#pragma unroll
  for (int i = 0; i < MPT; ++i) idx[threadIdx.x + i * kThreads] = v[i];
}

__device__ inline void load_chunk_rows(const GradArgs& a, const Item& it, int* idx) {
  if (it.nk <= 0) return;
  if ((it.isB ? a.split_b : a.split) > kSplitRows) load_chunk_rows_n<kMaxSplit / kThreads>(a, it, idx);
  else load_chunk_rows_n<kSplitRows / kThreads>(a, it, idx);
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

template <int RB>
__device__ inline void finish_item(const GradArgs& a, const Item& it, int item,
                                   const f32x4 (&acc)[2][RB]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nrb = (a.keys.rank[it.q] + 15) >> 4;
  if (it.ns == 1) {
#pragma unroll
    for (int cbi = 0; cbi < 2; ++cbi)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        if (rb < nrb) store_grad(a, it.isB, it.q, it.cb * kColBlk, wave, cbi, rb, lane, acc[cbi][rb]);
  } else {
    f32x4* part = reinterpret_cast<f32x4*>(a.part) + (size_t)item * (4 * 2 * RB * 64);
#pragma unroll
    for (int cbi = 0; cbi < 2; ++cbi)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)   // rank blocks past r_q are never read
        if (rb < nrb) part[((wave * 2 + cbi) * RB + rb) * 64 + lane] = acc[cbi][rb];
  }
}

// ----------------------------------------------------------------- bf16 path

typedef __attribute__((ext_vector_type(4))) short s16x4;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

template <int RB>
struct DmaGeo {
  static constexpr int RS = 64;                     // contraction indices per stage
  // stages in LDS: two (one in flight while the other is contracted); the
  // smaller footprint fits more blocks per CU, which hides more of the gather
  // latency than a third stage per block did
  static constexpr int NBUF = 2;
  static constexpr int LBYTES = RS * 256;           // 64 rows x 128 bf16
  static constexpr int SROWS = 16 * RB;             // rank rows of the S slice
  static constexpr int SBYTES = SROWS * RS * 2;     // rank rows x 64 bf16
  static constexpr int NL = 4;                      // L copies per wave per stage
  static constexpr int NS = RB / 2;                 // S copies per wave per stage
};

// 16-byte chunk position of chunk c of L row r (0..63) inside the LDS row:
// spreads the 16 rows that one transposed read touches over the banks.
__device__ inline int l_swz(int r) { return 2 * ((r & 3) | (((r >> 3) & 1) << 2)); }

template <int RB>
struct DmaSmem {
  __attribute__((aligned(16))) char L[DmaGeo<RB>::NBUF][DmaGeo<RB>::LBYTES];
  __attribute__((aligned(16))) char S[DmaGeo<RB>::NBUF][DmaGeo<RB>::SBYTES];
  GradTable tb;
  int scan[kThreads / 64];
};

// Where the L row of a contraction index comes from: src0[kabs], or, when
// slots is set, src0[kabs] * k + (first slot of src1[kabs]) (a row's first
// pair).  src1 aliases src0 when it is not needed (the load is then unused).
struct RowSrc {
  const int32_t* src0;
  const uint32_t* src1;
  bool slots;
};

template <bool ISB>
__device__ inline RowSrc row_src(const GradArgs& a) {
  RowSrc r;
  if (a.combined) {   // dB rows: dY of the row's token; dA rows: x of the pair
    r.src0 = ISB ? a.row_token : a.plist;
    r.slots = false;
  } else if (ISB && a.plist) {
    r.src0 = a.plist;
    r.slots = false;
  } else {
    r.src0 = a.row_token;
    r.slots = ISB || a.per_pair;
  }
  r.src1 = r.slots ? a.row_slots : reinterpret_cast<const uint32_t*>(r.src0);
  return r;
}

template <int RB, bool ISB, bool DH>
__device__ __forceinline__ void dma_item(const GradArgs& a, DmaSmem<RB>& sm, const Item& it,
                                         int item) {
  using G = DmaGeo<RB>;
  constexpr int RS = G::RS, NBUF = G::NBUF;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform, scalar
  const int c16 = lane & 15, g = lane >> 4;
  const int q = it.q;
  const int r_q = a.keys.rank[q], roff = a.keys.roff[q];
  const __bf16* L = static_cast<const __bf16*>(ISB ? a.dy : a.x);
  const int ldl = ISB ? a.d_out : a.d_in;
  const __bf16* S = static_cast<const __bf16*>(ISB ? a.Hw : a.dHt);
  const int col0 = it.cb * kColBlk;
  const int nst = (it.nk + RS - 1) / RS;

  __syncthreads();  // the previous item is done with the buffers

  const int lrow_in = lane >> 4;   // row inside a 4-row copy
  const int lpos = lane & 15;      // 16-byte position in the LDS row
  const int srow_in = lane >> 3;   // rank row inside an 8-row copy
  const int spos = lane & 7;
  // rows that this launch reads for the last time are copied with the
  // non-temporal policy: dY (its other reader, the dH contraction, runs
  // before) and per-pair x; shared x rows are gathered again by other keys
  const bool l_last = ISB || a.per_pair;   // block-uniform
  // Wave w copies stage rows 16w .. 16w+15.  Lane j of the wave loads the row
  // metadata of stage row 16w + (j & 15) one stage ahead (two loads, kept raw
  // across the stage so that nothing waits on them early); the row itself is
  // formed when the copies are issued and handed to the lanes that copy it by
  // shuffles.  No row-index table in LDS.
  const RowSrc rs = row_src<ISB>(a);
  const int kfirst = it.kbase + it.k0;
  int raw0 = 0;
  uint32_t raw1 = 0u;
  auto fetch = [&](int st) {
    const int kabs = kfirst + min(st * RS + 16 * wave + (lane & 15), it.nk - 1);
    raw0 = rs.src0[kabs];
    raw1 = rs.src1[kabs];
  };
  auto issue = [&](int st) {
    const int b = st % NBUF;
    const int myrow = rs.slots ? raw0 * a.k + (__builtin_ctz(raw1 | 0x80000000u) & 31) : raw0;
    int rows[G::NL];
#pragma unroll
    for (int i = 0; i < G::NL; ++i) rows[i] = __shfl(myrow, 4 * i + lrow_in, 64);
    if (st + 1 < nst) fetch(st + 1);   // block-uniform
#pragma unroll
    for (int i = 0; i < G::NL; ++i) {
      const int r0 = 16 * wave + 4 * i;
      const int r = r0 + lrow_in;                       // row of the stage
      const int row = rows[i];
      const int c = lpos ^ l_swz(r);                    // chunk this lane copies
      const int col = min(col0 + 8 * c, ldl - 8);
      const uint32_t ldst = __builtin_amdgcn_readfirstlane(lds_addr(&sm.L[b][r0 * 256]));
      if (l_last) dma16_nt(L + (size_t)row * ldl + col, ldst);
      else dma16(L + (size_t)row * ldl + col, ldst);
    }
#pragma unroll
    for (int i = 0; i < G::NS; ++i) {
      const int rr0 = 8 * (wave * G::NS + i);
      const int rr = rr0 + srow_in;                     // rank row of the slice
      const int c = spos ^ (rr & 7);
      const long col = min((long)it.k0 + st * RS + 8 * c, a.ldh - 8);
      dma16(S + (size_t)(roff + min(rr, r_q - 1)) * a.ldh + col,
            __builtin_amdgcn_readfirstlane(lds_addr(&sm.S[b][rr0 * RS * 2])));
    }
  };

  f32x4 acc[2][RB];
#pragma unroll
  for (int cbi = 0; cbi < 2; ++cbi)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc[cbi][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
  // phase 1: B_q^T fragments of the block's columns (rank c16 < 16, columns
  // col0 + 32 kb + 8 g; zero past r_q and past d_out)
  bf16x8 bfr[4];
  if constexpr (DH) {
    const __bf16* Btp = static_cast<const __bf16*>(a.Bt) + (size_t)(roff + min(c16, r_q - 1)) * a.d_out;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const int c = col0 + 32 * kb + 8 * g;
      bfr[kb] = Tr<__bf16>::load(Btp + min(c, a.d_out - 8));
      if (c >= a.d_out || c16 >= r_q) bfr[kb] = Tr<__bf16>::zero();
    }
  }

  static_assert(NBUF == 2, "the row metadata is fetched one stage ahead");
  if (nst > 0) {
    fetch(0);
    issue(0);
  }
  // K-block kb of stage st (buffer b); the ragged form zeroes the
  // contraction indices past the chunk
  auto kblock = [&](int st, int b, int kb, bool ragged) {
    const int kk = st * RS + kb * 32;   // chunk-relative index of the K-block
    const int nv = it.nk - (kk + 8 * g);
    bf16x8 sf[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int rr = 16 * rb + c16;
      const int pos = (kb * 4 + g) ^ (rr & 7);
      bf16x8 f = *reinterpret_cast<const bf16x8*>(&sm.S[b][rr * RS * 2 + pos * 16]);
      if (ragged) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (e >= nv) f[e] = (__bf16)0.f;
      }
      sf[rb] = f;
    }
#pragma unroll
    for (int cbi = 0; cbi < 2; ++cbi) {
      const int n0 = 32 * wave + 16 * cbi;
      s16x4 h2[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int r = kb * 32 + 8 * g + 4 * h + (c16 >> 2);
        const int c = (n0 >> 3) + ((c16 & 3) >> 1);
        const int off = r * 256 + ((c ^ l_swz(r)) << 4) + ((c16 & 1) << 3);
        h2[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)&sm.L[b][off]);
      }
      const bf16x8 lf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(h2[0], h2[1], 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        if (ISB) acc[cbi][rb] = Tr<__bf16>::mma(lf, sf[rb], acc[cbi][rb]);   // D[n][r]
        else acc[cbi][rb] = Tr<__bf16>::mma(sf[rb], lf, acc[cbi][rb]);       // D[r][c]
      }
    }
  };
  // the stage's pairs against B_q^T over the block's 128 columns: wave w
  // takes stage rows 16w .. 16w+15 (row c16 per lane), D[rank][pair]
  auto dh_part = [&](int st, int b) {
    const int r = 16 * wave + c16;
    f32x4 h = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const int c = kb * 4 + g;
      const bf16x8 lf = *reinterpret_cast<const bf16x8*>(&sm.L[b][r * 256 + ((c ^ l_swz(r)) << 4)]);
      h = Tr<__bf16>::mma(bfr[kb], lf, h);
    }
    const int kk = st * RS + r;   // chunk index of this lane's pair (rows past nk are copies)
    if (kk < it.nk && 4 * g < a.dhs) {
      const long pos = (long)it.kbase + it.k0 + kk;
      *reinterpret_cast<f32x4*>(a.dHp + ((size_t)it.cb * a.npos + pos) * a.dhs + 4 * g) = h;
    }
  };
  // this wave's copies of stage st (and the row metadata of stage st + 1)
  // are done; the barrier then publishes every wave's copies
  auto begin_stage = [&](int st) {
    wait_vmcnt<0>();
    __syncthreads();
    if (st + NBUF - 1 < nst) issue(st + NBUF - 1);
  };
  // full stages: no test around the matrix work; then the last, partial one
  const int nst_full = it.nk / RS;
  for (int st = 0; st < nst_full; ++st) {
    begin_stage(st);
    const int b = st % NBUF;
#pragma unroll
    for (int kb = 0; kb < RS / 32; ++kb) kblock(st, b, kb, false);
    if constexpr (DH) dh_part(st, b);
  }
  if (nst_full < nst) {   // block-uniform
    const int st = nst_full;
    begin_stage(st);
    const int b = st % NBUF;
#pragma unroll
    for (int kb = 0; kb < RS / 32; ++kb) {
      const int kk = st * RS + kb * 32;
      if (kk < it.nk) kblock(st, b, kb, kk + 32 > it.nk);
    }
    if constexpr (DH) dh_part(st, b);
  }
  finish_item<RB>(a, it, item, acc);
}

template <int RB>
__global__ __launch_bounds__(kThreads, RB <= 4 ? 3 : 1) void grad_dma_kernel(GradArgs a) {
  __shared__ DmaSmem<RB> sm;
  build_grad_table(a, sm.tb, sm.scan);
  const int n_keys = a.keys.n_keys;
  const int total = a.phase == 0 ? sm.tb.istart[n_keys] : sm.tb.pstart[n_keys];
  for (int i = blockIdx.x; i < total; i += gridDim.x) {
    const int item = a.phase == 0 ? i : phase_item(a, sm.tb, i);
    const Item it = decode_item(a, sm.tb, item);
    if (it.isB) {
      if (a.phase == 1) dma_item<RB, true, true>(a, sm, it, item);
      else dma_item<RB, true, false>(a, sm, it, item);
    } else {
      dma_item<RB, false, false>(a, sm, it, item);
    }
  }
}

// ------------------------------------------- wide dB items with dH partials
// Shared input at ranks 33..64 with wide outputs (bf16): dY is read once per
// call.  A dB item takes 512 dY columns (four 128-column sub-tiles, each laid
// out like the L tile above) of a chunk of the key's pairs; from the same
// stage in LDS it also contracts every pair's 512 columns against B_q^T into
// an fp32 dH partial per pair position and 512-column block, laid out pair
// by pair ([npos][nbW][64]: a row's partials are one contiguous run), which
// dh_reduce_wide sums per row.  The dH contraction over all of d_out before
// the weight gradients, and its second read of dY, are not run.
// Eight waves in two roles: waves 0-3 accumulate dB of one 128-column
// sub-tile each for all 64 ranks; waves 4-7 compute dH, each for two rank
// blocks and two pair blocks of every stage, with their B_q^T fragments over
// the item's 512 columns held in registers for the whole item (so every dY
// fragment a dH wave reads from LDS feeds two rank blocks).  The dB results
// go out in the layout of the four 128-column items they cover (direct
// stores or split partials), so the split reduce after the dA items is the
// usual one.
constexpr int kWideWaves = 8;
constexpr int kWideThreads = 64 * kWideWaves;

struct WideGeo {
  static constexpr int RB = 4;                          // ranks up to 64
  static constexpr int RS = 64;                         // pairs per stage
  static constexpr int SUB = kWideCols / kColBlk;       // 128-column sub-tiles
  static constexpr int SUBBYTES = RS * 256;             // 64 rows x 128 bf16
  static constexpr int LBYTES = SUB * SUBBYTES;         // 64 KB
  static constexpr int SROWS = 16 * RB;                 // rank rows of the Hw slice
  static constexpr int SBYTES = SROWS * RS * 2;         // 8 KB
  static constexpr int NL = SUB * RS / 4 / kWideWaves;  // 4-row dY copies per wave and stage
  static_assert(SROWS == 8 * kWideWaves, "one 8-row Hw copy per wave and stage");
  static_assert(NL == 2 * SUB, "wave w copies stage rows 8w .. 8w+7 of every sub-tile");
};

struct WideSmem {
  __attribute__((aligned(16))) char L[2][WideGeo::LBYTES];
  __attribute__((aligned(16))) char S[2][WideGeo::SBYTES];
  GradTable tb;                 // the 128-column items (partial positions, chunks)
  int wstart[kMaxKeys + 1];     // first wide item of each key
  int scan[kWideWaves];
};

__device__ __forceinline__ void wide_item(const GradArgs& a, WideSmem& sm, int q, int s, int cbw,
                                          int ns, int k0, int nk) {
  using G = WideGeo;
  constexpr int RB = G::RB, RS = G::RS, SUB = G::SUB;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c16 = lane & 15, g = lane >> 4;
  const int r_q = a.keys.rank[q], roff = a.keys.roff[q];
  const int kbase = sm.tb.bseg[q];
  const __bf16* L = static_cast<const __bf16*>(a.dy);
  const int ldl = a.d_out;
  const __bf16* S = static_cast<const __bf16*>(a.Hw);
  const int col0 = cbw * kWideCols;
  const int nst = (nk + RS - 1) / RS;

  __syncthreads();  // the previous item is done with the buffers

  const int lrow_in = lane >> 4;   // row inside a 4-row copy
  const int lpos = lane & 15;      // 16-byte position in the sub-tile row
  const int srow_in = lane >> 3;   // rank row inside the 8-row Hw copy
  const int spos = lane & 7;
  // Lane j of wave w loads the row metadata of stage row 8w + (j & 7) one
  // stage ahead; the copying lanes get their rows by shuffles.
  const RowSrc rs = row_src<true>(a);
  const int kfirst = kbase + k0;
  int raw0 = 0;
  uint32_t raw1 = 0u;
  auto fetch = [&](int st) {
    const int kabs = kfirst + min(st * RS + 8 * wave + (lane & 7), nk - 1);
    raw0 = rs.src0[kabs];
    raw1 = rs.src1[kabs];
  };
  auto issue = [&](int st) {
    const int b = st & 1;
    const int myrow = rs.slots ? raw0 * a.k + (__builtin_ctz(raw1 | 0x80000000u) & 31) : raw0;
    int rows[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) rows[h] = __shfl(myrow, 4 * h + lrow_in, 64);
    if (st + 1 < nst) fetch(st + 1);   // block-uniform
#pragma unroll
    for (int i = 0; i < G::NL; ++i) {
      const int sub = i >> 1, h = i & 1;
      const int r0 = 8 * wave + 4 * h;
      const int r = r0 + lrow_in;                       // row of the stage
      const int c = lpos ^ l_swz(r);                    // chunk this lane copies
      const int col = min(col0 + kColBlk * sub + 8 * c, ldl - 8);
      dma16_nt(L + (size_t)rows[h] * ldl + col,
               __builtin_amdgcn_readfirstlane(lds_addr(&sm.L[b][sub * G::SUBBYTES + r0 * 256])));
    }
    const int rr0 = 8 * wave;
    const int rr = rr0 + srow_in;                       // rank row of the slice
    const int c = spos ^ (rr & 7);
    const long col = min((long)k0 + st * RS + 8 * c, a.ldh - 8);
    dma16(S + (size_t)(roff + min(rr, r_q - 1)) * a.ldh + col,
          __builtin_amdgcn_readfirstlane(lds_addr(&sm.S[b][rr0 * RS * 2])));
  };

  if (nst > 0) {
    fetch(0);
    issue(0);
  }
  // this wave's copies of stage st (and the row metadata of stage st + 1)
  // are done; the barrier then publishes every wave's copies
  auto begin_stage = [&](int st) {
    wait_vmcnt<0>();
    __syncthreads();
    if (st + 1 < nst) issue(st + 1);
  };
  const int nst_full = nk / RS;

  if (wave < kWideWaves / 2) {
    // ---- dB waves: wave d accumulates the item's sub-tile d (128 columns)
    // for all ranks, D[n][r]
    const int sub_b = wave;
    f32x4 acc[8][RB];
#pragma unroll
    for (int cbi = 0; cbi < 8; ++cbi)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) acc[cbi][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
    // K-block kb of stage st (buffer b); the ragged form zeroes the pairs
    // past the chunk
    auto kblock = [&](int st, int b, int kb, bool ragged) {
      const int nv = nk - (st * RS + kb * 32 + 8 * g);
      bf16x8 sf[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int rr = 16 * rb + c16;
        const int pos = (kb * 4 + g) ^ (rr & 7);
        bf16x8 f = *reinterpret_cast<const bf16x8*>(&sm.S[b][rr * RS * 2 + pos * 16]);
        if (ragged) {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (e >= nv) f[e] = (__bf16)0.f;
        }
        sf[rb] = f;
      }
      const char* Lb = &sm.L[b][sub_b * G::SUBBYTES];
#pragma unroll
      for (int cbi = 0; cbi < 8; ++cbi) {
        const int n0 = 16 * cbi;
        s16x4 h2[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int r = kb * 32 + 8 * g + 4 * h + (c16 >> 2);
          const int c = (n0 >> 3) + ((c16 & 3) >> 1);
          const int off = r * 256 + ((c ^ l_swz(r)) << 4) + ((c16 & 1) << 3);
          h2[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(Lb + off));
        }
        const bf16x8 lf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(h2[0], h2[1], 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) acc[cbi][rb] = Tr<__bf16>::mma(lf, sf[rb], acc[cbi][rb]);
      }
    };
    for (int st = 0; st < nst_full; ++st) {
      begin_stage(st);
#pragma unroll
      for (int kb = 0; kb < RS / 32; ++kb) kblock(st, st & 1, kb, false);
    }
    if (nst_full < nst) {   // block-uniform: the last, partial stage
      const int st = nst_full;
      begin_stage(st);
#pragma unroll
      for (int kb = 0; kb < RS / 32; ++kb) {
        const int kk = st * RS + kb * 32;
        if (kk < nk) kblock(st, st & 1, kb, kk + 32 > nk);
      }
    }
    // columns 16 cbi of the 128-column item (q, s, 4 cbw + d), i.e. its wave
    // cbi / 2, block cbi % 2
    const int cb = SUB * cbw + sub_b;
    if (cb >= a.nbB) return;   // wave-uniform: a sub-tile past d_out
    const int nrb = (r_q + 15) >> 4;
    if (ns == 1) {
#pragma unroll
      for (int cbi = 0; cbi < 8; ++cbi)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          if (rb < nrb) store_grad(a, true, q, cb * kColBlk, cbi >> 1, cbi & 1, rb, lane, acc[cbi][rb]);
    } else {
      const int item = sm.tb.istart[q] + s * a.nbB + cb;
      f32x4* part = reinterpret_cast<f32x4*>(a.part) + (size_t)item * (4 * 2 * RB * 64);
#pragma unroll
      for (int cbi = 0; cbi < 8; ++cbi)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          if (rb < nrb) part[(cbi * RB + rb) * 64 + lane] = acc[cbi][rb];
    }
  } else {
    // ---- dH waves: wave 4 + h takes rank blocks 2 (h & 1) and 2 (h & 1) + 1
    // and pair blocks h >> 1 and (h >> 1) + 2 of every stage, so that each
    // dY fragment read from LDS feeds two rank blocks; B_q^T fragments of its
    // two rank blocks over the item's columns (zero past r_q and past d_out)
    // stay in registers for the whole item.  D[rank][pair], stored per
    // pair position.
    const int h = wave - kWideWaves / 2;
    const int rb0 = 2 * (h & 1), pb0 = h >> 1;
    const int nbW = (a.d_out + kWideCols - 1) / kWideCols;
    const bool live0 = 16 * rb0 < r_q, live1 = 16 * (rb0 + 1) < r_q;   // wave-uniform
    bf16x8 bt[2][kWideCols / 32];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int rr = 16 * (rb0 + i) + c16;
      const __bf16* Btp = static_cast<const __bf16*>(a.Bt) + (size_t)(roff + min(rr, r_q - 1)) * a.d_out;
#pragma unroll
      for (int kb = 0; kb < kWideCols / 32; ++kb) {
        const int c = col0 + 32 * kb + 8 * g;
        bt[i][kb] = Tr<__bf16>::load(Btp + min(c, a.d_out - 8));
        if (c >= a.d_out || rr >= r_q) bt[i][kb] = Tr<__bf16>::zero();
      }
    }
    auto dh_part = [&](int st, int b) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int r = 16 * (pb0 + 2 * j) + c16;   // stage row (pair) of this lane
        f32x4 hv[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
        for (int kb = 0; kb < kWideCols / 32; ++kb) {
          const int c = (kb & 3) * 4 + g;
          const bf16x8 lf = *reinterpret_cast<const bf16x8*>(
              &sm.L[b][(kb >> 2) * G::SUBBYTES + r * 256 + ((c ^ l_swz(r)) << 4)]);
#pragma unroll
          for (int i = 0; i < 2; ++i) hv[i] = Tr<__bf16>::mma(bt[i][kb], lf, hv[i]);
        }
        const int kk = st * RS + r;   // chunk index of this lane's pair (rows past nk are copies)
        if (kk < nk) {
          float* dst = a.dHp + ((size_t)(kfirst + kk) * nbW + cbw) * (16 * RB) + 16 * rb0 + 4 * g;
          *reinterpret_cast<f32x4*>(dst) = hv[0];
          if (live1) *reinterpret_cast<f32x4*>(dst + 16) = hv[1];
        }
      }
    };
    // rank blocks at or past r_q are neither formed nor stored (the reduce
    // reads no rank at or past r_q): a key of rank 16 or 32 writes a quarter
    // or a half of the 64-rank partials
    for (int st = 0; st < nst_full; ++st) {
      begin_stage(st);
      if (live0) dh_part(st, st & 1);
    }
    if (nst_full < nst) {
      const int st = nst_full;
      begin_stage(st);
      if (live0) dh_part(st, st & 1);
    }
  }
}

__global__ __launch_bounds__(kWideThreads, 2) void grad_wide_kernel(GradArgs a) {
  __shared__ WideSmem sm;
  build_grad_table(a, sm.tb, sm.scan);
  const int n_keys = a.keys.n_keys;
  const int nbW = (a.d_out + kWideCols - 1) / kWideCols;
  {
    // wide items of key q: nsB(q) * nbW, key-major
    const int t = threadIdx.x;
    const int cnt = t < n_keys ? n_split(sm.tb.bseg[t + 1] - sm.tb.bseg[t], a.split_b) * nbW : 0;
    int total;
    const int ex = block_exclusive_scan(cnt, sm.scan, &total);
    if (t < n_keys) sm.wstart[t] = ex;
    if (t == 0) sm.wstart[n_keys] = total;
    __syncthreads();
  }
  const int total = sm.wstart[n_keys];
  for (int i = blockIdx.x; i < total; i += gridDim.x) {
    const int q = upper_index(sm.wstart, n_keys, i);
    const int local = i - sm.wstart[q];
    const int s = local / nbW, cbw = local - s * nbW;
    const int cnt = sm.tb.bseg[q + 1] - sm.tb.bseg[q];
    const int ns = n_split(cnt, a.split_b);
    const int clen = chunk_len(cnt, ns, a.split_b);
    const int k0 = s * clen;
    wide_item(a, sm, q, s, cbw, ns, k0, max(0, min(cnt - k0, clen)));
  }
}

// dH per row from the phase-1 partials.  Thread t takes row blk * (256 / nq)
// + t / nq and rank quad t % nq (nq = dhs / 4); the partials of the nbB column
// blocks are loaded NL at a time and summed in block order.
template <int NL>
__global__ __launch_bounds__(kThreads) void dh_reduce_kernel(DhReduceArgs a) {
  __shared__ int seg[kMaxKeys + 1];
  const int n_keys = a.keys.n_keys;
  for (int i = threadIdx.x; i <= n_keys; i += kThreads) seg[i] = a.offsets[i];
  __syncthreads();
  const int nq = a.dhs / 4;
  const int u = blockIdx.x * (kThreads / nq) + threadIdx.x / nq;
  const int quad = threadIdx.x % nq;
  if (u >= seg[n_keys]) return;
  const int q = upper_index(seg, n_keys, u);
  const int r_q = a.keys.rank[q], roff = a.keys.roff[q], R = a.keys.R;
  const int r0 = 4 * quad;
  const int p0 = a.ppos ? a.ppos[u] : u, p1 = a.ppos ? a.ppos[u + 1] : u + 1;
  const int tok = a.row_token[u];
  const float s = a.alpha / (float)r_q;
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  if (r0 < r_q) {
    for (int p = p0; p < p1; ++p) {
      float w = 1.f;
      if (a.pair_w)
        w = a.pair_w[a.ppos ? a.plist[p] : tok * a.k + (__builtin_ctz(a.row_slots[u] | 0x80000000u) & 31)];
      f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
      const f32x4* src = reinterpret_cast<const f32x4*>(a.dHp + (size_t)p * a.dhs + r0);
      const size_t cstride = (size_t)a.npos * a.dhs / 4;
      for (int c0 = 0; c0 < a.nbB; c0 += NL) {
        f32x4 t[NL];
#pragma unroll
        for (int j = 0; j < NL; ++j) t[j] = src[(size_t)min(c0 + j, a.nbB - 1) * cstride];
#pragma unroll
        for (int j = 0; j < NL; ++j)
          if (c0 + j < a.nbB) v += t[j];
      }
      const f32x4 h = (v * s) * w;
      if (p == p0) acc = h;
      else acc += h;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (r0 + e >= r_q) acc[e] = 0.f;
  }
  const __bf16 hv[4] = {(__bf16)acc[0], (__bf16)acc[1], (__bf16)acc[2], (__bf16)acc[3]};
  if (a.dHt) {
    __bf16* dt = static_cast<__bf16*>(a.dHt);
    const long col = u - seg[q];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (r0 + e < r_q) dt[(size_t)(roff + r0 + e) * a.ldh + col] = hv[e];
  }
  if (a.dHrow) {   // zeros past r_q up to rpad
    __bf16* dr = static_cast<__bf16*>(a.dHrow) + (size_t)u * a.rpad;
#pragma unroll
    for (int e = 0; e < 4; ++e) dr[r0 + e] = hv[e];
    if (quad == 0)
      for (int r = a.dhs; r < a.rpad; ++r) dr[r] = (__bf16)0.f;
  }
  if (a.dHf) {
    const int j0 = __builtin_ctz(a.row_slots[u] | 0x80000000u) & 31;
    const size_t drow = (size_t)tok * a.kslots + (a.kslots > 1 ? j0 : 0);
    __bf16* df = static_cast<__bf16*>(a.dHf) + drow * R + roff;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (r0 + e < r_q) df[r0 + e] = hv[e];
  }
}

// dH per row from the partials of the wide items ([npos][nbW][64] fp32, so a
// row's pairs and their column blocks form one contiguous run of pieces of
// 64 ranks).  Thread t takes row blockIdx.x * kWRows + t / 16 and ranks
// 4 (t % 16) .. +3; it sums the run's pieces NL at a time (weighted per pair
// when pair weights are given).  The block's dH pass through LDS so that dHt
// ([r][u - offsets[q]] per key) is written in runs of kWRows columns.  Blocks
// of 512 threads: 256 (more, smaller blocks) and 1024 (fewer blocks resident
// per CU) measured slower at the Mixtral-like shape.
constexpr int kWThreads = 512;
constexpr int kWRows = kWThreads / 16;

template <int NL>
__global__ __launch_bounds__(kWThreads) void dh_reduce_wide_kernel(DhReduceArgs a) {
  __shared__ int seg[kMaxKeys + 1];
  __shared__ float sh[kWRows][65];
  __shared__ int sq[kWRows];
  const int n_keys = a.keys.n_keys;
  for (int i = threadIdx.x; i <= n_keys; i += kWThreads) seg[i] = a.offsets[i];
  __syncthreads();
  const int U = seg[n_keys];
  const int u0 = blockIdx.x * kWRows;
  if (u0 >= U) return;   // block-uniform
  const int lr = threadIdx.x >> 4, quad = threadIdx.x & 15;
  const int r0 = 4 * quad;
  const int nbW = a.nbB;
  const int u = u0 + lr;
  if (u < U) {
    const int q = upper_index(seg, n_keys, u);
    const int p0 = a.ppos ? a.ppos[u] : u, p1 = a.ppos ? a.ppos[u + 1] : u + 1;
    const f32x4* src = reinterpret_cast<const f32x4*>(a.dHp + (size_t)p0 * nbW * 64) + quad;
    const int r_q = a.keys.rank[q], roff = a.keys.roff[q];
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
    if (r0 >= r_q) {
      // ranks past r_q: the wide items wrote no partials there
    } else if (!a.pair_w) {
      const int n = (p1 - p0) * nbW;   // pieces of the row's run
      for (int c0 = 0; c0 < n; c0 += NL) {
        f32x4 t[NL];
#pragma unroll
        for (int j = 0; j < NL; ++j) t[j] = src[(size_t)min(c0 + j, n - 1) * 16];
#pragma unroll
        for (int j = 0; j < NL; ++j)
          if (c0 + j < n) acc += t[j];
      }
    } else {
      const int tok = a.row_token[u];
      for (int p = p0; p < p1; ++p) {
        const float w = a.pair_w[a.ppos ? a.plist[p] : tok * a.k + (__builtin_ctz(a.row_slots[u] | 0x80000000u) & 31)];
        const f32x4* sp = src + (size_t)(p - p0) * nbW * 16;
        f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int c0 = 0; c0 < nbW; c0 += NL) {
          f32x4 t[NL];
#pragma unroll
          for (int j = 0; j < NL; ++j) t[j] = sp[(size_t)min(c0 + j, nbW - 1) * 16];
#pragma unroll
          for (int j = 0; j < NL; ++j)
            if (c0 + j < nbW) v += t[j];
        }
        acc += v * w;
      }
    }
    const float s = a.alpha / (float)r_q;
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = r0 + e < r_q ? acc[e] * s : 0.f;
    const __bf16 hv[4] = {(__bf16)acc[0], (__bf16)acc[1], (__bf16)acc[2], (__bf16)acc[3]};
#pragma unroll
    for (int e = 0; e < 4; ++e) sh[lr][r0 + e] = acc[e];
    if (quad == 0) sq[lr] = q;
    if (a.dHrow) {   // zeros past r_q up to rpad
      __bf16* dr = static_cast<__bf16*>(a.dHrow) + (size_t)u * a.rpad;
#pragma unroll
      for (int e = 0; e < 4; ++e) dr[r0 + e] = hv[e];
      if (quad == 0)
        for (int r = 64; r < a.rpad; ++r) dr[r] = (__bf16)0.f;
    }
    if (a.dHf) {
      const int tok = a.row_token[u];
      const int j0 = __builtin_ctz(a.row_slots[u] | 0x80000000u) & 31;
      const size_t drow = (size_t)tok * a.kslots + (a.kslots > 1 ? j0 : 0);
      __bf16* df = static_cast<__bf16*>(a.dHf) + drow * a.keys.R + roff;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (r0 + e < r_q) df[r0 + e] = hv[e];
    }
  }
  if (!a.dHt) return;   // block-uniform
  __syncthreads();
  __bf16* dt = static_cast<__bf16*>(a.dHt);
#pragma unroll
  for (int i = 0; i < 64 * kWRows / kWThreads; ++i) {
    const int idx = threadIdx.x + i * kWThreads;
    const int r = idx / kWRows, c = idx % kWRows;
    const int uc = u0 + c;
    if (uc >= U) continue;
    const int q = sq[c];
    if (r < a.keys.rank[q])
      dt[(size_t)(a.keys.roff[q] + r) * a.ldh + (uc - seg[q])] = (__bf16)sh[c][r];
  }
}

// ----------------------------------------------------------------- fp32 path

template <typename T>
__device__ inline typename Tr<T>::frag load_masked(const T* p, int nvalid) {
  typename Tr<T>::frag f = Tr<T>::load(p);
#pragma unroll
  for (int e = 0; e < Tr<T>::PER; ++e)
    if (e >= nvalid) f[e] = (T)0.f;
  return f;
}

template <int RB>
__global__ __launch_bounds__(kThreads) void grad_reg_kernel(GradArgs a) {
  using F = f32x4;
  constexpr int PER = 4, KB = 16;
  constexpr int NKB = 4;                      // K-blocks per stage
  constexpr int RPS = NKB * KB;               // contraction indices per stage (64)
  constexpr int NI = RPS / PER;               // row groups of 4 (16)
  constexpr int NJ = kColBlk / PER;           // 16-byte column pieces (32)
  constexpr int NBLK = NI * NJ / kThreads;    // 4 x 4 blocks per thread (2)
  constexpr int TI = NI / 8;
  constexpr int SLD = RPS + PER;              // LDS stride of a transposed column
  __shared__ __attribute__((aligned(16))) float Sl[kColBlk * SLD];
  __shared__ int idx[kMaxSplit];
  __shared__ GradTable tb;
  build_grad_table(a, tb, idx);
  const int total = tb.istart[a.keys.n_keys];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int c16 = lane & 15, g = lane >> 4;
  int bi[NBLK], bj[NBLK];
#pragma unroll
  for (int x = 0; x < NBLK; ++x) {
    const int tile = wave + 4 * x;
    bi[x] = (tile % TI) * 8 + (lane & 7);
    bj[x] = (tile / TI) * 8 + (lane >> 3);
  }

  for (int item = blockIdx.x; item < total; item += gridDim.x) {
    const Item it = decode_item(a, tb, item);
    const int q = it.q;
    const int r_q = a.keys.rank[q], roff = a.keys.roff[q];
    const int nrb = (r_q + 15) >> 4;
    const float* L = static_cast<const float*>(it.isB ? a.dy : a.x);
    const int ldl = it.isB ? a.d_out : a.d_in;
    const int ncol = ldl;
    const float* S = static_cast<const float*>(it.isB ? a.Hw : a.dHt);
    const int col0 = it.cb * kColBlk;
    const long scol0 = it.k0;   // S columns count from the key's first index
    const long hmax = a.ldh - PER;
    const int nst = (it.nk + RPS - 1) / RPS;

    __syncthreads();
    load_chunk_rows(a, it, idx);
    __syncthreads();

    f32x4 acc[2][RB];
#pragma unroll
    for (int cbi = 0; cbi < 2; ++cbi)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) acc[cbi][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
    F v[NBLK][PER];
    auto load_stage = [&](int st) {
#pragma unroll
      for (int x = 0; x < NBLK; ++x) {
        const int cc = min(col0 + PER * bj[x], ncol - PER);
#pragma unroll
        for (int r = 0; r < PER; ++r) {
          const int row = idx[min(st * RPS + PER * bi[x] + r, it.nk - 1)];
          v[x][r] = *reinterpret_cast<const F*>(L + (size_t)row * ldl + cc);
        }
      }
    };
    auto write_stage = [&](int st) {
#pragma unroll
      for (int x = 0; x < NBLK; ++x) {
        const bool cok = col0 + PER * bj[x] < ncol;
#pragma unroll
        for (int e = 0; e < PER; ++e) {
          F o;
#pragma unroll
          for (int r = 0; r < PER; ++r) {
            const bool ok = cok && st * RPS + PER * bi[x] + r < it.nk;
            o[r] = ok ? v[x][r][e] : 0.f;
          }
          *reinterpret_cast<F*>(&Sl[(PER * bj[x] + e) * SLD + PER * bi[x]]) = o;
        }
      }
    };
    if (nst > 0) load_stage(0);
    for (int st = 0; st < nst; ++st) {
      write_stage(st);
      __syncthreads();
      if (st + 1 < nst) load_stage(st + 1);
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        const int ul = st * RPS + kb * KB;
        if (ul >= it.nk) break;
        const int nv = it.nk - (ul + PER * g);
        const long hc = min(scol0 + ul + PER * g, hmax);
        F tf[RB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          if (rb < nrb) {
            const int rr = min(16 * rb + c16, r_q - 1);
            tf[rb] = load_masked<float>(S + (size_t)(roff + rr) * a.ldh + hc, nv);
          }
        }
#pragma unroll
        for (int cbi = 0; cbi < 2; ++cbi) {
          const F sf = *reinterpret_cast<const F*>(&Sl[(32 * wave + 16 * cbi + c16) * SLD + kb * KB + PER * g]);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            if (rb < nrb) {
              if (it.isB) acc[cbi][rb] = Tr<float>::mma(sf, tf[rb], acc[cbi][rb]);
              else acc[cbi][rb] = Tr<float>::mma(tf[rb], sf, acc[cbi][rb]);
            }
          }
        }
      }
      __syncthreads();
    }
    finish_item<RB>(a, it, item, acc);
  }
}

// Blocks of one (key, dB|dA column block) sum its chunk partials in chunk
// order: Red::SPLIT blocks share an item's elements, two per thread, and the
// partials of eight chunks are loaded at once (clamped, masked in the sum).
template <int RB>
struct Red {
  static constexpr int PER_ITEM = 4 * 2 * RB * 64;   // f32x4 elements of a partial
  static constexpr int EPT = 2;                      // elements per thread
  static constexpr int CB = 8;                       // chunks per batch of loads
  static constexpr int SPLIT = PER_ITEM / (kThreads * EPT);
};

template <int RB>
__global__ __launch_bounds__(kThreads) void grad_reduce_kernel(GradArgs a) {
  using G = Red<RB>;
  constexpr int EPT = G::EPT, PER_ITEM = G::PER_ITEM, CB = G::CB;
  const int nb = a.nbB + a.nbA;
  const int blk = blockIdx.x / G::SPLIT, sub = blockIdx.x % G::SPLIT;
  const int q = blk / nb, rem = blk % nb;
  const bool isB = rem < a.nbB;
  const int cb = isB ? rem : rem - a.nbB;
  const int nsB = a.itab[kItabStride + q];
  const int ns = isB ? nsB : a.itab[2 * kItabStride + q];
  if (ns == 1) return;  // written directly by the gradient kernel
  const int first = a.itab[q] + (isB ? cb : nsB * a.nbB + cb);
  const size_t cstride = (size_t)(isB ? a.nbB : a.nbA) * PER_ITEM;
  const int nrb = (a.keys.rank[q] + 15) >> 4;
  const f32x4* part = reinterpret_cast<const f32x4*>(a.part) + (size_t)first * PER_ITEM;
  int e[EPT];
  bool live[EPT];
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    e[i] = (sub * EPT + i) * kThreads + threadIdx.x;
    live[i] = (e[i] >> 6) % RB < nrb;   // wave-uniform
  }
  f32x4 acc[EPT];
#pragma unroll
  for (int i = 0; i < EPT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int c0 = 0; c0 < ns; c0 += CB) {
    f32x4 v[CB][EPT];
#pragma unroll
    for (int j = 0; j < CB; ++j) {
      const size_t off = (size_t)min(c0 + j, ns - 1) * cstride;
#pragma unroll
      for (int i = 0; i < EPT; ++i) v[j][i] = live[i] ? part[off + e[i]] : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int j = 0; j < CB; ++j)
      if (c0 + j < ns) {
#pragma unroll
        for (int i = 0; i < EPT; ++i) acc[i] += v[j][i];
      }
  }
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    if (!live[i]) continue;
    const int lane = e[i] & 63, rb = (e[i] >> 6) % RB, wc = (e[i] >> 6) / RB;  // wc = wave * 2 + cbi
    store_grad(a, isB, q, cb * kColBlk, wc >> 1, wc & 1, rb, lane, acc[i]);
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

// bf16 dx GEMM with LDS staging: stages of one K-block (32 contraction
// indices) of the tile's 128 dHdense rows (64-byte row pieces) and of the
// matching rows of A itself ([R][d_in], 256-byte row pieces read transposed
// with ds_read_b64_tr_b16, so A^T is not needed), NBUF stages in LDS, all
// copied global -> LDS directly.  dHdense rows keep 16-byte chunk c at
// position c ^ ((row >> 2) & 3), so the 16 rows of one fragment read fall in
// distinct banks.
constexpr int kDxKC = 32;
constexpr int kDxNbuf = 4;
constexpr int kDxHBytes = 128 * kDxKC * 2;                // 8 KB
constexpr int kDxStage = kDxHBytes + kDxKC * kDxTile * 2;  // 8 KB + 8 KB

__global__ __launch_bounds__(kThreads) void dx_dma_kernel(DxArgs a) {
  constexpr int CST = kDxTile + 8;
  __shared__ __attribute__((aligned(16))) char smem[kDxNbuf * kDxStage];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int c16 = lane & 15, g = lane >> 4;
  const int wy = wave >> 1, wx = wave & 1;
  const int ntc = (a.d_in + kDxTile - 1) / kDxTile;
  const int t0 = (blockIdx.x / ntc) * kDxTile, c0 = (blockIdx.x % ntc) * kDxTile;
  const __bf16* H = static_cast<const __bf16*>(a.dHf);
  const __bf16* Am = static_cast<const __bf16*>(a.A);
  __bf16* DX = static_cast<__bf16*>(a.dx);
  const int KR = a.KR, R = a.R, d_in = a.d_in;
  const int nst = (KR + kDxKC - 1) / kDxKC;
  // dHdense copies: wave w copies tile rows 32w + 16i + (lane >> 2), chunk
  // position lane & 3 (global chunk (lane & 3) ^ sw(row))
  const int hpos = lane & 3, hrl = lane >> 2;
  const __bf16* hrow[2];
  int hcol[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int rl = 32 * wave + 16 * i + hrl;
    hrow[i] = H + (size_t)min(t0 + rl, a.T - 1) * KR;
    hcol[i] = 8 * (hpos ^ ((rl >> 2) & 3));
  }
  // A copies: wave w copies K rows 8w + 4i + (lane >> 4), chunk (lane & 15) ^ swizzle
  const int arow = lane >> 4, apos = lane & 15;
  int acol[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int kr = 8 * wave + 4 * i + arow;
    acol[i] = min(c0 + 8 * (apos ^ l_swz(kr)), d_in - 8);
  }
  auto issue = [&](int st) {
    char* Hs = smem + (st % kDxNbuf) * kDxStage;
    char* As = Hs + kDxHBytes;
    const int k0 = st * kDxKC;
#pragma unroll
    for (int i = 0; i < 2; ++i)
      dma16(hrow[i] + min(k0 + hcol[i], KR - 8),
            __builtin_amdgcn_readfirstlane(lds_addr(Hs + (32 * wave + 16 * i) * kDxKC * 2)));
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int kr = 8 * wave + 4 * i + arow;
      const int krow = min(k0 + kr, KR - 1) % R;
      dma16(Am + (size_t)krow * d_in + acol[i],
            __builtin_amdgcn_readfirstlane(lds_addr(As + (8 * wave + 4 * i) * kDxTile * 2)));
    }
  };
  constexpr int PER_STAGE = 4;   // copies per wave per stage
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int p = 0; p < kDxNbuf - 1; ++p)
    if (p < nst) issue(p);
  for (int st = 0; st < nst; ++st) {
    // this wave's copies of stage st are done once at most those of the
    // stages issued after it are outstanding; the barrier publishes them
    wait_vmcnt_upto<(kDxNbuf - 2) * PER_STAGE>(min(kDxNbuf - 2, nst - 1 - st) * PER_STAGE);
    __syncthreads();
    if (st + kDxNbuf - 1 < nst) issue(st + kDxNbuf - 1);
    const char* Hs = smem + (st % kDxNbuf) * kDxStage;
    const char* As = Hs + kDxHBytes;
    const int kk = st * kDxKC;
    // KR is a multiple of 8, so a lane's 8 contraction indices are all below
    // KR or all past it (those copies re-read the last valid chunk and are
    // zeroed here); only a ragged last stage has such lanes
    const bool ragged = kk + kDxKC > KR;   // block-uniform
    const bool past = kk + 8 * g >= KR;
    bf16x8 hf[4];
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      const int rl = 64 * wy + 16 * tb + c16;
      bf16x8 f = *reinterpret_cast<const bf16x8*>(Hs + rl * kDxKC * 2 + ((g ^ ((rl >> 2) & 3)) << 4));
      if (ragged && past) f = bf16x8{};
      hf[tb] = f;
    }
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const int n0 = 64 * wx + 16 * cb;
      s16x4 h2[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int r = 8 * g + 4 * h + (c16 >> 2);
        const int c = (n0 >> 3) + ((c16 & 3) >> 1);
        const int off = r * kDxTile * 2 + ((c ^ l_swz(r)) << 4) + ((c16 & 1) << 3);
        h2[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(As + off));
      }
      const bf16x8 af = __builtin_bit_cast(bf16x8, __builtin_shufflevector(h2[0], h2[1], 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) acc[cb][tb] = Tr<__bf16>::mma(af, hf[tb], acc[cb][tb]);  // D[c][t]
    }
  }
  // tile -> LDS as [t][c] (over the stage buffers), then a coalesced read-modify-write of dx
  __syncthreads();
  __bf16* Cs = reinterpret_cast<__bf16*>(smem);
#pragma unroll
  for (int cb = 0; cb < 4; ++cb)
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      __bf16* cp = &Cs[(64 * wy + 16 * tb + c16) * CST + 64 * wx + 16 * cb + 4 * g];
#pragma unroll
      for (int v = 0; v < 4; ++v) cp[v] = (__bf16)acc[cb][tb][v];
    }
  __syncthreads();
  constexpr int PPR = kDxTile / 8;
  constexpr int NP = kDxTile * PPR / kThreads;
  bf16x8 old[NP];
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int it = tid + i * kThreads;
    const int tr = it / PPR, pc = (it % PPR) * 8;
    const int t = min(t0 + tr, a.T - 1), c = min(c0 + pc, d_in - 8);
    old[i] = Tr<__bf16>::load(DX + (size_t)t * d_in + c);
  }
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int it = tid + i * kThreads;
    const int tr = it / PPR, pc = (it % PPR) * 8;
    if (t0 + tr < a.T && c0 + pc < d_in) {
      float o[8], cv[8];
      Tr<__bf16>::to_f32(old[i], o);
      Tr<__bf16>::to_f32(*reinterpret_cast<const bf16x8*>(&Cs[tr * CST + pc]), cv);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] += cv[e];
      Tr<__bf16>::store(DX + (size_t)(t0 + tr) * d_in + c0 + pc, Tr<__bf16>::from_f32(o));
    }
  }
}

// split 0 means kSplitRows, split_b 0 means split; the dA items take 1024 or
// 2048 indices, the dB items any multiple of 64 from 512 to 2048.
bool normalize_splits(GradArgs& g) {
  if (g.split == 0) g.split = kSplitRows;
  if (g.split_b == 0) g.split_b = g.split;
  return (g.split == kSplitRows || g.split == kMaxSplit) && g.split_b >= kMinSplit &&
         g.split_b <= kMaxSplitB && g.split_b % 64 == 0;
}

// Bytes of split partials (the item table follows them): bounded for the
// shortest chunks.
size_t partial_bytes(long P, int n_keys, long nb, int rb) {
  const long items = ((P + kMinSplit - 1) / kMinSplit + n_keys) * nb;
  return (size_t)items * 4 * 2 * rb * 64 * sizeof(f32x4);
}

template <int RB>
hipError_t launch_grads_rb(int dtype, GradArgs g, long P, hipStream_t stream) {
  if (g.phase != 0 && dtype != ACE_BF16) return hipErrorInvalidValue;
  if (!normalize_splits(g)) return hipErrorInvalidValue;
  const int nb = g.nbB + g.nbA;
  const int smin = g.split < g.split_b ? g.split : g.split_b;
  const long items = ((P + smin - 1) / smin + g.keys.n_keys) * nb;
  g.itab = reinterpret_cast<int32_t*>(static_cast<char*>(g.part) +
                                      partial_bytes(P, g.keys.n_keys, nb, RB));
  const long cap = 8L * device_cu_count();
  const int grid = (int)(items < cap ? items : cap);
  if (grid > 0) {
    if (dtype == ACE_BF16) {
      grad_dma_kernel<RB><<<grid, kThreads, 0, stream>>>(g);
    }
    else grad_reg_kernel<RB><<<grid, kThreads, 0, stream>>>(g);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (P > smin && g.phase != 1)   // the dB partials of phase 1 are reduced after phase 2
    grad_reduce_kernel<RB><<<g.keys.n_keys * nb * Red<RB>::SPLIT, kThreads, 0, stream>>>(g);
  return hipGetLastError();
}

}  // namespace

size_t grads_part_bytes(int T, int k, int d_in, int d_out, int n_keys, int r_max) {
  const long P = (long)T * k;
  const long nb = (d_out + kColBlk - 1) / kColBlk + (d_in + kColBlk - 1) / kColBlk;
  return partial_bytes(P, n_keys, nb, rank_blocks(r_max)) + kItabInts * sizeof(int32_t);
}

hipError_t launch_grads(int dtype, GradArgs g, int r_max, long P, hipStream_t stream) {
  g.nbB = (g.d_out + kColBlk - 1) / kColBlk;
  g.nbA = (g.d_in + kColBlk - 1) / kColBlk;
  const int rb = rank_blocks(r_max);
  if (rb == 2) return launch_grads_rb<2>(dtype, g, P, stream);
  if (rb == 4) return launch_grads_rb<4>(dtype, g, P, stream);
  if (rb == 8) return launch_grads_rb<8>(dtype, g, P, stream);
  return launch_grads_rb<16>(dtype, g, P, stream);
}

hipError_t launch_grads_wide(GradArgs g, long P, hipStream_t stream) {
  g.nbB = (g.d_out + kColBlk - 1) / kColBlk;
  g.nbA = (g.d_in + kColBlk - 1) / kColBlk;
  if (!normalize_splits(g)) return hipErrorInvalidValue;
  const int nb = g.nbB + g.nbA;
  g.itab = reinterpret_cast<int32_t*>(static_cast<char*>(g.part) +
                                      partial_bytes(P, g.keys.n_keys, nb, WideGeo::RB));
  const long nbW = (g.d_out + kWideCols - 1) / kWideCols;
  const long items = ((P + g.split_b - 1) / g.split_b + g.keys.n_keys) * nbW;
  const long cap = device_cu_count();
  const int grid = (int)(items < cap ? items : cap);
  if (grid > 0) grad_wide_kernel<<<grid, kWideThreads, 0, stream>>>(g);
  return hipGetLastError();
}

hipError_t launch_dh_reduce(const DhReduceArgs& d, long U, hipStream_t stream) {
  if (d.dhs != 8 && d.dhs != 16 && d.dhs != 64) return hipErrorInvalidValue;
  if (d.pos_major) {
    if (d.dhs != 64) return hipErrorInvalidValue;
    const long blocks = (U + kWRows - 1) / kWRows;
    if (blocks <= 0) return hipSuccess;
    // loads in flight per thread: at most a pair's column blocks
    if (d.nbB >= 16) dh_reduce_wide_kernel<8><<<(int)blocks, kWThreads, 0, stream>>>(d);
    else if (d.nbB >= 8) dh_reduce_wide_kernel<8><<<(int)blocks, kWThreads, 0, stream>>>(d);
    else dh_reduce_wide_kernel<4><<<(int)blocks, kWThreads, 0, stream>>>(d);
    return hipGetLastError();
  }
  const int rows_per_block = kThreads / (d.dhs / 4);
  const long blocks = (U + rows_per_block - 1) / rows_per_block;
  if (blocks > 0) {
    // loads in flight per thread: at most the column blocks (more would
    // re-read the last one)
    if (d.nbB >= 16) dh_reduce_kernel<16><<<(int)blocks, kThreads, 0, stream>>>(d);
    else if (d.nbB >= 8) dh_reduce_kernel<8><<<(int)blocks, kThreads, 0, stream>>>(d);
    else dh_reduce_kernel<4><<<(int)blocks, kThreads, 0, stream>>>(d);
  }
  return hipGetLastError();
}

hipError_t launch_dx_gemm(int dtype, const DxArgs& d, hipStream_t stream) {
  const int tiles = ((d.T + kDxTile - 1) / kDxTile) * ((d.d_in + kDxTile - 1) / kDxTile);
  if (tiles <= 0) return hipSuccess;
  if (dtype == ACE_BF16 && d.KR % 8 == 0) dx_dma_kernel<<<tiles, kThreads, 0, stream>>>(d);
  else if (dtype == ACE_BF16) dx_gemm_kernel<__bf16><<<tiles, kThreads, 0, stream>>>(d);
  else dx_gemm_kernel<float><<<tiles, kThreads, 0, stream>>>(d);
  return hipGetLastError();
}

}  // namespace ace
