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
//                per-token dH buffer used for dx.
//   contract  -- Hs per row (x against A), stored per key as [r][u].
//   contract  -- dH per row (gathered G against B^T), stored per key as
//                [r][u] and either as dense per-token rows (shared input) or
//                row-major for the expand below (per-pair input).
//   expand    -- per-pair input only: dx[t*k+j] += A_q^T dH_u (each row owns
//                its input row).
//   col       -- one block per output block: dB_q (64 columns of d_out) and
//                dA_q (64 columns of d_in), reducing over the key's rows in
//                128-row stages whose large operand (G or x) is staged
//                transposed in LDS (double buffered, one barrier per stage);
//                and, for shared input, dx = dHdense A as a dense GEMM over
//                K = R (token-major).
#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

constexpr int kTile = 64;   // transpose tile / column block
constexpr int kMaxJobs = kMaxKeys + 2;

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

struct WsLayout {
  size_t At, Bt, Ht, dHt, dHf, dHrow, total;
};

// Workspace regions for element size es: At [d_in][R], Bt [R][d_out],
// Ht/dHt [R][ldh] (column = row index inside the key's segment), dense dH
// [T*kslots][R] (kslots <= k), row-major dH [P][rpad].
WsLayout ws_layout(int T, int k, int d_in, int d_out, int R, int rpad, size_t es) {
  const size_t P = (size_t)T * k;
  const size_t ldh = (P + 7) & ~(size_t)7;
  WsLayout w{};
  size_t o = 0;
  w.At = o;    o += align256(es * d_in * R);
  w.Bt = o;    o += align256(es * (size_t)R * d_out);
  w.Ht = o;    o += align256(es * (size_t)R * ldh);
  w.dHt = o;   o += align256(es * (size_t)R * ldh);
  w.dHf = o;   o += align256(es * P * R);
  w.dHrow = o; o += align256(es * P * rpad);
  w.total = o;
  return w;
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
  int32_t job_start[kMaxJobs + 1];  // block ranges: job 0 = A, 1..n_keys = B_q, last = zero
  int32_t job_cols_tiles[kMaxJobs];
  KeyTable keys;
};

template <typename T>
__global__ __launch_bounds__(kThreads) void bwd_prep_kernel(PrepArgs a) {
  __shared__ T tile[kTile][kTile + 1];
  const int b = blockIdx.x;
  const int job = upper_index(a.job_start, a.n_jobs, b);
  const int tb = b - a.job_start[job];
  const int n_keys = a.keys.n_keys;
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
  const int ct = a.job_cols_tiles[job];
  const int r0 = (tb / ct) * kTile, c0 = (tb % ct) * kTile;
  for (int i = threadIdx.x; i < kTile * kTile; i += kThreads) {
    const int rr = i / kTile, cc = i % kTile;
    if (r0 + rr < rows && c0 + cc < cols) tile[rr][cc] = src[(size_t)(r0 + rr) * lds + c0 + cc];
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kTile * kTile; i += kThreads) {
    const int cc = i / kTile, rr = i % kTile;
    if (r0 + rr < rows && c0 + cc < cols) dst[(size_t)(c0 + cc) * ldd + r0 + rr] = tile[rr][cc];
  }
}

// ------------------------------------------------------------ column pass

struct BwdArgs {
  const void* x;
  const float* pair_w;
  const void* dy;
  void* dx;
  float* dA;
  float* dB;
  const int32_t* offsets;
  const int32_t* row_token;
  const uint32_t* row_slots;
  int32_t T, k, d_in, d_out, per_pair, kslots;
  long ldh;
  const void* At;
  const void* Ht;
  const void* dHt;
  const void* dHf;
  int32_t nB, nA, nX;      // column-pass item counts
  KeyTable keys;
};


template <typename T, int RB>
__global__ __launch_bounds__(kThreads) void bwd_col_kernel(BwdArgs a) {
  using F = typename Tr<T>::frag;
  constexpr int PER = Tr<T>::PER;
  constexpr int KB = Tr<T>::KB;
  constexpr int NKB = 4;                 // K-blocks per stage
  constexpr int KC = NKB * KB;           // rows per stage
  constexpr int SLD = KC + PER;          // LDS row stride (elements)
  constexpr int TPR = kTile / PER;       // staging threads per row
  constexpr int RPP = kThreads / TPR;    // rows per staging pass (= KB)
  __shared__ __attribute__((aligned(16))) T S[2][kTile * SLD];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c16 = lane & 15, g = lane >> 4;
  const int d_in = a.d_in, d_out = a.d_out, k = a.k, R = a.keys.R;
  int item = blockIdx.x;

  if (item < a.nB + a.nA) {
    const bool isB = item < a.nB;
    if (!isB) item -= a.nB;
    const int nbk = isB ? (d_out + kTile - 1) / kTile : (d_in + kTile - 1) / kTile;
    const int q = item / nbk;
    const int col0 = (item % nbk) * kTile;
    const int ncol = isB ? d_out : d_in;
    const int lo = a.offsets[q], hi = a.offsets[q + 1];
    const int r_q = a.keys.rank[q], roff = a.keys.roff[q];
    const int nrb = (r_q + 15) >> 4;
    const T* small = static_cast<const T*>(isB ? a.Ht : a.dHt);
    const T* X = static_cast<const T*>(a.x);
    const T* DY = static_cast<const T*>(a.dy);
    f32x4 acc[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int ul = threadIdx.x / TPR, cs = (threadIdx.x % TPR) * PER;
    const int cc = col0 + cs;
    const bool cok = cc < ncol;
    // staged values of one stage: NKB passes of PER columns
    float v[NKB][PER];
    auto load_stage = [&](int u0) {
#pragma unroll
      for (int ps = 0; ps < NKB; ++ps) {
#pragma unroll
        for (int e = 0; e < PER; ++e) v[ps][e] = 0.f;
        const int u = u0 + ps * RPP + ul;
        if (u < hi && cok) {
          const int tok = a.row_token[u];
          const uint32_t slots = a.row_slots[u];
          if (isB) {
            for (uint32_t mm = slots; mm; mm &= mm - 1u) {
              const int p = tok * k + __builtin_ctz(mm);
              const float w = a.pair_w ? a.pair_w[p] : 1.f;
              float f[PER];
              Tr<T>::to_f32(Tr<T>::load(DY + (size_t)p * d_out + cc), f);
#pragma unroll
              for (int e = 0; e < PER; ++e) v[ps][e] += w * f[e];
            }
          } else {
            const int xr = a.per_pair ? tok * k + __builtin_ctz(slots) : tok;
            Tr<T>::to_f32(Tr<T>::load(X + (size_t)xr * d_in + cc), v[ps]);
          }
        }
      }
    };
    int buf = 0;
    if (lo < hi) load_stage(lo);
    for (int u0 = lo; u0 < hi; u0 += KC) {
      T* Sb = S[buf];
#pragma unroll
      for (int ps = 0; ps < NKB; ++ps)
#pragma unroll
        for (int e = 0; e < PER; ++e) Sb[(cs + e) * SLD + ps * RPP + ul] = (T)v[ps][e];
      __syncthreads();
      if (u0 + KC < hi) load_stage(u0 + KC);
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        const int ubase = u0 + kb * KB;
        if (ubase >= hi) break;
        const F sf = *reinterpret_cast<const F*>(&Sb[(16 * wave + c16) * SLD + kb * KB + PER * g]);
        const int kvalid = hi - (ubase + PER * g);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          if (rb < nrb) {
            const int r = rb * 16 + c16;
            const F tf = (r < r_q)
                ? load_frag<T>(small + (size_t)(roff + r) * a.ldh + (ubase - lo) + PER * g, kvalid, true)
                : Tr<T>::zero();
            if (isB) acc[rb] = Tr<T>::mma(sf, tf, acc[rb]);   // D[n][r]
            else acc[rb] = Tr<T>::mma(tf, sf, acc[rb]);       // D[r][c]
          }
        }
      }
      buf ^= 1;
    }
    if (isB) {
      float* dst = a.dB + (size_t)d_out * roff;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        if (rb < nrb) {
          const int r = rb * 16 + c16;
#pragma unroll
          for (int vv = 0; vv < 4; ++vv) {
            const int n = col0 + 16 * wave + 4 * g + vv;
            if (r < r_q && n < d_out) dst[(size_t)n * r_q + r] = acc[rb][vv];
          }
        }
      }
    } else {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        if (rb < nrb) {
          const int c = col0 + 16 * wave + c16;
#pragma unroll
          for (int vv = 0; vv < 4; ++vv) {
            const int r = rb * 16 + 4 * g + vv;
            if (r < r_q && c < d_in) a.dA[(size_t)(roff + r) * d_in + c] = acc[rb][vv];
          }
        }
      }
    }
    return;
  }

  // ---- dx items (shared input): dx[t][c] += sum_K dHf[t][K] A^T[c][K mod R]
  item -= a.nB + a.nA;
  const int nbc = (d_in + kTile - 1) / kTile;
  const int t0 = (item / nbc) * kTile;
  const int c0 = (item % nbc) * kTile;
  const int t = t0 + 16 * wave + c16;
  const bool tok_ok = t < a.T;
  const T* At = static_cast<const T*>(a.At);
  const T* dHf = static_cast<const T*>(a.dHf);
  T* DX = static_cast<T*>(a.dx);
  const int KR = a.kslots * R;
  const bool vec = (R % PER) == 0;
  constexpr int UX = 4;
  f32x4 c[4];
#pragma unroll
  for (int ch = 0; ch < 4; ++ch) c[ch] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int kk0 = 0; kk0 < KR; kk0 += UX * KB) {
    F df[UX], wf[UX][4];
#pragma unroll
    for (int s = 0; s < UX; ++s) {
      const int kof = kk0 + s * KB + PER * g;
      df[s] = Tr<T>::zero();
      if (tok_ok && kof < KR) {
        const T* src = dHf + (size_t)t * KR + kof;
        df[s] = load_frag<T>(src, KR - kof, vec);
      }
#pragma unroll
      for (int ch = 0; ch < 4; ++ch) {
        const int cc = c0 + ch * 16 + c16;
        wf[s][ch] = Tr<T>::zero();
        if (cc < d_in && kof < KR) {
          if (vec) {
            wf[s][ch] = Tr<T>::load(At + (size_t)cc * R + (kof % R));
          } else {
#pragma unroll
            for (int e = 0; e < PER; ++e)
              if (kof + e < KR) wf[s][ch][e] = At[(size_t)cc * R + ((kof + e) % R)];
          }
        }
      }
    }
#pragma unroll
    for (int s = 0; s < UX; ++s)
#pragma unroll
      for (int ch = 0; ch < 4; ++ch) c[ch] = Tr<T>::mma(wf[s][ch], df[s], c[ch]);   // D[c][t]
  }
  if (tok_ok) {
    T* drow = DX + (size_t)t * d_in + c0 + 4 * g;
#pragma unroll
    for (int ch = 0; ch < 4; ++ch) {
      const int cc = c0 + ch * 16 + 4 * g;
      if (cc < d_in) {
        T* p = drow + ch * 16;
#pragma unroll
        for (int vv = 0; vv < 4; ++vv) p[vv] = (T)((float)p[vv] + c[ch][vv]);
      }
    }
  }
}

template <typename T>
hipError_t launch_bwd_t(const Problem& p, const void* dy, void* dx, float* dA, float* dB,
                        void* ws, hipStream_t stream) {
  const int R = p.keys.R;
  const int n_keys = p.keys.n_keys;
  const int rpad = rank_pad(p.dtype, p.r_max);
  const WsLayout L = ws_layout(p.T, p.k, p.d_in, p.d_out, R, rpad, sizeof(T));
  char* base = static_cast<char*>(ws);
  const long P = (long)p.T * p.k;
  const long ldh = (long)((((size_t)P) + 7) & ~(size_t)7);
  // kslots: rows of the dense dH buffer per token (1 when (token, key) is unique)
  const int kslots = (!p.per_pair && p.rt->mode == ACE_ROWS_GROUP_PAIRS) ? p.k : 1;

  PrepArgs pa{};
  pa.A = p.A;
  pa.B = p.B;
  pa.At = base + L.At;
  pa.Bt = base + L.Bt;
  pa.dHf = base + L.dHf;
  pa.d_in = p.d_in;
  pa.d_out = p.d_out;
  pa.R = R;
  const long dHf_bytes = p.per_pair ? 0 : (long)p.T * kslots * R * (long)sizeof(T);
  pa.dHf_vecs = (dHf_bytes + 15) / 16;   // the region is 256-byte padded
  pa.keys = p.keys;
  pa.n_jobs = n_keys + 2;
  long nb = 0;
  auto tiles = [](long x) { return (x + kTile - 1) / kTile; };
  pa.job_start[0] = 0;
  pa.job_cols_tiles[0] = (int)tiles(p.d_in);
  nb += tiles(R) * tiles(p.d_in);
  for (int q = 0; q < n_keys; ++q) {
    pa.job_start[q + 1] = (int)nb;
    pa.job_cols_tiles[q + 1] = (int)tiles(p.keys.rank[q]);
    nb += tiles(p.d_out) * tiles(p.keys.rank[q]);
  }
  pa.job_start[n_keys + 1] = (int)nb;
  pa.job_cols_tiles[n_keys + 1] = 1;
  nb += (pa.dHf_vecs + 4 * kThreads - 1) / (4 * kThreads);
  pa.job_start[n_keys + 2] = (int)nb;
  if (nb > 0) bwd_prep_kernel<T><<<(int)nb, kThreads, 0, stream>>>(pa);
  hipError_t e = hipGetLastError();
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
  // Hs = s A x, per key [r][u]
  c.src = p.x;
  c.W = p.A;
  c.ldw = p.d_in;
  c.K = p.d_in;
  c.src_mode = p.per_pair ? kSrcPerPair : kSrcShared;
  c.out_t = base + L.Ht;
  e = launch_contract(p.dtype, c, p.r_max, P, stream);
  if (e != hipSuccess) return e;
  // dH = s B^T G
  c.src = dy;
  c.W = base + L.Bt;
  c.ldw = p.d_out;
  c.K = p.d_out;
  c.src_mode = kSrcGather;
  c.pair_w = p.pair_w;
  c.out_t = base + L.dHt;
  c.out_dense = p.per_pair ? nullptr : base + L.dHf;
  c.out_row = p.per_pair ? base + L.dHrow : nullptr;
  e = launch_contract(p.dtype, c, p.r_max, P, stream);
  if (e != hipSuccess) return e;
  if (p.per_pair) {
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
    e = launch_expand(p.dtype, x, p.r_max, P, stream);
    if (e != hipSuccess) return e;
  }

  BwdArgs a{};
  a.x = p.x;
  a.pair_w = p.pair_w;
  a.dy = dy;
  a.dx = dx;
  a.dA = dA;
  a.dB = dB;
  a.offsets = p.rt->offsets;
  a.row_token = p.rt->row_token;
  a.row_slots = p.rt->row_slots;
  a.T = p.T;
  a.k = p.k;
  a.d_in = p.d_in;
  a.d_out = p.d_out;
  a.per_pair = p.per_pair;
  a.kslots = kslots;
  a.ldh = ldh;
  a.At = base + L.At;
  a.Ht = base + L.Ht;
  a.dHt = base + L.dHt;
  a.dHf = base + L.dHf;
  a.keys = p.keys;
  a.nB = n_keys * (int)tiles(p.d_out);
  a.nA = n_keys * (int)tiles(p.d_in);
  a.nX = p.per_pair ? 0 : (int)(tiles(p.T) * tiles(p.d_in));
  const int items = a.nB + a.nA + a.nX;
  if (items > 0) {
    const int rb = rank_blocks(p.r_max);
    if (rb == 2) bwd_col_kernel<T, 2><<<items, kThreads, 0, stream>>>(a);
    else if (rb == 4) bwd_col_kernel<T, 4><<<items, kThreads, 0, stream>>>(a);
    else if (rb == 8) bwd_col_kernel<T, 8><<<items, kThreads, 0, stream>>>(a);
    else bwd_col_kernel<T, 16><<<items, kThreads, 0, stream>>>(a);
  }
  return hipGetLastError();
}

}  // namespace

size_t bwd_ws_bytes(int T, int k, int d_in, int d_out, int R, int r_max) {
  return ws_layout(T, k, d_in, d_out, R, rank_pad(ACE_F32, r_max), sizeof(float)).total;
}

hipError_t launch_bwd(const Problem& p, const void* dy, void* dx, float* dA, float* dB, void* ws,
                      hipStream_t stream) {
  if (p.dtype == ACE_BF16) return launch_bwd_t<__bf16>(p, dy, dx, dA, dB, ws, stream);
  return launch_bwd_t<float>(p, dy, dx, dA, dB, ws, stream);
}

}  // namespace ace
