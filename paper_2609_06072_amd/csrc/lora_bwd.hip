// Grouped LoRA backward: gradients of L = <dY, Y_out> (Sec. 3.1.2 and 3.4 --
// a shared adapter collects the gradient of every routed pair of its group).
//
// With G_u = sum_{j in slots(u)} w_j dY[t*k+j] (the row's output gradient),
// H_u = A_q x_u and s_q = alpha / r_q:
//   dH_u  = s_q B_q^T G_u                       (per row, K = d_out)
//   dB_q  = s_q sum_u G_u H_u^T                 (per key, K = rows of q)
//   dA_q  = sum_u dH_u x_u^T                    (per key, K = rows of q)
//   dx    += sum over the rows that read x      (token-major)
//
// Three launches, all deterministic (each output reduced in a fixed order):
//   prep  -- transposes of the parameters (A^T, B_q^T) into the workspace, so
//            that every MFMA operand is contiguous along its contraction
//            index, and zeroes the dense dH buffer used for dx.
//   row   -- persistent over 64-row tiles of each key's segment: recomputes
//            H, gathers G, forms dH; stores H^T and dH^T per key (for the
//            column pass) and either scatters dH into the dense per-token
//            buffer (shared input) or applies dx_u += dH_u A_q directly
//            (per-pair input: every row owns its input row).
//   col   -- one block per output block: dB_q (64 columns of d_out), dA_q (64
//            columns of d_in), both reducing over the key's rows with the
//            large operand staged transposed in LDS; and, for shared input,
//            dx = dHdense A as a dense GEMM over K = R (token-major).
#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

constexpr int kBM = 64;
constexpr int kNCH = 4;
constexpr int kTile = 64;   // transpose tile / column block
constexpr int kMaxJobs = kMaxKeys + 2;

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

struct WsLayout {
  size_t At, Bt, Ht, dHt, dHf, total;
};

// Workspace regions for element size es: At [d_in][R], Bt [R][d_out],
// Ht/dHt [R][ldh] (column = row index inside the key's segment), dense dH
// [T*kslots][R].
WsLayout ws_layout(int T, int k, int d_in, int d_out, int R, size_t es) {
  const size_t P = (size_t)T * k;
  const size_t ldh = (P + 7) & ~(size_t)7;
  WsLayout w{};
  size_t o = 0;
  w.At = o;  o += align256(es * d_in * R);
  w.Bt = o;  o += align256(es * (size_t)R * d_out);
  w.Ht = o;  o += align256(es * (size_t)R * ldh);
  w.dHt = o; o += align256(es * (size_t)R * ldh);
  w.dHf = o; o += align256(es * P * R);
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
  long dHf_elems;
  int32_t n_jobs;
  int32_t job_start[kMaxJobs + 1];  // block ranges: job 0 = A, 1..n_keys = B_q, last = zero
  int32_t job_cols_tiles[kMaxJobs];
  KeyTable keys;
};

template <typename T>
__global__ __launch_bounds__(kThreads) void bwd_prep_kernel(PrepArgs a) {
  __shared__ T tile[kTile][kTile + 1];
  const int b = blockIdx.x;
  int job = 0;
  while (job + 1 < a.n_jobs && a.job_start[job + 1] <= b) ++job;
  const int tb = b - a.job_start[job];
  const int n_keys = a.keys.n_keys;
  if (job == n_keys + 1) {  // zero the dense dH buffer
    T* d = static_cast<T*>(a.dHf);
    const long base = (long)tb * kTile * kTile;
    for (int i = threadIdx.x; i < kTile * kTile; i += kThreads) {
      const long e = base + i;
      if (e < a.dHf_elems) d[e] = (T)0.f;
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

// --------------------------------------------------------------- row pass

struct BwdArgs {
  const void* x;
  const void* A;
  const float* pair_w;
  const void* dy;
  void* dx;
  float* dA;
  float* dB;
  const int32_t* offsets;
  const int32_t* row_token;
  const uint32_t* row_slots;
  int32_t T, k, d_in, d_out, per_pair, kslots;
  float alpha;
  long ldh;
  const void* At;
  const void* Bt;
  void* Ht;
  void* dHt;
  void* dHf;
  int32_t nB, nA, nX;      // column-pass item counts
  KeyTable keys;
};

template <typename T, int RB>
__global__ __launch_bounds__(kThreads) void bwd_row_kernel(BwdArgs a) {
  using F = typename Tr<T>::frag;
  constexpr int APF = Tr<T>::ACC_PER_FRAG;
  constexpr int NM = RB / APF;
  constexpr int PER = Tr<T>::PER;
  __shared__ int seg[kMaxKeys + 1];
  __shared__ int tstart[kMaxKeys + 1];
  __shared__ int scan[kThreads];
  const int n_keys = a.keys.n_keys;
  build_tile_table(a.offsets, n_keys, kBM, seg, tstart, scan);
  const int total = tstart[n_keys];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c16 = lane & 15, g = lane >> 4;
  const T* X = static_cast<const T*>(a.x);
  const T* Aw = static_cast<const T*>(a.A);
  const T* DY = static_cast<const T*>(a.dy);
  const T* At = static_cast<const T*>(a.At);
  const T* Bt = static_cast<const T*>(a.Bt);
  T* Ht = static_cast<T*>(a.Ht);
  T* dHt = static_cast<T*>(a.dHt);
  T* dHf = static_cast<T*>(a.dHf);
  T* DX = static_cast<T*>(a.dx);
  const int d_in = a.d_in, d_out = a.d_out, k = a.k, R = a.keys.R;

  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    const int q = find_key(tstart, n_keys, tile);
    const int lo = seg[q];
    const int u_begin = lo + (tile - tstart[q]) * kBM + wave * 16;
    const int u_end = seg[q + 1];
    if (u_begin >= u_end) continue;
    const int r_q = a.keys.rank[q], roff = a.keys.roff[q];
    const int nrb = (r_q + 15) >> 4;
    const int nmb = (r_q + 16 * APF - 1) / (16 * APF);
    const int u = u_begin + c16;
    const bool valid = u < u_end;
    int tok = 0;
    uint32_t slots = 0u;
    if (valid) {
      tok = a.row_token[u];
      slots = a.row_slots[u];
    }
    const int j0 = __builtin_ctz(slots | 0x80000000u);
    const int xr = a.per_pair ? tok * k + j0 : tok;

    // ---- H (recomputed): hacc[rb][v] = H[u][16 rb + 4 g + v]
    f32x4 hacc[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) hacc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
    const T* xrow = X + (size_t)xr * d_in;
    for (int kk = 0; kk < d_in; kk += Tr<T>::KB) {
      const int kof = kk + PER * g;
      const bool kok = kof < d_in;
      const F xf = (valid && kok) ? Tr<T>::load(xrow + kof) : Tr<T>::zero();
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        if (rb < nrb) {
          const int r = rb * 16 + c16;
          const F af = (r < r_q && kok) ? Tr<T>::load(Aw + (size_t)(roff + r) * d_in + kof)
                                        : Tr<T>::zero();
          hacc[rb] = Tr<T>::mma(af, xf, hacc[rb]);
        }
      }
    }

    // ---- dH: dacc[rb][v] = (B_q^T G_u)[16 rb + 4 g + v]
    f32x4 dacc[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) dacc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int kk = 0; kk < d_out; kk += Tr<T>::KB) {
      const int n = kk + PER * g;
      const bool nok = n < d_out;
      float gs[PER];
#pragma unroll
      for (int e = 0; e < PER; ++e) gs[e] = 0.f;
      if (valid && nok) {
        for (uint32_t mm = slots; mm; mm &= mm - 1u) {
          const int p = tok * k + __builtin_ctz(mm);
          const float w = a.pair_w ? a.pair_w[p] : 1.f;
          const F v = Tr<T>::load(DY + (size_t)p * d_out + n);
#pragma unroll
          for (int e = 0; e < PER; ++e) gs[e] += w * (float)v[e];
        }
      }
      const F gf = Tr<T>::from_f32(gs);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        if (rb < nrb) {
          const int r = rb * 16 + c16;
          const F bf = (r < r_q && nok) ? Tr<T>::load(Bt + (size_t)(roff + r) * d_out + n)
                                        : Tr<T>::zero();
          dacc[rb] = Tr<T>::mma(bf, gf, dacc[rb]);
        }
      }
    }
    const float s = a.alpha / (float)r_q;

    // ---- store H^T and dH^T (key block rows, column = u - lo)
    if (valid) {
      const long col = u - lo;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        if (rb < nrb) {
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int r = rb * 16 + 4 * g + v;
            if (r < r_q) {
              Ht[(size_t)(roff + r) * a.ldh + col] = (T)hacc[rb][v];
              dHt[(size_t)(roff + r) * a.ldh + col] = (T)(s * dacc[rb][v]);
            }
          }
        }
      }
    }

    if (!a.per_pair) {
      // dense dH row of the token (one column block per key)
      if (valid) {
        const size_t drow = (size_t)tok * a.kslots + (a.kslots > 1 ? j0 : 0);
        T* dst = dHf + drow * R + roff;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          if (rb < nrb) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const int r = rb * 16 + 4 * g + v;
              if (r < r_q) dst[r] = (T)(s * dacc[rb][v]);
            }
          }
        }
      }
    } else {
      // per-pair input: dx[xr] += dH_u A_q   (C^T = A_q^T dH^T, K = r_q)
      F df[NM];
#pragma unroll
      for (int m = 0; m < NM; ++m) df[m] = Tr<T>::from_acc(dacc, m, s);
      const bool al4 = (R & 3) == 0 && (roff & 3) == 0;
      for (int c0 = 0; c0 < d_in; c0 += 16 * kNCH) {
        f32x4 c[kNCH];
#pragma unroll
        for (int ch = 0; ch < kNCH; ++ch) {
          c[ch] = f32x4{0.f, 0.f, 0.f, 0.f};
          const int cc = c0 + ch * 16 + c16;
          const bool cok = cc < d_in;
#pragma unroll
          for (int m = 0; m < NM; ++m) {
            if (m < nmb) {
              const F wf = load_acc_order<T>(At + (size_t)(cok ? cc : 0) * R + roff, r_q, m, g,
                                             cok, al4);
              c[ch] = Tr<T>::mma(wf, df[m], c[ch]);
            }
          }
        }
        if (valid) {
          T* drow = DX + (size_t)xr * d_in + c0 + 4 * g;
          f32x4 old[kNCH];
#pragma unroll
          for (int ch = 0; ch < kNCH; ++ch)
            if (c0 + ch * 16 + 4 * g < d_in) old[ch] = Tr<T>::load4(drow + ch * 16);
#pragma unroll
          for (int ch = 0; ch < kNCH; ++ch)
            if (c0 + ch * 16 + 4 * g < d_in) Tr<T>::store4(drow + ch * 16, old[ch] + c[ch]);
        }
      }
    }
  }
}

// ------------------------------------------------------------ column pass

template <typename T>
__device__ inline typename Tr<T>::frag load_frag_masked(const T* p, int nvalid) {
  // PER consecutive elements, those at index >= nvalid read as zero
  constexpr int PER = Tr<T>::PER;
  if (nvalid >= PER) return Tr<T>::load(p);
  typename Tr<T>::frag f = Tr<T>::zero();
#pragma unroll
  for (int e = 0; e < PER; ++e)
    if (e < nvalid) f[e] = p[e];
  return f;
}

template <typename T, int RB>
__global__ __launch_bounds__(kThreads) void bwd_col_kernel(BwdArgs a) {
  using F = typename Tr<T>::frag;
  constexpr int PER = Tr<T>::PER;
  constexpr int KB = Tr<T>::KB;
  constexpr int SLD = KB + PER;  // LDS row stride (elements): 80 bytes
  __shared__ __attribute__((aligned(16))) T S[kTile * SLD];
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
    // staging assignment: thread -> (row ul of the K-block, PER columns at cs)
    constexpr int TPR = kTile / PER;  // threads per staged row
    const int ul = threadIdx.x / TPR, cs = (threadIdx.x % TPR) * PER;
    for (int u0 = lo; u0 < hi; u0 += KB) {
      float v[PER];
#pragma unroll
      for (int e = 0; e < PER; ++e) v[e] = 0.f;
      const int u = u0 + ul;
      const int cc = col0 + cs;
      if (u < hi && cc < ncol) {
        const int tok = a.row_token[u];
        const uint32_t slots = a.row_slots[u];
        if (isB) {
          for (uint32_t mm = slots; mm; mm &= mm - 1u) {
            const int p = tok * k + __builtin_ctz(mm);
            const float w = a.pair_w ? a.pair_w[p] : 1.f;
            const F f = Tr<T>::load(DY + (size_t)p * d_out + cc);
#pragma unroll
            for (int e = 0; e < PER; ++e) v[e] += w * (float)f[e];
          }
        } else {
          const int xr = a.per_pair ? tok * k + __builtin_ctz(slots) : tok;
          const F f = Tr<T>::load(X + (size_t)xr * d_in + cc);
#pragma unroll
          for (int e = 0; e < PER; ++e) v[e] = (float)f[e];
        }
      }
#pragma unroll
      for (int e = 0; e < PER; ++e) S[(cs + e) * SLD + ul] = (T)v[e];
      __syncthreads();
      const F sf = *reinterpret_cast<const F*>(&S[(16 * wave + c16) * SLD + PER * g]);
      const int kvalid = hi - (u0 + PER * g);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        if (rb < nrb) {
          const int r = rb * 16 + c16;
          F tf = Tr<T>::zero();
          if (r < r_q && kvalid > 0)
            tf = load_frag_masked<T>(small + (size_t)(roff + r) * a.ldh + (u0 - lo) + PER * g,
                                     kvalid);
          if (isB) acc[rb] = Tr<T>::mma(sf, tf, acc[rb]);   // D[n][r]
          else acc[rb] = Tr<T>::mma(tf, sf, acc[rb]);       // D[r][c]
        }
      }
      __syncthreads();
    }
    if (isB) {
      const float s = a.alpha / (float)r_q;
      float* dst = a.dB + (size_t)d_out * roff;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        if (rb < nrb) {
          const int r = rb * 16 + c16;
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int n = col0 + 16 * wave + 4 * g + v;
            if (r < r_q && n < d_out) dst[(size_t)n * r_q + r] = s * acc[rb][v];
          }
        }
      }
    } else {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        if (rb < nrb) {
          const int c = col0 + 16 * wave + c16;
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int r = rb * 16 + 4 * g + v;
            if (r < r_q && c < d_in) a.dA[(size_t)(roff + r) * d_in + c] = acc[rb][v];
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
  f32x4 c[kNCH];
#pragma unroll
  for (int ch = 0; ch < kNCH; ++ch) c[ch] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int kk = 0; kk < KR; kk += KB) {
    const int kof = kk + PER * g;
    F df = Tr<T>::zero();
    if (tok_ok && kof < KR) {
      const T* src = dHf + (size_t)t * KR + kof;
      df = vec ? Tr<T>::load(src) : load_frag_masked<T>(src, KR - kof);
    }
#pragma unroll
    for (int ch = 0; ch < kNCH; ++ch) {
      const int cc = c0 + ch * 16 + c16;
      F wf = Tr<T>::zero();
      if (cc < d_in && kof < KR) {
        if (vec) {
          wf = Tr<T>::load(At + (size_t)cc * R + (kof % R));
        } else {
#pragma unroll
          for (int e = 0; e < PER; ++e)
            if (kof + e < KR) wf[e] = At[(size_t)cc * R + ((kof + e) % R)];
        }
      }
      c[ch] = Tr<T>::mma(wf, df, c[ch]);   // D[c][t]
    }
  }
  if (tok_ok) {
    T* drow = DX + (size_t)t * d_in + c0 + 4 * g;
    f32x4 old[kNCH];
#pragma unroll
    for (int ch = 0; ch < kNCH; ++ch)
      if (c0 + ch * 16 + 4 * g < d_in) old[ch] = Tr<T>::load4(drow + ch * 16);
#pragma unroll
    for (int ch = 0; ch < kNCH; ++ch)
      if (c0 + ch * 16 + 4 * g < d_in) Tr<T>::store4(drow + ch * 16, old[ch] + c[ch]);
  }
}

template <typename T, int RB>
hipError_t launch_bwd_rb(const Problem& p, BwdArgs& a, int row_grid, hipStream_t stream) {
  if (row_grid > 0) bwd_row_kernel<T, RB><<<row_grid, kThreads, 0, stream>>>(a);
  const int items = a.nB + a.nA + a.nX;
  if (items > 0) bwd_col_kernel<T, RB><<<items, kThreads, 0, stream>>>(a);
  (void)p;
  return hipGetLastError();
}

template <typename T>
hipError_t launch_bwd_t(const Problem& p, const void* dy, void* dx, float* dA, float* dB,
                        void* ws, hipStream_t stream) {
  const int R = p.keys.R;
  const int n_keys = p.keys.n_keys;
  const WsLayout L = ws_layout(p.T, p.k, p.d_in, p.d_out, R, sizeof(T));
  char* base = static_cast<char*>(ws);
  // kslots: rows of the dense dH buffer per token (1 when (token, key) is unique)
  const int kslots = (!p.per_pair && p.rt->mode == ACE_ROWS_GROUP_PAIRS) ? p.k : 1;

  // prep: A^T, B_q^T, zero the dense dH buffer
  PrepArgs pa{};
  pa.A = p.A;
  pa.B = p.B;
  pa.At = base + L.At;
  pa.Bt = base + L.Bt;
  pa.dHf = base + L.dHf;
  pa.d_in = p.d_in;
  pa.d_out = p.d_out;
  pa.R = R;
  pa.dHf_elems = p.per_pair ? 0 : (long)p.T * kslots * R;
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
  nb += (pa.dHf_elems + kTile * kTile - 1) / (kTile * kTile);
  pa.job_start[n_keys + 2] = (int)nb;
  if (nb > 0) bwd_prep_kernel<T><<<(int)nb, kThreads, 0, stream>>>(pa);

  BwdArgs a{};
  a.x = p.x;
  a.A = p.A;
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
  a.alpha = p.alpha;
  a.ldh = (long)((((size_t)p.T * p.k) + 7) & ~(size_t)7);
  a.At = base + L.At;
  a.Bt = base + L.Bt;
  a.Ht = base + L.Ht;
  a.dHt = base + L.dHt;
  a.dHf = base + L.dHf;
  a.keys = p.keys;
  a.nB = n_keys * (int)tiles(p.d_out);
  a.nA = n_keys * (int)tiles(p.d_in);
  a.nX = p.per_pair ? 0 : (int)(tiles(p.T) * tiles(p.d_in));
  const long P = (long)p.T * p.k;
  const long bound = P > 0 ? (P + kBM - 1) / kBM + n_keys : 0;
  const long cap = 4L * device_cu_count();
  const int row_grid = (int)(bound < cap ? bound : cap);
  const int rb = (p.r_max + 15) / 16;
  if (rb <= 2) return launch_bwd_rb<T, 2>(p, a, row_grid, stream);
  if (rb <= 4) return launch_bwd_rb<T, 4>(p, a, row_grid, stream);
  if (rb <= 8) return launch_bwd_rb<T, 8>(p, a, row_grid, stream);
  return launch_bwd_rb<T, 16>(p, a, row_grid, stream);
}

}  // namespace

size_t bwd_ws_bytes(int T, int k, int d_in, int d_out, int R) {
  return ws_layout(T, k, d_in, d_out, R, sizeof(float)).total;
}

hipError_t launch_bwd(const Problem& p, const void* dy, void* dx, float* dA, float* dB, void* ws,
                      hipStream_t stream) {
  if (p.dtype == ACE_BF16) return launch_bwd_t<__bf16>(p, dy, dx, dA, dB, ws, stream);
  return launch_bwd_t<float>(p, dy, dx, dA, dB, ws, stream);
}

}  // namespace ace
