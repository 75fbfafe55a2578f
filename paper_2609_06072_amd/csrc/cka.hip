// Pairwise linear CKA of the expert adapters on a shared probe set (Sec. 3.3,
// rank consolidation): the similarity that decides which experts share an
// adapter.
//
// The paper forms Z_e = X (B_e A_e)^T (N x d_out for every expert), centres
// it over the N probe rows and compares two experts with
//   s_ij = ||Zc_i^T Zc_j||_F^2 / (||Zc_i^T Zc_i||_F ||Zc_j^T Zc_j||_F).
// Centring commutes with the adapter (Zc_e = Pc_e B_e^T with Pc_e = Xc A_e^T,
// N x r), so with M = Pc^T Pc over all experts (R x R, block M_ij) and
// G_e = B_e^T B_e (r x r):
//   ||Zc_i^T Zc_j||_F^2 = tr(M_ij^T G_i M_ij G_j) = <G_i M_ij, M_ij G_j>_F,
// exact up to rounding; no N x d_out matrix is ever formed.
//
// Launches (all deterministic):
//   project -- Pt = A X^T, [R][ldp] fp32: a 128 x 128-tile MFMA GEMM over
//              K = d_in, operands staged through LDS, double buffered
//   mean    -- the probe mean of every row of Pt
//   gram    -- partial M over chunks of the probe: upper-triangle 64 x 64
//              tiles, centring on load, fp32 MFMA, one partial per chunk
//   bgram   -- G_e = B_e^T B_e
//   pairs   -- num_ij = <G_i M_ij, M_ij G_j> for i <= j (partials summed in
//              chunk order)
//   score   -- S_ij = num_ij / sqrt(num_ii num_jj); 0 when a norm is 0
#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

constexpr int kPT = 128;   // projection tile edge (probe rows and adapter rows)
constexpr int kGT = 64;    // Gram tile edge
constexpr int kGK = 1024;  // probe rows per Gram chunk (at least)

size_t a256(size_t b) { return (b + 255) & ~(size_t)255; }

struct CkaLayout {
  size_t Pt, mean, part, Gb, num, total;
  int ldp, splits, kchunk;
};

CkaLayout cka_layout(int N, int E, int r) {
  CkaLayout L{};
  const size_t R = (size_t)E * r;
  L.ldp = ((N > 0 ? N : 1) + 15) & ~15;
  // chunks of the probe for the Gram: at least kGK rows each, at most 16
  // chunks, and at most 256 MB of partials
  int splits = (N + kGK - 1) / kGK;
  const size_t cap = (size_t)(256u << 20) / (R * R * 4 > 0 ? R * R * 4 : 1);
  if ((size_t)splits > cap) splits = (int)cap;
  if (splits > 16) splits = 16;
  if (splits < 1) splits = 1;
  L.splits = splits;
  L.kchunk = (((N + splits - 1) / splits) + 15) & ~15;
  size_t o = 0;
  L.Pt = o;   o += a256(R * L.ldp * 4);
  L.mean = o; o += a256(R * 4);
  L.part = o; o += a256((size_t)splits * R * R * 4);
  L.Gb = o;   o += a256((size_t)E * r * r * 4);
  L.num = o;  o += a256((size_t)E * E * 4);
  L.total = o;
  return L;
}

struct CkaArgs {
  const void* X;     // [N][d_in]
  const void* A;     // [R][d_in]
  const void* B;     // expert e: [d_out][r] at d_out * r * e
  float* Pt;         // [R][ldp]
  float* mean;       // [R]
  float* part;       // [splits][R][R]
  float* Gb;         // [E][r][r]
  float* num;        // [E][E]
  float* S;          // [E][E]
  int32_t N, d_in, d_out, E, r, R, ldp, splits, kchunk;
};

// Upper-triangle index p -> (a, b), a <= b < n, row-major.
__device__ inline void upper_pair(int p, int n, int* a, int* b) {
  int i = 0;
  while (p >= n - i) {
    p -= n - i;
    ++i;
  }
  *a = i;
  *b = i + p;
}

// ---------------------------------------------------------------- project

template <typename T>
__global__ __launch_bounds__(kThreads) void cka_project_kernel(CkaArgs a) {
  using F = typename Tr<T>::frag;
  constexpr int PER = Tr<T>::PER, KB = Tr<T>::KB;
  constexpr int RS = KB + PER;  // LDS row stride in elements (80 bytes: conflict-free fragments)
  __shared__ __attribute__((aligned(16))) T xs[2][kPT * RS];
  __shared__ __attribute__((aligned(16))) T as[2][kPT * RS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c16 = lane & 15, g = lane >> 4;
  const int n0 = blockIdx.x * kPT, c0 = blockIdx.y * kPT;
  const int wn = (wave & 1) * 64, wc = (wave >> 1) * 64;
  const T* X = static_cast<const T*>(a.X);
  const T* A = static_cast<const T*>(a.A);
  const int N = a.N, R = a.R, d_in = a.d_in;

  // a stage is KB contraction indices (64 bytes) of 128 rows of each operand:
  // 512 16-byte pieces per operand, two per thread
  F xr[2], ar[2];
  auto load_stage = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int id = tid + kThreads * i, row = id >> 2, kk = k0 + (id & 3) * PER;
      const bool ok = kk < d_in;  // d_in is a multiple of PER: a piece is wholly in or out
      const F xv = Tr<T>::load(X + (size_t)min(n0 + row, N - 1) * d_in + (ok ? kk : 0));
      const F av = Tr<T>::load(A + (size_t)min(c0 + row, R - 1) * d_in + (ok ? kk : 0));
      xr[i] = ok ? xv : Tr<T>::zero();
      ar[i] = ok ? av : Tr<T>::zero();
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int id = tid + kThreads * i, row = id >> 2, ch = id & 3;
      *reinterpret_cast<F*>(&xs[buf][row * RS + ch * PER]) = xr[i];
      *reinterpret_cast<F*>(&as[buf][row * RS + ch * PER]) = ar[i];
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  load_stage(0);
  store_stage(0);
  __syncthreads();
  int buf = 0;
  for (int k0 = 0; k0 < d_in; k0 += KB) {
    const bool more = k0 + KB < d_in;
    if (more) load_stage(k0 + KB);
    F xf[4], af[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      xf[j] = *reinterpret_cast<const F*>(&xs[buf][(wn + 16 * j + c16) * RS + g * PER]);
      af[j] = *reinterpret_cast<const F*>(&as[buf][(wc + 16 * j + c16) * RS + g * PER]);
    }
#pragma unroll
    for (int jn = 0; jn < 4; ++jn)
#pragma unroll
      for (int jc = 0; jc < 4; ++jc) acc[jn][jc] = Tr<T>::mma(xf[jn], af[jc], acc[jn][jc]);
    if (more) store_stage(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }
  // acc[jn][jc] element v = P[n][c] with n = n0+wn+16jn+4g+v, c = c0+wc+16jc+c16:
  // four consecutive probe rows of Pt row c per lane
#pragma unroll
  for (int jn = 0; jn < 4; ++jn)
#pragma unroll
    for (int jc = 0; jc < 4; ++jc) {
      const int c = c0 + wc + 16 * jc + c16, n = n0 + wn + 16 * jn + 4 * g;
      if (c < R && n < N) {
        float* dst = a.Pt + (size_t)c * a.ldp + n;
        if (n + 3 < N) {
          *reinterpret_cast<f32x4*>(dst) = acc[jn][jc];
        } else {
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (n + v < N) dst[v] = acc[jn][jc][v];
        }
      }
    }
}

// ---------------------------------------------------------------- mean

__global__ __launch_bounds__(kThreads) void cka_mean_kernel(CkaArgs a) {
  __shared__ float red[kThreads];
  const float* row = a.Pt + (size_t)blockIdx.x * a.ldp;
  float s = 0.f;
  for (int n = threadIdx.x; n < a.N; n += kThreads) s += row[n];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = kThreads / 2; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) a.mean[blockIdx.x] = a.N > 0 ? red[0] / (float)a.N : 0.f;
}

// ---------------------------------------------------------------- gram

// Block (tile pair p, chunk s): the 64 x 64 tile (ta, tb), ta <= tb, of
// sum over the chunk's probe rows of (Pt[a][n] - mean[a]) (Pt[b][n] - mean[b]).
// Wave w owns a 32 x 32 quarter; fragments are 16-byte loads of Pt rows.
__global__ __launch_bounds__(kThreads) void cka_gram_kernel(CkaArgs a) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c16 = lane & 15, g = lane >> 4;
  const int R = a.R;
  const int nt = (R + kGT - 1) / kGT;
  int ta, tb;
  upper_pair(blockIdx.x, nt, &ta, &tb);
  const int s = blockIdx.y;
  const int abase = ta * kGT + (wave & 1) * 32, bbase = tb * kGT + (wave >> 1) * 32;
  const int k_beg = s * a.kchunk, k_end = min(a.N, k_beg + a.kchunk);
  const float* pa[2];
  const float* pb[2];
  float ma[2], mb[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int ra = min(abase + 16 * j + c16, R - 1), rb = min(bbase + 16 * j + c16, R - 1);
    pa[j] = a.Pt + (size_t)ra * a.ldp;
    pb[j] = a.Pt + (size_t)rb * a.ldp;
    ma[j] = a.mean[ra];
    mb[j] = a.mean[rb];
  }
  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  constexpr int U = 4;  // 16-row steps loaded ahead of their MFMAs
  for (int k = k_beg; k < k_end; k += 16 * U) {
    f32x4 fa[U][2], fb[U][2];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      // rows past k_end (the chunk end, <= ldp) are read but masked below;
      // starts are multiples of 16 and ldp is too, so a fragment never
      // crosses the end of its Pt row
      const int kk = min(k + 16 * u, a.ldp - 16) + 4 * g;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        fa[u][j] = *reinterpret_cast<const f32x4*>(pa[j] + kk);
        fb[u][j] = *reinterpret_cast<const f32x4*>(pb[j] + kk);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kk = k + 16 * u + 4 * g;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bool ok = kk + e < k_end;
          fa[u][j][e] = ok ? fa[u][j][e] - ma[j] : 0.f;
          fb[u][j][e] = ok ? fb[u][j][e] - mb[j] : 0.f;
        }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = Tr<float>::mma(fa[u][i], fb[u][j], acc[i][j]);
    }
  }
  float* out = a.part + (size_t)s * R * R;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = bbase + 16 * j + c16;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = abase + 16 * i + 4 * g + v;
        if (row < R && col < R) out[(size_t)row * R + col] = acc[i][j][v];
      }
    }
}

// ---------------------------------------------------------------- B^T B

template <typename T>
__global__ __launch_bounds__(kThreads) void cka_bgram_kernel(CkaArgs a) {
  constexpr int CH = 64;                 // rows of B_e staged per step
  __shared__ float bs[CH * 64];
  const int e = blockIdx.x, r = a.r, rr = r * r;
  const T* B = static_cast<const T*>(a.B) + (size_t)a.d_out * r * e;
  float acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;
  for (int o0 = 0; o0 < a.d_out; o0 += CH) {
    const int rows = min(CH, a.d_out - o0);
    __syncthreads();
    for (int i = threadIdx.x; i < rows * r; i += kThreads) bs[i] = (float)B[(size_t)o0 * r + i];
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int pq = threadIdx.x + kThreads * i;
      if (pq < rr) {
        const int p = pq / r, q = pq % r;
        float s = acc[i];
        for (int o = 0; o < rows; ++o) s += bs[o * r + p] * bs[o * r + q];
        acc[i] = s;
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int pq = threadIdx.x + kThreads * i;
    if (pq < rr) a.Gb[(size_t)e * rr + pq] = acc[i];
  }
}

// ---------------------------------------------------------------- pairs

// Block per expert pair i <= j: M_ij (partials summed in chunk order, read
// from the upper triangle of the symmetric M), then <G_i M_ij, M_ij G_j>.
__global__ __launch_bounds__(kThreads) void cka_pairs_kernel(CkaArgs a) {
  __shared__ float Gi[64 * 64], Gj[64 * 64], Mij[64 * 64];
  __shared__ float red[kThreads];
  int i, j;
  upper_pair(blockIdx.x, a.E, &i, &j);
  const int r = a.r, rr = r * r, R = a.R;
  for (int t = threadIdx.x; t < rr; t += kThreads) {
    Gi[t] = a.Gb[(size_t)i * rr + t];
    Gj[t] = a.Gb[(size_t)j * rr + t];
    const int row = i * r + t / r, col = j * r + t % r;
    const size_t off = (size_t)min(row, col) * R + max(row, col);
    float m = 0.f;
    for (int s = 0; s < a.splits; ++s) m += a.part[(size_t)s * R * R + off];
    Mij[t] = m;
  }
  __syncthreads();
  float acc = 0.f;
  for (int t = threadIdx.x; t < rr; t += kThreads) {
    const int p = t / r, q = t % r;
    float t1 = 0.f, t2 = 0.f;
    for (int u = 0; u < r; ++u) {
      t1 += Gi[p * r + u] * Mij[u * r + q];   // (G_i M_ij)[p][q]
      t2 += Mij[p * r + u] * Gj[u * r + q];   // (M_ij G_j)[p][q]
    }
    acc += t1 * t2;
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int w = kThreads / 2; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    a.num[(size_t)i * a.E + j] = red[0];
    a.num[(size_t)j * a.E + i] = red[0];
  }
}

__global__ __launch_bounds__(kThreads) void cka_score_kernel(CkaArgs a) {
  const int t = blockIdx.x * kThreads + threadIdx.x;
  const int E = a.E;
  if (t >= E * E) return;
  const int i = t / E, j = t % E;
  const float den = sqrtf(a.num[(size_t)i * E + i]) * sqrtf(a.num[(size_t)j * E + j]);
  const float v = den > 0.f ? a.num[t] / den : 0.f;
  a.S[t] = isfinite(v) ? v : 0.f;
}

template <typename T>
hipError_t launch_cka_t(const CkaProblem& p, void* ws, hipStream_t stream) {
  const CkaLayout L = cka_layout(p.N, p.E, p.r);
  char* base = static_cast<char*>(ws);
  CkaArgs a{};
  a.X = p.X;
  a.A = p.A;
  a.B = p.B;
  a.Pt = reinterpret_cast<float*>(base + L.Pt);
  a.mean = reinterpret_cast<float*>(base + L.mean);
  a.part = reinterpret_cast<float*>(base + L.part);
  a.Gb = reinterpret_cast<float*>(base + L.Gb);
  a.num = reinterpret_cast<float*>(base + L.num);
  a.S = p.S;
  a.N = p.N;
  a.d_in = p.d_in;
  a.d_out = p.d_out;
  a.E = p.E;
  a.r = p.r;
  a.R = p.E * p.r;
  a.ldp = L.ldp;
  a.splits = L.splits;
  a.kchunk = L.kchunk;
  const int R = a.R;
  if (p.N > 0) {
    dim3 grid((p.N + kPT - 1) / kPT, (R + kPT - 1) / kPT);
    cka_project_kernel<T><<<grid, kThreads, 0, stream>>>(a);
  }
  cka_mean_kernel<<<R, kThreads, 0, stream>>>(a);
  {
    const int nt = (R + kGT - 1) / kGT;
    dim3 grid(nt * (nt + 1) / 2, L.splits);
    cka_gram_kernel<<<grid, kThreads, 0, stream>>>(a);
  }
  cka_bgram_kernel<T><<<p.E, kThreads, 0, stream>>>(a);
  cka_pairs_kernel<<<p.E * (p.E + 1) / 2, kThreads, 0, stream>>>(a);
  cka_score_kernel<<<(p.E * p.E + kThreads - 1) / kThreads, kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace

size_t cka_ws_bytes(int N, int E, int r) { return cka_layout(N, E, r).total; }

hipError_t launch_cka(const CkaProblem& p, void* ws, hipStream_t stream) {
  if (p.dtype == ACE_BF16) return launch_cka_t<__bf16>(p, ws, stream);
  return launch_cka_t<float>(p, ws, stream);
}

}  // namespace ace
