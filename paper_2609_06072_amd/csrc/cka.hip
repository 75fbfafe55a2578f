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
//   project -- Pt = A X^T, [R][ldp] fp32: a 64 x 256-tile MFMA GEMM over
//              K = d_in (eight waves), operands copied global -> LDS
//              directly, two stages of 128 bytes per row in LDS (128 x 256
//              tiles with two or three stages measured no faster)
//   mean    -- the probe mean of every row of Pt; bf16 inputs: also the
//              centred rows split as v = hi + lo (both bf16, |lo| <= 2^-9 |v|)
//   gram    -- partial M over chunks of the probe (at least kGK rows): upper-triangle tiles
//              (128 x 128 staged through LDS for bf16 inputs, 64 x 64 for
//              fp32), one partial per chunk.  bf16 inputs:
//              M = hi^T hi + hi^T lo + lo^T hi on the bf16 matrix cores (the
//              dropped lo^T lo is below 2^-16 of |v_a v_b|).  fp32 inputs:
//              fp32 MFMA, centring on load.
//   msum    -- M: the Gram partials summed in chunk order (elements on or
//              above the diagonal), eight chunks' loads in flight; at ranks up
//              to 8 the same launch also forms the partials of B_e^T B_e
//   bgram   -- (ranks above 8) partial G_e over chunks of 256 rows of B_e
//   pairs   -- num_ij = <G_i M_ij, M_ij G_j> for i <= j; at ranks up to 8 one
//              wave per pair, which also forms num_ii and num_jj and writes
//              S_ij directly; otherwise one block per pair, then
//   score   -- S_ij = num_ij / sqrt(num_ii num_jj); 0 when a norm is 0
#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

constexpr int kPN = 64;    // projection tile: probe rows
constexpr int kPBuf = 2;   // projection stages in LDS (80 KB: two blocks per CU)
constexpr int kPC = 256;   // projection tile: adapter rows (eight waves)
constexpr int kPThreads = 2 * kPC;
constexpr int kGT = 64;    // Gram tile edge (fp32 inputs)
constexpr int kGT2 = 128;  // Gram tile edge (bf16 inputs, staged through LDS)
constexpr int kGK = 400;   // probe rows per Gram chunk (at least)
constexpr int kGBuf = 3;   // Gram stages in LDS (bf16 inputs; 96 KB: one block per CU)
constexpr int kMaxSplits = 64;
constexpr int kBO = 256;   // rows of B_e per B^T B chunk

size_t a256(size_t b) { return (b + 255) & ~(size_t)255; }

struct CkaLayout {
  size_t Pt, mean, part, M, Gb, num, Phi, Plo, total;
  int ldp, splits, kchunk, nbo;
};

CkaLayout cka_layout(int N, int d_out, int E, int r) {
  CkaLayout L{};
  const size_t R = (size_t)E * r;
  L.ldp = ((N > 0 ? N : 1) + 31) & ~31;
  // chunks of the probe for the Gram: at least kGK rows each, at most
  // kMaxSplits chunks, and at most 256 MB of partials
  int splits = (N + kGK - 1) / kGK;
  const size_t cap = (size_t)(256u << 20) / (R * R * 4 > 0 ? R * R * 4 : 1);
  if ((size_t)splits > cap) splits = (int)cap;
  if (splits > kMaxSplits) splits = kMaxSplits;
  if (splits < 1) splits = 1;
  L.splits = splits;
  L.kchunk = (((N + splits - 1) / splits) + 31) & ~31;
  size_t o = 0;
  L.Pt = o;   o += a256(R * L.ldp * 4);
  L.mean = o; o += a256(R * 4);
  L.part = o; o += a256((size_t)splits * R * R * 4);
  L.M = o;    o += a256(R * R * 4);
  L.nbo = (d_out + kBO - 1) / kBO;
  L.Gb = o;   o += a256((size_t)E * L.nbo * r * r * 4);
  L.num = o;  o += a256((size_t)E * E * 4);
  L.Phi = o;  o += a256(R * L.ldp * 2);
  L.Plo = o;  o += a256(R * L.ldp * 2);
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
  float* M;          // [R][R], upper-triangle tiles
  float* Gb;         // [E][nbo][r][r] partials of B_e^T B_e
  float* num;        // [E][E]
  __bf16* Phi;       // [R][ldp] centred Pt split as hi + lo (bf16 inputs; zero past N)
  __bf16* Plo;
  float* S;          // [E][E]
  int32_t N, d_in, d_out, E, r, R, ldp, splits, kchunk, nbo;
  int32_t bf16;      // storage type of X, A and B
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

// A block takes PN probe rows x 256 adapter rows (eight waves, so that X is
// staged once per 256 adapter rows); wave (wn, wc) owns PN / 2 x 64.
// Stages of two K-blocks (128 bytes of every row) of both operands are
// copied global -> LDS with global_load_lds_dwordx4, NBUF stages in LDS (no
// register staging; NBUF - 1 stages in flight while one is read), so that a
// barrier is paid per 8 PN / 32 matrix instructions of a wave.  A copy
// instruction moves 8 rows; lane l lands at row l/8, position l%8 of the
// 128-byte LDS row and fetches the global 16-byte chunk (l%8) ^ sw(row),
// sw(row) = (row >> 1) & 7, so that the 16 rows one fragment read touches
// (two per 256-byte bank line) fall in distinct banks.  Chunks past d_in (a
// multiple of 16 bytes) are fetched clamped and zeroed at the read.
__device__ inline int cka_sw(int row) { return (row >> 1) & 7; }
// The same for 64-byte rows (four chunks; the Gram's stages): (row >> 2) & 3.
__device__ inline int cka_sw4(int row) { return (row >> 2) & 3; }

template <typename T, int PN, int NBUF>
__global__ __launch_bounds__(kPThreads) void cka_project_kernel(CkaArgs a) {
  using F = typename Tr<T>::frag;
  constexpr int PER = Tr<T>::PER, KB = Tr<T>::KB;   // KB * sizeof(T) = 64 bytes
  constexpr int KS = 2 * KB;                        // contraction indices per stage (128 bytes)
  constexpr int RB = 128;                           // bytes of a row per stage
  constexpr int XB = PN * RB, AB = kPC * RB;        // stage bytes of each operand
  constexpr int NW = kPThreads / 64;
  constexpr int XC = PN / 8 / NW;                   // X copies per wave and stage
  constexpr int AC = kPC / 8 / NW;                  // A copies per wave and stage
  constexpr int CP = XC + AC;
  constexpr int JN = PN / 32;                       // 16-row probe blocks per wave
  static_assert(PN % (8 * NW) == 0 && kPC == 32 * NW && NBUF >= 2 && NBUF <= 4, "copy plan");
  __shared__ __attribute__((aligned(16))) char xs[NBUF][XB];
  __shared__ __attribute__((aligned(16))) char as[NBUF][AB];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c16 = lane & 15, g = lane >> 4;
  const int n0 = blockIdx.x * PN, c0 = blockIdx.y * kPC;
  const int wn = (wave & 1) * (PN / 2), wc = (wave >> 1) * 64;   // wave: PN/2 probe rows x 64 adapter rows
  const T* X = static_cast<const T*>(a.X);
  const T* A = static_cast<const T*>(a.A);
  const int N = a.N, R = a.R, d_in = a.d_in;
  const int nst = (d_in + KS - 1) / KS;

  // copy plan: X rows 8 (XC w + i) .. +7 (XC instructions per wave), A rows
  // 32w .. 32w+31 (four); lane l copies row (l >> 3) of its instruction (a
  // chunk past d_in is fetched from column d_in - PER instead, inside the
  // row, and zeroed at the read)
  const int crow = lane >> 3, cpos = lane & 7;
  const T* xsrc[XC];
  int xch[XC];
#pragma unroll
  for (int i = 0; i < XC; ++i) {
    const int xr = 8 * (XC * wave + i) + crow;
    xsrc[i] = X + (size_t)min(n0 + xr, N - 1) * d_in;
    xch[i] = PER * (cpos ^ cka_sw(xr));
  }
  const T* asrc[AC];
  int ach[AC];
#pragma unroll
  for (int i = 0; i < AC; ++i) {
    const int ar = 32 * wave + 8 * i + crow;
    asrc[i] = A + (size_t)min(c0 + ar, R - 1) * d_in;
    ach[i] = PER * (cpos ^ cka_sw(ar));
  }
  auto issue = [&](int st) {
    const int b = st % NBUF;
    const int k0 = st * KS;
#pragma unroll
    for (int i = 0; i < XC; ++i)
      dma16(xsrc[i] + min(k0 + xch[i], d_in - PER),
            __builtin_amdgcn_readfirstlane(lds_addr(&xs[b][8 * (XC * wave + i) * RB])));
#pragma unroll
    for (int i = 0; i < AC; ++i)
      dma16(asrc[i] + min(k0 + ach[i], d_in - PER),
            __builtin_amdgcn_readfirstlane(lds_addr(&as[b][(32 * wave + 8 * i) * RB])));
  };

  f32x4 acc[JN][4];
#pragma unroll
  for (int i = 0; i < JN; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int s = 0; s < NBUF - 1; ++s)
    if (s < nst) issue(s);
  // this wave's copies of stage st are done once at most those of the stages
  // issued after it are outstanding; the barrier publishes every wave's
  // copies and tells that stage st - 1's buffer is no longer read
  auto begin_stage = [&](int st) {
    wait_vmcnt_upto<(NBUF - 2) * CP>(min(NBUF - 2, nst - 1 - st) * CP);
    __syncthreads();
    if (st + NBUF - 1 < nst) issue(st + NBUF - 1);
  };
  // fragments of K-block kb (chunks 4 kb + g) of stage st; with MASK the
  // chunks past d_in (copies of the last one) read as zero
  auto read_kb = [&](int st, int kb, bool mask, F (&xf)[JN], F (&af)[4]) {
    const int b = st % NBUF;
    const int cc = 4 * kb + g;
    const bool kin = !mask || st * KS + PER * cc < d_in;
#pragma unroll
    for (int j = 0; j < JN; ++j) {
      const int r = wn + 16 * j + c16;
      xf[j] = *reinterpret_cast<const F*>(&xs[b][r * RB + 16 * (cc ^ cka_sw(r))]);
      if (mask && !kin) xf[j] = Tr<T>::zero();
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = wc + 16 * j + c16;
      af[j] = *reinterpret_cast<const F*>(&as[b][r * RB + 16 * (cc ^ cka_sw(r))]);
      if (mask && !kin) af[j] = Tr<T>::zero();
    }
  };
  auto mma_kb = [&](const F (&xf)[JN], const F (&af)[4]) {
#pragma unroll
    for (int jn = 0; jn < JN; ++jn)
#pragma unroll
      for (int jc = 0; jc < 4; ++jc) acc[jn][jc] = Tr<T>::mma(xf[jn], af[jc], acc[jn][jc]);
  };
  // whole stages: both K-blocks' fragments are read before the matrix work,
  // with no masks (no branches around the reads)
  const int nst_full = d_in / KS;
  for (int st = 0; st < nst_full; ++st) {
    begin_stage(st);
    F x0[JN], a0[4], x1[JN], a1[4];
    read_kb(st, 0, false, x0, a0);
    read_kb(st, 1, false, x1, a1);
    mma_kb(x0, a0);
    mma_kb(x1, a1);
  }
  if (nst_full < nst) {   // the last stage reaches past d_in
    const int st = nst_full;
    begin_stage(st);
    F x0[JN], a0[4], x1[JN], a1[4];
    read_kb(st, 0, true, x0, a0);
    read_kb(st, 1, true, x1, a1);
    mma_kb(x0, a0);
    mma_kb(x1, a1);
  }
  // acc[jn][jc] element v = P[n][c] with n = n0+wn+16jn+4g+v, c = c0+wc+16jc+c16:
  // four consecutive probe rows of Pt row c per lane
#pragma unroll
  for (int jn = 0; jn < JN; ++jn)
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

// Block c: the probe mean of Pt row c; with SPLIT, also the centred row split
// as v = hi + lo in bf16 (hi = v rounded, lo = the remainder rounded), zero
// from N up to ldp, so the Gram reads ready matrix-core operands.
template <bool SPLIT>
__global__ __launch_bounds__(kThreads) void cka_mean_kernel(CkaArgs a) {
  __shared__ float red[kThreads];
  // ldp is a multiple of 32: whole 16-byte pieces, entries past N masked
  const f32x4* row = reinterpret_cast<const f32x4*>(a.Pt + (size_t)blockIdx.x * a.ldp);
  const int n4 = (a.N + 3) / 4;
  float s = 0.f;
#pragma unroll 4
  for (int i = threadIdx.x; i < n4; i += kThreads) {
    const f32x4 v = row[i];
#pragma unroll
    for (int e = 0; e < 4; ++e) s += 4 * i + e < a.N ? v[e] : 0.f;
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = kThreads / 2; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  const float mean = a.N > 0 ? red[0] / (float)a.N : 0.f;
  if (threadIdx.x == 0) a.mean[blockIdx.x] = mean;
  if constexpr (SPLIT) {
    bf16x4* hi = reinterpret_cast<bf16x4*>(a.Phi + (size_t)blockIdx.x * a.ldp);
    bf16x4* lo = reinterpret_cast<bf16x4*>(a.Plo + (size_t)blockIdx.x * a.ldp);
#pragma unroll 4
    for (int i = threadIdx.x; i < a.ldp / 4; i += kThreads) {
      const f32x4 v = row[min(i, max(n4 - 1, 0))];
      bf16x4 h, l;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float c = 4 * i + e < a.N ? v[e] - mean : 0.f;
        h[e] = (__bf16)c;
        l[e] = (__bf16)(c - (float)h[e]);
      }
      hi[i] = h;
      lo[i] = l;
    }
  }
}

// ---------------------------------------------------------------- gram

// Block (tile pair p, chunk s): the 64 x 64 tile (ta, tb), ta <= tb, of
// sum over the chunk's probe rows of (Pt[a][n] - mean[a]) (Pt[b][n] - mean[b]).
// Wave w owns a 32 x 32 quarter; fragments are read straight from the Pt rows
// (contiguous along the probe).  SPLIT: bf16 matrix cores on the hi/lo split
// (K-blocks of 32), else fp32 matrix cores (K-blocks of 16).
template <bool SPLIT>
__global__ __launch_bounds__(kThreads) void cka_gram_kernel(CkaArgs a);

// bf16 inputs: block (tile pair p, chunk s) takes the 128 x 128 tile (ta, tb)
// of M; wave (w & 1, w >> 1) owns a 64 x 64 quarter (4 x 4 MFMA tiles).  Per
// stage, 32 probe rows of the hi and lo splits of the tile's 128 a rows and
// 128 b rows (centred, zero past N) are copied global -> LDS with
// global_load_lds_dwordx4 (64-byte rows, chunk l % 4 of a 16-row copy at
// position (l % 4) ^ sw4(row)), kGBuf stages in LDS (two in flight while one
// is read); every fragment read from LDS feeds four MFMA tiles.  Chunks of
// about 400 probe rows give 250 blocks at N = 10,000, one per CU (chunks of
// 256 rows with two blocks per CU and two stages: 21 against 19 us).  A chunk is a whole number of 32-row K-blocks,
// so nothing is masked.
template <>
__global__ __launch_bounds__(kThreads, kGBuf <= 2 ? 2 : 1) void cka_gram_kernel<true>(CkaArgs a) {
  constexpr int NBUF = kGBuf;
  static_assert(NBUF >= 2 && NBUF <= 4, "stages in LDS");
  constexpr int ROWS = kGT2;                  // rows of each operand tile
  constexpr int OB = ROWS * 64;               // bytes of one operand array per stage
  constexpr int STAGE = 4 * OB;               // a hi, a lo, b hi, b lo
  __shared__ __attribute__((aligned(16))) char sm[NBUF * STAGE];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c16 = lane & 15, g = lane >> 4;
  const int R = a.R;
  const int nt = (R + kGT2 - 1) / kGT2;
  int ta, tb;
  upper_pair(blockIdx.x, nt, &ta, &tb);
  const int s = blockIdx.y;
  const int k_beg = s * a.kchunk;
  const int k_end = min(((a.N + 31) & ~31), k_beg + a.kchunk);   // <= ldp
  const int nst = max(0, (k_end - k_beg) / 32);
  // copy plan: 4 arrays x 128 rows = 32 copies of 16 rows per stage, eight
  // per wave: wave w copies rows 32 (w & 3) .. + 31 of every array
  const int crow = lane >> 2, cpos = lane & 3;
  const __bf16* src[8];
  int dst[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int arr = i >> 1;                            // 0 a hi, 1 a lo, 2 b hi, 3 b lo
    const int r0 = 32 * wave + 16 * (i & 1);           // first row of the copy
    const int r = r0 + crow;
    const int grow = min((arr < 2 ? ta : tb) * kGT2 + r, R - 1);
    src[i] = ((arr & 1) ? a.Plo : a.Phi) + (size_t)grow * a.ldp + 8 * (cpos ^ cka_sw4(r));
    dst[i] = arr * OB + r0 * 64;
  }
  const uint32_t sbase = lds_addr(sm);
  auto issue = [&](int st) {
    const int k0 = k_beg + 32 * st;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      dma16(src[i] + k0, __builtin_amdgcn_readfirstlane(sbase + (st % NBUF) * STAGE + dst[i]));
  };
  const int ar0 = 64 * (wave & 1), br0 = 64 * (wave >> 1);
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int p = 0; p < NBUF - 1; ++p)
    if (p < nst) issue(p);
  for (int st = 0; st < nst; ++st) {
    // this wave's copies of stage st are done once at most those of the
    // stages issued after it are outstanding (eight per stage)
    wait_vmcnt_upto<(NBUF - 2) * 8>(min(NBUF - 2, nst - 1 - st) * 8);
    __syncthreads();   // stage st landed everywhere; stage st - 1 is no longer read
    if (st + NBUF - 1 < nst) issue(st + NBUF - 1);
    const char* S = sm + (st % NBUF) * STAGE;
    bf16x8 ah[4], al[4], bh[4], bl[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ra = ar0 + 16 * i + c16, rb = br0 + 16 * i + c16;
      ah[i] = *reinterpret_cast<const bf16x8*>(S + 0 * OB + ra * 64 + 16 * (g ^ cka_sw4(ra)));
      al[i] = *reinterpret_cast<const bf16x8*>(S + 1 * OB + ra * 64 + 16 * (g ^ cka_sw4(ra)));
      bh[i] = *reinterpret_cast<const bf16x8*>(S + 2 * OB + rb * 64 + 16 * (g ^ cka_sw4(rb)));
      bl[i] = *reinterpret_cast<const bf16x8*>(S + 3 * OB + rb * 64 + 16 * (g ^ cka_sw4(rb)));
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[i], bh[j], acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[i], bl[j], acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[i], bh[j], acc[i][j], 0, 0, 0);
      }
  }
  float* out = a.part + (size_t)s * R * R;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = tb * kGT2 + br0 + 16 * j + c16;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = ta * kGT2 + ar0 + 16 * i + 4 * g + v;
        if (row < R && col < R) out[(size_t)row * R + col] = acc[i][j][v];
      }
    }
}

// fp32 inputs: fp32 matrix cores, centring and masking on load.
template <>
__global__ __launch_bounds__(kThreads) void cka_gram_kernel<false>(CkaArgs a) {
  constexpr bool SPLIT = false;
  constexpr int KS = SPLIT ? 32 : 16;      // probe rows per MFMA K-block
  constexpr int PL = KS / 4;               // probe rows per lane per K-block
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
  constexpr int U = SPLIT ? 2 : 4;  // K-blocks loaded ahead of their MFMAs
  for (int k = k_beg; k < k_end; k += KS * U) {
    f32x4 fa[U][2][PL / 4], fb[U][2][PL / 4];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      // rows past k_end (the chunk end, <= ldp) are read but masked below;
      // chunk starts are multiples of 32, ldp of 16 and the start is clamped
      // so that a fragment never crosses the end of its Pt row
      const int kk = min(k + KS * u, a.ldp - KS) + PL * g;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int h = 0; h < PL / 4; ++h) {
          fa[u][j][h] = *reinterpret_cast<const f32x4*>(pa[j] + kk + 4 * h);
          fb[u][j][h] = *reinterpret_cast<const f32x4*>(pb[j] + kk + 4 * h);
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kk = k + KS * u + PL * g;
      float va[2][PL], vb[2][PL];
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < PL; ++e) {
          const bool ok = kk + e < k_end;
          va[j][e] = ok ? fa[u][j][e / 4][e % 4] - ma[j] : 0.f;
          vb[j][e] = ok ? fb[u][j][e / 4][e % 4] - mb[j] : 0.f;
        }
      if constexpr (SPLIT) {
        bf16x8 ha[2], la[2], hb[2], lb[2];
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            ha[j][e] = (__bf16)va[j][e];
            la[j][e] = (__bf16)(va[j][e] - (float)ha[j][e]);
            hb[j][e] = (__bf16)vb[j][e];
            lb[j][e] = (__bf16)(vb[j][e] - (float)hb[j][e]);
          }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(la[i], hb[j], acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ha[i], lb[j], acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ha[i], hb[j], acc[i][j], 0, 0, 0);
          }
      } else {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = Tr<float>::mma(f32x4{va[i][0], va[i][1], va[i][2], va[i][3]},
                                       f32x4{vb[j][0], vb[j][1], vb[j][2], vb[j][3]}, acc[i][j]);
      }
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

// ---------------------------------------------------------------- M

// Thread e: element (e / R, e % R) of M when it lies on or above the
// diagonal (the Gram writes every such element), the sum of its chunks'
// partials in chunk order.  With GB, the last E x nbo blocks of the grid
// form the partials of G_e = B_e^T B_e for ranks up to 8 instead (see
// bgram_small), so that the two small passes share one launch.
__device__ void bgram_small(const CkaArgs& a, int e);

template <bool GB>
__global__ __launch_bounds__(kThreads) void cka_msum_kernel(CkaArgs a) {
  const int R = a.R;
  const int mblocks = (int)(((long)R * R + kThreads - 1) / kThreads);
  if (GB && (int)blockIdx.x >= mblocks) {
    bgram_small(a, (int)blockIdx.x - mblocks);
    return;
  }
  const long e = (long)blockIdx.x * kThreads + threadIdx.x;
  if (e >= (long)R * R) return;
  const int row = (int)(e / R), col = (int)(e % R);
  if (row > col) return;
  const size_t off = (size_t)e, cs = (size_t)R * R;
  float m = 0.f;
  for (int s = 0; s < a.splits; s += 8) {
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = a.part[(size_t)min(s + i, a.splits - 1) * cs + off];
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (s + i < a.splits) m += v[i];
  }
  a.M[off] = m;
}

// ---------------------------------------------------------------- B^T B

// Block (e, c): partial G_e over rows c*kBO .. of B_e, all rows loaded at once.
template <typename T>
__global__ __launch_bounds__(kThreads) void cka_bgram_kernel(CkaArgs a) {
  __shared__ float bs[kBO * 64];
  const int e = blockIdx.x, c = blockIdx.y, r = a.r, rr = r * r;
  const int o0 = c * kBO, rows = min(kBO, a.d_out - o0);
  const T* B = static_cast<const T*>(a.B) + (size_t)a.d_out * r * e + (size_t)o0 * r;
#pragma unroll 8
  for (int i = threadIdx.x; i < rows * r; i += kThreads) bs[i] = (float)B[i];
  __syncthreads();
  for (int pq = threadIdx.x; pq < rr; pq += kThreads) {
    const int p = pq / r, q = pq % r;
    float acc = 0.f;
    for (int o = 0; o < rows; ++o) acc += bs[o * r + p] * bs[o * r + q];
    a.Gb[((size_t)e * a.nbo + c) * rr + pq] = acc;
  }
}

// Ranks up to 8: block (e, c) of the msum launch forms the partial G_e over
// rows c*kBO .. of B_e (like cka_bgram).  The chunk is staged in LDS as fp32;
// lane t of wave w sums B[o][p] B[o][q], (p, q) = (t / r, t % r), over the
// chunk rows o = w, w + 4, ... in order, and the four waves' sums are added in
// wave order (deterministic).
template <typename T>
__device__ void bgram_small_t(const CkaArgs& a, int blk) {
  __shared__ float bs[kBO * 8];
  __shared__ float wsum[kThreads / 64][64];
  const int e = blk / a.nbo, c = blk % a.nbo;
  const int r = a.r, rr = r * r;
  const int o0 = c * kBO, rows = min(kBO, a.d_out - o0);
  const T* B = static_cast<const T*>(a.B) + (size_t)a.d_out * r * e + (size_t)o0 * r;
  for (int i = threadIdx.x; i < rows * r; i += kThreads) bs[i] = (float)B[i];
  __syncthreads();
  const int t = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float acc = 0.f;
  if (t < rr) {
    const int p = t / r, q = t % r;
#pragma unroll 8
    for (int o = wave; o < rows; o += kThreads / 64) acc += bs[o * r + p] * bs[o * r + q];
  }
  wsum[wave][t] = acc;
  __syncthreads();
  if (threadIdx.x < rr) {
    float g = 0.f;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) g += wsum[w][threadIdx.x];
    a.Gb[((size_t)e * a.nbo + c) * rr + threadIdx.x] = g;
  }
}

// ---------------------------------------------------------------- pairs

// Block per expert pair i <= j: M_ij (read from the upper triangle of the
// symmetric M), then <G_i M_ij, M_ij G_j>.
__global__ __launch_bounds__(kThreads) void cka_pairs_kernel(CkaArgs a) {
  __shared__ float Gi[64 * 64], Gj[64 * 64], Mij[64 * 64];
  __shared__ float red[kThreads];
  int i, j;
  upper_pair(blockIdx.x, a.E, &i, &j);
  const int r = a.r, rr = r * r, R = a.R;
  for (int t = threadIdx.x; t < rr; t += kThreads) {
    float gi = 0.f, gj = 0.f;
    for (int c = 0; c < a.nbo; ++c) {
      gi += a.Gb[((size_t)i * a.nbo + c) * rr + t];
      gj += a.Gb[((size_t)j * a.nbo + c) * rr + t];
    }
    Gi[t] = gi;
    Gj[t] = gj;
    const int row = i * r + t / r, col = j * r + t % r;
    Mij[t] = a.M[(size_t)min(row, col) * R + max(row, col)];
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

// Ranks up to 8: one wave per expert pair i <= j, four pairs per block; lane
// t < r * r holds element t of G_i, G_j (chunk partials summed in order) and
// of M_ij, M_ii, M_jj (wave-private LDS rows); the lanes' products are summed
// by shuffles into num_ij, num_ii and num_jj, and the wave writes S_ij = S_ji
// directly (num_ii is formed by the same code from the same operands in
// every wave that needs it, so the diagonal agrees everywhere).
__device__ inline float pair_num8(const float* Ga, const float* Mab, const float* Gb, int r, int t) {
  float acc = 0.f;
  if (t < r * r) {
    const int p = t / r, q = t % r;
    float t1 = 0.f, t2 = 0.f;
    for (int u = 0; u < r; ++u) {
      t1 += Ga[p * r + u] * Mab[u * r + q];   // (G_a M_ab)[p][q]
      t2 += Mab[p * r + u] * Gb[u * r + q];   // (M_ab G_b)[p][q]
    }
    acc = t1 * t2;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
  return acc;
}

__device__ inline float cka_score(float nij, float nii, float njj) {
  const float den = sqrtf(nii) * sqrtf(njj);
  const float v = den > 0.f ? nij / den : 0.f;
  return isfinite(v) ? v : 0.f;
}

__global__ __launch_bounds__(kThreads) void cka_pairs8_kernel(CkaArgs a) {
  __shared__ float Gi[kThreads / 64][64], Gj[kThreads / 64][64];
  __shared__ float Mij[kThreads / 64][64], Mii[kThreads / 64][64], Mjj[kThreads / 64][64];
  const int wave = threadIdx.x >> 6, t = threadIdx.x & 63;
  const int pidx = blockIdx.x * (kThreads / 64) + wave;
  const bool live = pidx < a.E * (a.E + 1) / 2;   // wave-uniform
  const int r = a.r, rr = r * r, R = a.R;
  int i = 0, j = 0;
  if (live) upper_pair(pidx, a.E, &i, &j);
  if (live && t < rr) {
    float gi = 0.f, gj = 0.f;
    for (int c = 0; c < a.nbo; ++c) {
      gi += a.Gb[((size_t)i * a.nbo + c) * rr + t];
      gj += a.Gb[((size_t)j * a.nbo + c) * rr + t];
    }
    Gi[wave][t] = gi;
    Gj[wave][t] = gj;
    const int p = t / r, q = t % r;
    const int row = i * r + p, col = j * r + q;
    Mij[wave][t] = a.M[(size_t)min(row, col) * R + max(row, col)];
    Mii[wave][t] = a.M[(size_t)(i * r + min(p, q)) * R + i * r + max(p, q)];
    Mjj[wave][t] = a.M[(size_t)(j * r + min(p, q)) * R + j * r + max(p, q)];
  }
  __syncthreads();
  if (!live) return;   // wave-uniform
  const float nij = pair_num8(Gi[wave], Mij[wave], Gj[wave], r, t);
  const float nii = pair_num8(Gi[wave], Mii[wave], Gi[wave], r, t);
  const float njj = pair_num8(Gj[wave], Mjj[wave], Gj[wave], r, t);
  if (t == 0) {
    const float v = cka_score(nij, nii, njj);
    a.S[(size_t)i * a.E + j] = v;
    a.S[(size_t)j * a.E + i] = v;
  }
}

__global__ __launch_bounds__(kThreads) void cka_score_kernel(CkaArgs a) {
  const int t = blockIdx.x * kThreads + threadIdx.x;
  const int E = a.E;
  if (t >= E * E) return;
  const int i = t / E, j = t % E;
  a.S[t] = cka_score(a.num[t], a.num[(size_t)i * E + i], a.num[(size_t)j * E + j]);
}

__device__ void bgram_small(const CkaArgs& a, int e) {
  if (a.bf16) bgram_small_t<__bf16>(a, e);
  else bgram_small_t<float>(a, e);
}

template <typename T>
hipError_t launch_cka_t(const CkaProblem& p, void* ws, hipStream_t stream) {
  const CkaLayout L = cka_layout(p.N, p.d_out, p.E, p.r);
  char* base = static_cast<char*>(ws);
  CkaArgs a{};
  a.X = p.X;
  a.A = p.A;
  a.B = p.B;
  a.Pt = reinterpret_cast<float*>(base + L.Pt);
  a.mean = reinterpret_cast<float*>(base + L.mean);
  a.part = reinterpret_cast<float*>(base + L.part);
  a.M = reinterpret_cast<float*>(base + L.M);
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
  a.nbo = L.nbo;
  a.Phi = reinterpret_cast<__bf16*>(base + L.Phi);
  a.Plo = reinterpret_cast<__bf16*>(base + L.Plo);
  a.bf16 = p.dtype == ACE_BF16 ? 1 : 0;
  const int R = a.R;
  if (p.N > 0) {
    dim3 grid((p.N + kPN - 1) / kPN, (R + kPC - 1) / kPC);
    cka_project_kernel<T, kPN, kPBuf><<<grid, kPThreads, 0, stream>>>(a);
  }
  if (p.dtype == ACE_BF16)
    cka_mean_kernel<true><<<R, kThreads, 0, stream>>>(a);
  else
    cka_mean_kernel<false><<<R, kThreads, 0, stream>>>(a);
  if (p.dtype == ACE_BF16) {
    const int nt = (R + kGT2 - 1) / kGT2;
    cka_gram_kernel<true><<<dim3(nt * (nt + 1) / 2, L.splits), kThreads, 0, stream>>>(a);
  } else {
    const int nt = (R + kGT - 1) / kGT;
    cka_gram_kernel<false><<<dim3(nt * (nt + 1) / 2, L.splits), kThreads, 0, stream>>>(a);
  }
  const int mblocks = (int)(((long)R * R + kThreads - 1) / kThreads);
  if (p.r <= 8) {
    // B^T B partials in the msum launch, then one wave per pair writing the
    // scores
    cka_msum_kernel<true><<<mblocks + p.E * L.nbo, kThreads, 0, stream>>>(a);
    cka_pairs8_kernel<<<(p.E * (p.E + 1) / 2 + kThreads / 64 - 1) / (kThreads / 64), kThreads, 0, stream>>>(a);
  } else {
    cka_msum_kernel<false><<<mblocks, kThreads, 0, stream>>>(a);
    cka_bgram_kernel<T><<<dim3(p.E, L.nbo), kThreads, 0, stream>>>(a);
    cka_pairs_kernel<<<p.E * (p.E + 1) / 2, kThreads, 0, stream>>>(a);
    cka_score_kernel<<<(p.E * p.E + kThreads - 1) / kThreads, kThreads, 0, stream>>>(a);
  }
  return hipGetLastError();
}

}  // namespace

size_t cka_ws_bytes(int N, int d_out, int E, int r) { return cka_layout(N, d_out, E, r).total; }

hipError_t launch_cka(const CkaProblem& p, void* ws, hipStream_t stream) {
  if (p.dtype == ACE_BF16) return launch_cka_t<__bf16>(p, ws, stream);
  return launch_cka_t<float>(p, ws, stream);
}

}  // namespace ace
