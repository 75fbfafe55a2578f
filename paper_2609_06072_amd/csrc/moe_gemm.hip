// Adapted expert projection: the frozen expert GEMM of an MoE layer with the
// adapter update added in its epilogue (Sec. 3.1 base projection W_e x plus
// the Sec. 3.4 shared-adapter update, executed as in Sec. 3.5):
//   y[t*k + j] = W_e xin(t, j) + B_q h_u,   e = topk_ids[t, j], q = key of e,
// where h_u = (alpha / r_q) A_q xin is the shrink of the adapter row u that
// serves the pair (one row per (token, active group) for grouped execution,
// one per pair for expert-wise LoRA), computed beforehand by the contract
// kernel.  y is written once: the adapter's read-modify-write of y is gone.
//
// Tiles.  The rows of the expert routing (sorted by expert, then token) are
// cut into tiles of BM rows of one expert; a block computes a BM x BN
// output tile (GCfg).  The contraction runs over d_in (x rows against W_e rows, both
// K-contiguous) and then over the adapter rank (h rows against B_q rows, also
// K-contiguous), all into the same fp32 accumulators.
//
// Data movement.  One K-block (64 bytes of every row: 32 bf16 or 16 fp32) per
// stage; x and W_e pieces are copied global -> LDS directly
// (global_load_lds_dwordx4), NBUF stages in LDS.  Within a stage a row's
// four 16-byte chunks sit XOR-swizzled (g_swz), so the fragment reads of 16
// consecutive rows hit distinct banks.  The adapter K-blocks (one
// or two) are read straight into registers while the first stages are in
// flight.
//
// Waves.  WM x WN waves over the tile: wave (wy, wx) owns rows 64*wy .. +64
// and columns 128*wx .. +128, i.e. 4 x 8 blocks of 16 x 16.  The
// weight rows are the first MFMA operand, so a lane's accumulator holds four
// consecutive output columns of one row; the epilogue stages the tile in LDS
// and writes y with 16-byte stores of whole row pieces.
//
// Block order.  Blocks are dealt to the 8 XCDs round-robin; block b takes
// tile (b % 8) * ceil(n_tiles / 8) + b / 8, so each XCD walks a contiguous
// run of tiles (expert-major): an expert's weight slices stay in one L2.
#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

constexpr int kGRowBytes = 64;           // bytes of a row per stage (one K-block)

// Tile geometry: WM x WN waves of 64 rows x 128 columns each, NBUF stages of
// (BM + BN) rows x 64 bytes in LDS.
template <int WM_, int WN_, int NBUF_>
struct GCfg {
  static constexpr int WM = WM_, WN = WN_, NBUF = NBUF_;
  static constexpr int NW = WM * WN, THREADS = 64 * NW;
  static constexpr int BM = 64 * WM, BN = 128 * WN;
  static constexpr int XBYTES = BM * kGRowBytes, STAGE = (BM + BN) * kGRowBytes;
  static constexpr int COPIES = (BM + BN) / 16 / NW;   // 16-row copies per wave per stage
  static_assert((BM + BN) / 16 % NW == 0, "copies must split evenly over the waves");
  static_assert(THREADS >= BM, "one thread per tile row fills the row tables");
};
// Two launch shapes.  Experts with few rows each (the fine-grained MoEs):
// 128-row x 256-column tiles, four waves, three stages (72 KB of LDS, two
// blocks per CU), so that an expert's last tile wastes little.  Experts with
// many rows (>= kBigRows on average): 256 x 256 tiles, eight waves, four
// stages (128 KB, one block per CU): a third fewer bytes per flop through the
// L2 and 1.5x the work covered by the copies in flight.
using MoeSmall = GCfg<2, 2, 3>;
using MoeBig = GCfg<4, 2, 4>;
constexpr long kBigRows = 1024;

// Epilogue passes over column slices so that the C tile [BM][BN/NH + pad]
// fits the stage buffers.
template <class C, typename T>
constexpr int epi_passes() {
  int nh = 1;
  while (C::BM * (C::BN / nh + 16 / (int)sizeof(T)) * (int)sizeof(T) > C::NBUF * C::STAGE) nh *= 2;
  return nh;
}

// Chunk position of a row's 16-byte chunk 0.  Rows 64 bytes apart share a
// bank line; the position differs for any two rows among 8 consecutive ones
// with the same parity and among 16 consecutive ones with the same residue
// mod 4, so a fragment read (16 rows, one chunk each) is free of bank
// conflicts whether the LDS serves 8 or 16 lanes of a 16-byte read per cycle.
__device__ inline int g_swz(int row) { return (((row >> 1) ^ (row >> 3)) & 1) | ((row >> 1) & 2); }

// Number of tiles of BM rows over the key segments offsets[0 .. n_keys]
// (wave-level; every lane gets the total).
__device__ inline int count_tiles(const int32_t* offsets, int n_keys, int BM) {
  constexpr int KPL = kMaxKeys / 64;
  const int lane = threadIdx.x & 63;
  int cnt = 0;
  int prev = offsets[min(lane * KPL, n_keys)];
#pragma unroll
  for (int i = 0; i < KPL; ++i) {
    const int nxt = offsets[min(lane * KPL + i + 1, n_keys)];
    cnt += (nxt - prev + BM - 1) / BM;
    prev = nxt;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
  return cnt;
}

template <typename T, class C>
__global__ __launch_bounds__(C::THREADS, 512 / C::THREADS) void moe_gemm_kernel(MoeArgs a) {
  using F = typename Tr<T>::frag;
  constexpr int PER = Tr<T>::PER, KB = Tr<T>::KB;
  constexpr int BM = C::BM, BN = C::BN, NBUF = C::NBUF, STAGE = C::STAGE, COPIES = C::COPIES;
  constexpr int NT = C::THREADS;
  constexpr int NH = epi_passes<C, T>();       // epilogue passes over column slices
  constexpr int HC = BN / NH;                  // columns per pass
  constexpr int CST = HC + 16 / (int)sizeof(T);
  __shared__ __attribute__((aligned(16))) char smem[NBUF * STAGE];
  __shared__ int s_src[BM];    // x row of each tile row (clamped into the segment)
  __shared__ int s_out[BM];    // y row, -1 past the segment
  __shared__ int s_h[BM];      // adapter row, -1 for none

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c16 = lane & 15, g = lane >> 4;
  const int wy = wave / C::WN, wx = wave % C::WN;

  // ---- which tile
  const int n_mt = count_tiles(a.offsets, a.E, BM);
  const int n_tiles = n_mt * a.nt;
  const int per_xcd = (n_tiles + kXcds - 1) / kXcds;
  const int bi = blockIdx.x / kXcds;
  const int tile = (blockIdx.x % kXcds) * per_xcd + bi;
  if (bi >= per_xcd || tile >= n_tiles) return;
  const int mt = tile / a.nt, n0 = (tile % a.nt) * BN;
  int e, u0, uend;
  locate_tile(a.offsets, a.E, BM, mt, &e, &u0, &uend);

  if (tid < BM) {
    const int u = u0 + tid;
    const int uc = min(u, uend - 1);
    const int tok = a.row_token[uc];
    const int j = __builtin_ctz(a.row_slots[uc] | 0x80000000u) & 31;
    const int p = tok * a.k + j;
    s_src[tid] = a.per_pair ? p : tok;
    s_out[tid] = u < uend ? p : -1;
    s_h[tid] = (u < uend && a.H) ? a.h_row[p] : -1;
  }
  __syncthreads();

  // A wave whose 64 rows all lie past the expert's last row (the tail of its
  // last tile) skips its matrix work; it still takes part in the copies, the
  // LDS reads and the barriers.  Its accumulators stay zero and are never
  // stored.
  const bool active = u0 + 64 * wy < uend;
  const T* X = static_cast<const T*>(a.x);
  const T* Wt = static_cast<const T*>(a.W) + (size_t)e * a.d_out * a.d_in;
  const int d_in = a.d_in, d_out = a.d_out;
  const int nst = (d_in + KB - 1) / KB;

  // ---- copy assignment: lane covers row (lane >> 2) of each 16-row copy,
  // chunk position lane & 3 (global chunk (lane & 3) ^ g_swz(row)).  The
  // swizzle only sees bits 1..3 of the row, i.e. of lane >> 2, so one chunk
  // offset serves every copy; rows are 32-bit element offsets from X or W_e.
  const int cpos = lane & 3, crl = lane >> 2;
  const int coff = PER * (cpos ^ g_swz(crl));
  uint32_t roff[COPIES];
#pragma unroll
  for (int i = 0; i < COPIES; ++i) {
    const int blk = wave * COPIES + i;        // 16-row copy index over [x rows | W rows]
    const int row = 16 * blk + crl;
    roff[i] = 16 * blk < BM ? (uint32_t)s_src[row] * (uint32_t)d_in
                            : (uint32_t)min(n0 + row - BM, d_out - 1) * (uint32_t)d_in;
  }
  const uint32_t sbase = lds_addr(smem);
  auto issue = [&](int st) {
    const uint32_t buf = sbase + (st % NBUF) * STAGE;
    const uint32_t kk = (uint32_t)min(st * KB + coff, d_in - PER);
#pragma unroll
    for (int i = 0; i < COPIES; ++i) {
      const int blk = wave * COPIES + i;
      const bool xcopy = 16 * blk < BM;
      dma16((xcopy ? X : Wt) + (roff[i] + kk),
            __builtin_amdgcn_readfirstlane(buf + 16 * blk * kGRowBytes));
    }
  };
#pragma unroll
  for (int s = 0; s < NBUF; ++s)
    if (s < nst) issue(s);

  f32x4 acc[8][4];
#pragma unroll
  for (int nb = 0; nb < 8; ++nb)
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) acc[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // ---- adapter K-blocks: acc[n][m] += sum_rho B_q[n][rho] h_m[rho]
  if (a.H && active) {
    const int q = a.key_of[e];
    const int r_q = a.keys.rank[q];
    const T* Bq = static_cast<const T*>(a.B) + (size_t)d_out * a.keys.roff[q];
    const T* Hm = static_cast<const T*>(a.H);
    const bool bvec = (r_q % PER) == 0;
    for (int kb = 0; kb * KB < r_q; ++kb) {
      const int rho = kb * KB + PER * g;
      F hf[4], bf[8];
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        const int hr = s_h[64 * wy + 16 * mb + c16];
        hf[mb] = hr >= 0 ? Tr<T>::load(Hm + (size_t)hr * a.rpad + rho) : Tr<T>::zero();
      }
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) {
        const int n = min(n0 + 128 * wx + 16 * nb + c16, d_out - 1);
        bf[nb] = load_frag<T>(Bq + (size_t)n * r_q + rho, r_q - rho, bvec);
      }
#pragma unroll
      for (int nb = 0; nb < 8; ++nb)
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) acc[nb][mb] = Tr<T>::mma(bf[nb], hf[mb], acc[nb][mb]);
    }
  }

  // ---- main loop over d_in, fragments double-buffered in registers: the
  // LDS reads of K-block st + 1 are in flight while the matrix cores work on
  // K-block st.
  // fragment rows 64 wy + 16 mb + c16 (x) and 128 wx + 16 nb + c16 (W): the
  // swizzle again depends on c16 only, so a read is a lane base plus an
  // immediate offset
  const int xl = (64 * wy + c16) * kGRowBytes + ((g ^ g_swz(c16)) << 4);
  const int wl = C::XBYTES + (128 * wx + c16) * kGRowBytes + ((g ^ g_swz(c16)) << 4);
  auto read_frags = [&](int st, F (&xf)[4], F (&wf)[8]) {
    const char* S = smem + (st % NBUF) * STAGE;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) xf[mb] = *reinterpret_cast<const F*>(S + xl + mb * 16 * kGRowBytes);
#pragma unroll
    for (int nb = 0; nb < 8; ++nb)
      wf[nb] = *reinterpret_cast<const F*>(S + wl + nb * 16 * kGRowBytes);
  };
  auto mma_all = [&](const F (&xf)[4], const F (&wf)[8]) {
#pragma unroll
    for (int nb = 0; nb < 8; ++nb)
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) acc[nb][mb] = Tr<T>::mma(wf[nb], xf[mb], acc[nb][mb]);
  };
  // The last K-block may reach past d_in: once it has landed, its x chunks
  // past d_in (copies of the clamped last chunk) are cleared in LDS, so no
  // fragment read needs a mask.  Called with stage st landed and published
  // (possibly twice for the last stage: clearing again changes nothing).
  auto clear_tail = [&](int st) {
    if (st != nst - 1 || d_in % KB == 0) return;
    const int valid = (d_in - st * KB) / PER;   // chunks of this K-block inside d_in
    char* S = smem + (st % NBUF) * STAGE;
    for (int i = tid; i < BM * 4; i += NT) {
      const int row = i >> 2, pos = i & 3;
      if ((pos ^ g_swz(row)) >= valid) *reinterpret_cast<u32x4*>(S + row * kGRowBytes + pos * 16) = u32x4{0u, 0u, 0u, 0u};
    }
    __syncthreads();
  };
  // Stage st lives in buffer st % NBUF.  Before K-block st + 1 is read, the
  // barrier also tells that every wave holds K-block st in registers, so
  // its buffer takes stage st + NBUF.
  // Every half-step reads the next K-block unconditionally (clamped to the
  // last one: a repeated read of a landed buffer is harmless), so the reads
  // and the matrix work on the previous block share one basic block.
  F xa[4], wa[8], xb[4], wb[8];
  wait_vmcnt_upto<(NBUF - 1) * COPIES>(min(NBUF - 1, nst - 1) * COPIES);
  __syncthreads();
  clear_tail(0);
  read_frags(0, xa, wa);
  auto half = [&](int st, F (&xc)[4], F (&wc)[8], F (&xn)[4], F (&wn)[8]) {
    // K-block st is in (xc, wc); K-block st + 1 lands in (xn, wn)
    wait_vmcnt_upto<(NBUF - 2) * COPIES>(min(NBUF - 2, nst - 2 - st) * COPIES);
    __syncthreads();
    if (st + NBUF < nst) issue(st + NBUF);
    const int sn = min(st + 1, nst - 1);
    clear_tail(sn);
    read_frags(sn, xn, wn);
    if (active) mma_all(xc, wc);
  };
  for (int st = 0; st < nst; st += 2) {
    half(st, xa, wa, xb, wb);
    if (st + 1 >= nst) break;
    half(st + 1, xb, wb, xa, wa);
  }

  // ---- epilogue: C tile -> LDS [m][n] (over the stage buffers), then whole
  // 16-byte row pieces of y
  T* Cs = reinterpret_cast<T*>(smem);
  T* Y = static_cast<T*>(a.y);
  constexpr int CPR = HC / PER;                 // 16-byte pieces per row and pass
  constexpr int NP = BM * CPR / NT;
  static_assert(BM * CPR % NT == 0, "epilogue pieces must split evenly");
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    __syncthreads();
#pragma unroll
    for (int nb = 0; nb < 8; ++nb) {
      const int nl = 128 * wx + 16 * nb + 4 * g - h * HC;   // column inside this pass
      if (nl >= 0 && nl < HC) {
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) {
          T* cp = Cs + (64 * wy + 16 * mb + c16) * CST + nl;
#pragma unroll
          for (int v = 0; v < 4; ++v) cp[v] = (T)acc[nb][mb][v];
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const int it = tid + i * NT;
      const int m = it / CPR, pc = (it % CPR) * PER;
      const int orow = s_out[m];
      const int col = n0 + h * HC + pc;
      if (orow >= 0 && col < d_out)
        Tr<T>::store(Y + (size_t)orow * d_out + col, *reinterpret_cast<const F*>(Cs + m * CST + pc));
    }
  }
}

template <class C>
hipError_t launch_moe_cfg(int dtype, MoeArgs a, long P, hipStream_t stream) {
  a.nt = (a.d_out + C::BN - 1) / C::BN;
  const long max_tiles = ((P + C::BM - 1) / C::BM + a.E) * a.nt;
  const long grid = (max_tiles + kXcds - 1) / kXcds * kXcds;
  if (grid <= 0) return hipSuccess;
  if (dtype == ACE_BF16) moe_gemm_kernel<__bf16, C><<<(int)grid, C::THREADS, 0, stream>>>(a);
  else moe_gemm_kernel<float, C><<<(int)grid, C::THREADS, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_moe_gemm(int dtype, const MoeArgs& a, long P, hipStream_t stream) {
  if (P >= kBigRows * a.E) return launch_moe_cfg<MoeBig>(dtype, a, P, stream);
  return launch_moe_cfg<MoeSmall>(dtype, a, P, stream);
}

}  // namespace ace
