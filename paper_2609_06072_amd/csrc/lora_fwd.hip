// Grouped LoRA forward (Sec. 3.4 shared-adapter output, executed as in
// Sec. 3.5: c_g(x) = B_g (A_g x) once per row of the permutation, then handed
// to every slot the row serves).
//
// One persistent launch.  A tile is 64 rows of one key's segment; each of the
// 4 waves owns 16 rows.  Per wave:
//   shrink  H^T = A_q X^T     K = d_in, MFMA, H stays in registers (fp32)
//   expand  C^T = B_q H^T     K = r_q; the shrink accumulators are fed back
//                             as the MFMA operand (rank order of kmap_acc),
//                             scaled by alpha / r_q first
//   epilogue y[t*k + j] += w_tj * C for every slot j of the row
// Tiles are enumerated key-major from the device-side segment offsets, so the
// launch needs no host synchronisation on the row count.
#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

constexpr int kBM = 64;   // rows per tile (4 waves x 16)
constexpr int kNCH = 4;   // 16-column output blocks per epilogue batch

struct FwdArgs {
  const void* x;
  const void* A;
  const void* B;
  const float* pair_w;
  void* y;
  const int32_t* offsets;
  const int32_t* row_token;
  const uint32_t* row_slots;
  int32_t k, d_in, d_out, per_pair;
  float alpha;
  KeyTable keys;
};

template <typename T, int RB>
__global__ __launch_bounds__(kThreads) void lora_fwd_kernel(FwdArgs a) {
  using F = typename Tr<T>::frag;
  constexpr int APF = Tr<T>::ACC_PER_FRAG;
  constexpr int NM = RB / APF;  // rank K-blocks
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
  const T* Bw = static_cast<const T*>(a.B);
  T* Y = static_cast<T*>(a.y);
  const int d_in = a.d_in, d_out = a.d_out, k = a.k;

  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    const int q = find_key(tstart, n_keys, tile);
    const int u_begin = seg[q] + (tile - tstart[q]) * kBM + wave * 16;
    const int u_end = seg[q + 1];
    if (u_begin >= u_end) continue;  // wave-uniform: no rows for this wave
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
    const int xr = a.per_pair ? tok * k + __builtin_ctz(slots | 0x80000000u) : tok;

    // ---- shrink: acc[rb][v] = H[u][16 rb + 4 g + v]
    f32x4 acc[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
    const T* xrow = X + (size_t)xr * d_in;
    for (int kk = 0; kk < d_in; kk += Tr<T>::KB) {
      const int kof = kk + Tr<T>::PER * g;
      const bool kok = kof < d_in;
      const F xf = (valid && kok) ? Tr<T>::load(xrow + kof) : Tr<T>::zero();
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        if (rb < nrb) {
          const int r = rb * 16 + c16;
          const F af = (r < r_q && kok) ? Tr<T>::load(Aw + (size_t)(roff + r) * d_in + kof)
                                        : Tr<T>::zero();
          acc[rb] = Tr<T>::mma(af, xf, acc[rb]);
        }
      }
    }

    // ---- expand + scale + scatter-add
    const float s = a.alpha / (float)r_q;
    F hf[NM];
#pragma unroll
    for (int m = 0; m < NM; ++m) hf[m] = Tr<T>::from_acc(acc, m, s);
    const T* Bq = Bw + (size_t)d_out * roff;
    const bool al4 = (r_q & 3) == 0;
    for (int n0 = 0; n0 < d_out; n0 += 16 * kNCH) {
      f32x4 c[kNCH];
#pragma unroll
      for (int ch = 0; ch < kNCH; ++ch) {
        c[ch] = f32x4{0.f, 0.f, 0.f, 0.f};
        const int n = n0 + ch * 16 + c16;
        const bool nok = n < d_out;
#pragma unroll
        for (int m = 0; m < NM; ++m) {
          if (m < nmb) {
            const F bf = load_acc_order<T>(Bq + (size_t)(nok ? n : 0) * r_q, r_q, m, g, nok, al4);
            c[ch] = Tr<T>::mma(bf, hf[m], c[ch]);  // c[ch][v] = C[u][n0 + 16 ch + 4 g + v]
          }
        }
      }
      if (valid) {
        for (uint32_t mm = slots; mm; mm &= mm - 1u) {
          const int p = tok * k + __builtin_ctz(mm);
          const float w = a.pair_w ? a.pair_w[p] : 1.f;
          T* yrow = Y + (size_t)p * d_out + n0 + 4 * g;
          f32x4 old[kNCH];
#pragma unroll
          for (int ch = 0; ch < kNCH; ++ch)
            if (n0 + ch * 16 + 4 * g < d_out) old[ch] = Tr<T>::load4(yrow + ch * 16);
#pragma unroll
          for (int ch = 0; ch < kNCH; ++ch)
            if (n0 + ch * 16 + 4 * g < d_out) Tr<T>::store4(yrow + ch * 16, old[ch] + w * c[ch]);
        }
      }
    }
  }
}

template <typename T>
hipError_t launch_fwd_t(const Problem& p, void* y, hipStream_t stream) {
  FwdArgs a{};
  a.x = p.x;
  a.A = p.A;
  a.B = p.B;
  a.pair_w = p.pair_w;
  a.y = y;
  a.offsets = p.rt->offsets;
  a.row_token = p.rt->row_token;
  a.row_slots = p.rt->row_slots;
  a.k = p.k;
  a.d_in = p.d_in;
  a.d_out = p.d_out;
  a.per_pair = p.per_pair;
  a.alpha = p.alpha;
  a.keys = p.keys;
  const long P = (long)p.T * p.k;
  const long bound = (P + kBM - 1) / kBM + p.keys.n_keys;
  const long cap = 4L * device_cu_count();
  const int grid = (int)(bound < cap ? bound : cap);
  if (grid <= 0) return hipSuccess;
  const int rb = (p.r_max + 15) / 16;
  if (rb <= 2) {
    lora_fwd_kernel<T, 2><<<grid, kThreads, 0, stream>>>(a);
  } else if (rb <= 4) {
    lora_fwd_kernel<T, 4><<<grid, kThreads, 0, stream>>>(a);
  } else if (rb <= 8) {
    lora_fwd_kernel<T, 8><<<grid, kThreads, 0, stream>>>(a);
  } else {
    lora_fwd_kernel<T, 16><<<grid, kThreads, 0, stream>>>(a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_fwd(const Problem& p, void* y, hipStream_t stream) {
  if (p.dtype == ACE_BF16) return launch_fwd_t<__bf16>(p, y, stream);
  return launch_fwd_t<float>(p, y, stream);
}

}  // namespace ace
