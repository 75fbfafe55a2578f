// Pre-combined adapter input (ACE_INPUT_COMBINED): the down projection of an
// MoE layer whose output is combined over the routed experts with the
// routing weights (Sec. 3.1).  Because that combine is linear, the adapter
// part of the combined output of token t is
//   out[t] += sum_{u: rows of t} s_q B_q A_q z_u,   z_u = sum_{p in u} w_p x_p
// -- one input combination and one adapter evaluation per (token, active
// group) row, the compute-once reuse of Sec. 3.5 carried over to an input
// that differs per routed pair.  Since A_q is linear the launches evaluate
// h_u = s_q A_q z_u as sum_p w_p (s_q A_q x_p):
//
// Forward (h_p per pair position stays in the workspace for the backward):
//   prep      -- B^T rows [R][d_out] (matrix-core GEMM operand) or B
//                re-strided to [d_out][R] (register GEMM); zero the dense
//                per-token h rows.
//   contract  -- h_p = s_q A_q x_p for every routed pair, in pair order.
//   combine   -- h_u = sum_{p in u} w_p h_p into the dense rows Hd[t][roff_q..].
//   GEMM      -- out[t] += Hd[t] B^T over K = R (inactive groups hold zeros).
// Backward, with G_t = dOut[t] (every row of token t sees the same gradient):
//   dB_q = sum_u G_t h_u^T                (rows of q)
//   dH_u = s_q B_q^T G_t
//   dA_q = sum_p (w_p dH_{u(p)}) x_p^T    (pairs of q)
//   dx_p += w_p A_q^T dH_{u(p)}
// Launches: prep (A^T, B^T) -> [contract h_p unless the forward's is passed]
// -> combine (h_u, transposed per key) -> contract dH per row (stored per row
// and, times each pair's weight, per pair position) -> expand dx over the
// slots of every row -> weight gradients (dB over rows, dA over pairs).
#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

struct FwdLayout {
  size_t hp, Hd, Bm, total;
};

// hp [P][rpad] first (a backward reads it from there), dense h rows [T][R],
// the B operand of the GEMM ([R][d_out] or [d_out][R]); R <= n_keys * r_max.
FwdLayout fwd_layout(int T, int k, int d_out, int n_keys, int r_max, size_t es) {
  const size_t P = (size_t)T * k;
  const size_t Rb = (size_t)n_keys * r_max;
  FwdLayout w{};
  size_t o = 0;
  w.hp = o;  o += align256(es * P * rank_pad(ACE_F32, r_max));
  w.Hd = o;  o += align256(es * (size_t)T * Rb);
  w.Bm = o;  o += align256(es * Rb * d_out);
  w.total = o;
  return w;
}

struct BwdLayout {
  size_t At, Bt, hp, Ht, dHw, dHrow, part, total;
};

// At [d_in][R], Bt [R][d_out], hp [P][rpad], Ht / dHw [R][ldh], dH rows
// [P][rpad], weight-gradient partials; 256 bytes of slack (the gradient pass
// reads whole 16-byte fragments of Ht / dHw rows past a segment's end).
BwdLayout bwd_layout(int T, int k, int d_in, int d_out, int n_keys, int r_max, size_t es) {
  const size_t P = (size_t)T * k;
  const size_t Rb = (size_t)n_keys * r_max;
  const size_t ldh = (P + 7) & ~(size_t)7;
  const size_t rpad = rank_pad(ACE_F32, r_max);
  BwdLayout w{};
  size_t o = 0;
  w.At = o;    o += align256(es * d_in * Rb);
  w.Bt = o;    o += align256(es * Rb * d_out);
  w.hp = o;    o += align256(es * P * rpad);
  w.Ht = o;    o += align256(es * Rb * ldh);
  w.dHw = o;   o += align256(es * Rb * ldh);
  w.dHrow = o; o += align256(es * P * rpad);
  w.part = o;  o += align256(grads_part_bytes(T, k, d_in, d_out, n_keys, r_max));
  w.total = o + 256;
  return w;
}

// Bd[n][roff_q + r] = B_q[n][r]: B as one [d_out][R] matrix, the layout the
// register GEMM reads its second operand in.
template <typename T>
__global__ __launch_bounds__(kThreads) void restride_b_kernel(const T* B, T* Bd, int d_out,
                                                              KeyTable keys) {
  const int R = keys.R;
  const long i = (long)blockIdx.x * kThreads + threadIdx.x;
  if (i >= (long)d_out * R) return;
  const int n = (int)(i / R), K = (int)(i % R);
  const int q = upper_index(keys.roff, keys.n_keys, K);
  const int r_q = keys.rank[q], roff = keys.roff[q];
  Bd[i] = B[(size_t)d_out * roff + (size_t)n * r_q + (K - roff)];
}

// h_p = s_q A_q x_p for every routed pair, row-major per pair position.
ContractArgs pair_h_args(const Problem& p, void* hp, int rpad) {
  ContractArgs c{};
  c.src = p.x;
  c.W = p.A;
  c.ldw = p.d_in;
  c.K = p.d_in;
  c.src_mode = kSrcPairList;
  c.k = p.k;
  c.alpha = p.alpha;
  c.plist = p.rt->pair_list;
  c.ppos = p.rt->row_pair;
  c.offsets = p.rt->offsets;
  c.row_token = p.rt->row_token;
  c.row_slots = p.rt->row_slots;
  c.out_row = hp;
  c.rpad = rpad;
  c.keys = p.keys;
  return c;
}

}  // namespace

size_t fwd_combined_ws_bytes(int T, int k, int d_out, int n_keys, int r_max) {
  return fwd_layout(T, k, d_out, n_keys, r_max, sizeof(float)).total;
}

size_t bwd_combined_ws_bytes(int T, int k, int d_in, int d_out, int n_keys, int r_max) {
  return bwd_layout(T, k, d_in, d_out, n_keys, r_max, sizeof(float)).total;
}

hipError_t launch_fwd_combined(const Problem& p, void* y, void* ws, hipStream_t stream) {
  const long P = (long)p.T * p.k;
  const int R = p.keys.R;
  const size_t es = p.dtype == ACE_BF16 ? 2 : 4;
  const int rpad = rank_pad(p.dtype, p.r_max);
  const FwdLayout L = fwd_layout(p.T, p.k, p.d_out, p.keys.n_keys, p.r_max, es);
  char* base = static_cast<char*>(ws);
  // the bf16 GEMM with LDS staging reads B^T rows [R][d_out]; the register
  // GEMM reads [d_out][R]
  const bool rows_op = p.dtype == ACE_BF16 && R % 8 == 0;
  hipError_t e = launch_prep(p, nullptr, rows_op ? base + L.Bm : nullptr, base + L.Hd,
                             (long)p.T * R * (long)es, stream);
  if (e != hipSuccess) return e;
  if (!rows_op) {
    const long n = (long)p.d_out * R;
    const int blocks = (int)((n + kThreads - 1) / kThreads);
    if (p.dtype == ACE_BF16)
      restride_b_kernel<__bf16><<<blocks, kThreads, 0, stream>>>(
          static_cast<const __bf16*>(p.B), reinterpret_cast<__bf16*>(base + L.Bm), p.d_out, p.keys);
    else
      restride_b_kernel<float><<<blocks, kThreads, 0, stream>>>(
          static_cast<const float*>(p.B), reinterpret_cast<float*>(base + L.Bm), p.d_out, p.keys);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  e = launch_contract(p.dtype, pair_h_args(p, base + L.hp, rpad), p.r_max, P, stream);
  if (e != hipSuccess) return e;
  e = launch_combine(p, base + L.hp, rpad, nullptr, 0, base + L.Hd, stream);
  if (e != hipSuccess) return e;
  DxArgs d{};
  d.dHf = base + L.Hd;
  d.At = base + L.Bm;
  d.A = base + L.Bm;
  d.dx = y;
  d.T = p.T;
  d.d_in = p.d_out;
  d.R = R;
  d.KR = R;
  return launch_dx_gemm(p.dtype, d, stream);
}

hipError_t launch_bwd_combined(const Problem& p, const void* dy, void* dx, float* dA, float* dB,
                               void* ws, hipStream_t stream) {
  const long P = (long)p.T * p.k;
  const size_t es = p.dtype == ACE_BF16 ? 2 : 4;
  const int rpad = rank_pad(p.dtype, p.r_max);
  const BwdLayout L = bwd_layout(p.T, p.k, p.d_in, p.d_out, p.keys.n_keys, p.r_max, es);
  char* base = static_cast<char*>(ws);
  const long ldh = (long)((((size_t)P) + 7) & ~(size_t)7);
  hipError_t e = launch_prep(p, base + L.At, base + L.Bt, nullptr, 0, stream);
  if (e != hipSuccess) return e;
  // h per pair position: the forward's (its workspace starts with it) or recomputed
  const void* hp = p.h_fwd;
  if (!hp) {
    hp = base + L.hp;
    e = launch_contract(p.dtype, pair_h_args(p, base + L.hp, rpad), p.r_max, P, stream);
    if (e != hipSuccess) return e;
  }
  e = launch_combine(p, hp, rpad, base + L.Ht, ldh, nullptr, stream);
  if (e != hipSuccess) return e;
  // dH_u = s B^T dOut[t_u], per row (for dx) and times w_p per pair position (for dA)
  ContractArgs c{};
  c.src = dy;
  c.W = base + L.Bt;
  c.ldw = p.d_out;
  c.K = p.d_out;
  c.src_mode = kSrcShared;
  c.k = p.k;
  c.alpha = p.alpha;
  c.pair_w = p.pair_w;
  c.offsets = p.rt->offsets;
  c.row_token = p.rt->row_token;
  c.row_slots = p.rt->row_slots;
  c.out_row = base + L.dHrow;
  c.rpad = rpad;
  c.out_t = base + L.dHw;
  c.ldh = ldh;
  c.out_t_pairs = 1;
  c.ppos = p.rt->row_pair;
  c.keys = p.keys;
  e = launch_contract(p.dtype, c, p.r_max, P, stream);
  if (e != hipSuccess) return e;
  // dx_p += w_p A_q^T dH_u for every slot of row u
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
  x.pair_w = p.pair_w;
  x.keys = p.keys;
  x.multi_slot = p.rt->mode == ACE_ROWS_GROUP_DEDUP;
  e = launch_expand(p.dtype, x, p.r_max, P, stream);
  if (e != hipSuccess) return e;
  GradArgs gr{};
  gr.x = p.x;
  gr.dy = dy;
  gr.Hw = base + L.Ht;
  gr.dHt = base + L.dHw;
  gr.ldh = ldh;
  gr.dA = dA;
  gr.dB = dB;
  gr.part = base + L.part;
  gr.offsets = p.rt->offsets;
  gr.row_token = p.rt->row_token;
  gr.row_slots = p.rt->row_slots;
  gr.ppos = p.rt->row_pair;
  gr.plist = p.rt->pair_list;
  gr.k = p.k;
  gr.d_in = p.d_in;
  gr.d_out = p.d_out;
  gr.per_pair = 1;
  gr.combined = 1;
  gr.keys = p.keys;
  return launch_grads(p.dtype, gr, p.r_max, P, stream);
}

}  // namespace ace
