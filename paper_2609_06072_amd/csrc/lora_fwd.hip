// Grouped LoRA forward (Sec. 3.4 shared-adapter output executed as in
// Sec. 3.5): per row of the permutation -- one per (token, active group) --
//   H = (alpha / r_q) A_q x            contract kernel, once per row
//   y[t*k + j] += w_tj B_q H            expand kernel, for every slot of the row
// H (U x r_max, a few MB) is the only intermediate in the workspace.
#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

size_t fwd_ws_bytes(int T, int k, int r_max) {
  const size_t P = (size_t)T * k;
  return (P * (size_t)rank_pad(ACE_F32, r_max) * sizeof(float) + 255) & ~(size_t)255;
}

hipError_t launch_shrink(const Problem& p, void* h, hipStream_t stream) {
  ContractArgs c{};
  c.src = p.x;
  c.W = p.A;
  c.ldw = p.d_in;
  c.K = p.d_in;
  c.src_mode = p.per_pair ? kSrcPerPair : kSrcShared;
  c.k = p.k;
  c.alpha = p.alpha;
  c.pair_w = nullptr;
  c.offsets = p.rt->offsets;
  c.row_token = p.rt->row_token;
  c.row_slots = p.rt->row_slots;
  c.out_row = h;
  c.rpad = rank_pad(p.dtype, p.r_max);
  c.keys = p.keys;
  return launch_contract(p.dtype, c, p.r_max, (long)p.T * p.k, stream);
}

hipError_t launch_fwd(const Problem& p, void* y, void* ws, hipStream_t stream) {
  const long P = (long)p.T * p.k;
  const int rpad = rank_pad(p.dtype, p.r_max);
  hipError_t e = launch_shrink(p, ws, stream);
  if (e != hipSuccess) return e;
  ExpandArgs x{};
  x.H = ws;
  x.rpad = rpad;
  x.W = p.B;
  x.w_key_mul = p.d_out;
  x.w_stride_is_rank = 1;
  x.offsets = p.rt->offsets;
  x.row_token = p.rt->row_token;
  x.row_slots = p.rt->row_slots;
  x.k = p.k;
  x.n_out = p.d_out;
  x.out = y;
  x.pair_w = p.pair_w;
  x.keys = p.keys;
  x.multi_slot = p.rt->mode == ACE_ROWS_GROUP_DEDUP;
  return launch_expand(p.dtype, x, p.r_max, P, stream);
}

}  // namespace ace
