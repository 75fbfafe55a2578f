// C-ABI entry points of libace: argument validation on the host, then the
// kernel launches of permute.hip, lora_fwd.hip and lora_bwd.hip on the
// caller's stream.  No call allocates device memory or synchronises (except
// ace_routing_check).
#include <stdarg.h>
#include <stdio.h>

#include <cmath>
#include <mutex>
#include <string>
#include <vector>

#include "ace_internal.hpp"

namespace ace {

namespace {

thread_local std::string g_err;

ace_status fail(ace_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

ace_status ok() {
  g_err.clear();
  return ACE_OK;
}

ace_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(ACE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t round256(size_t b) { return (b + 255) & ~(size_t)255; }

// Scratch of ace_group_permute_noalloc: the permutation's cell tables live in
// this static device array instead of a caller workspace.  Every GPU the
// library runs on holds its own copy until the process ends.  In host code
// the name is only a stand-in: kernels get the device address obtained once
// per device with hipGetSymbolAddress.
constexpr size_t kNoAllocScratchBytes = (size_t)ACE_PERMUTE_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array (nullptr and the
// message set on failure).  Looked up once per device, with that device
// current, and kept.
void* device_scratch(ace_status* st) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    *st = fail(ACE_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    return nullptr;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    *st = fail(ACE_ERR_UNSUPPORTED, "device %d outside [0, %d)", dev, kMaxDevices);
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      *st = fail(ACE_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
      return nullptr;
    }
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

// Shared validation of the forward/backward calls; fills the Problem.
ace_status check_problem(Problem& p, ace_dtype dtype, ace_input_mode im, int32_t T, int32_t k,
                         int32_t d_in, int32_t d_out, int32_t n_keys, const int32_t* ranks,
                         int32_t uniform_rank, float alpha, const void* x, const void* A,
                         const void* B, const float* pair_w, const ace_routing* rt,
                         bool expertwise, bool any_rows = false) {
  if (dtype != ACE_F32 && dtype != ACE_BF16) return fail(ACE_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
  if (im != ACE_INPUT_SHARED && im != ACE_INPUT_PER_PAIR && im != ACE_INPUT_COMBINED)
    return fail(ACE_ERR_INVALID_ARG, "unknown input mode %d", (int)im);
  if (T < 0) return fail(ACE_ERR_INVALID_ARG, "T = %d < 0", T);
  if (k < 1 || k > kMaxK) return fail(ACE_ERR_UNSUPPORTED, "k = %d outside [1, %d]", k, kMaxK);
  if ((int64_t)T * k >= (int64_t)1 << 31) return fail(ACE_ERR_UNSUPPORTED, "T*k >= 2^31");
  const int vec = dtype == ACE_BF16 ? 8 : 4;
  if (d_in < 1 || d_out < 1) return fail(ACE_ERR_INVALID_ARG, "d_in = %d, d_out = %d", d_in, d_out);
  if (d_in % vec || d_out % vec)
    return fail(ACE_ERR_UNSUPPORTED, "d_in (%d) and d_out (%d) must be multiples of %d", d_in,
                d_out, vec);
  if (n_keys < 1 || n_keys > kMaxKeys)
    return fail(ACE_ERR_UNSUPPORTED, "%s count %d outside [1, %d]", expertwise ? "expert" : "group",
                n_keys, kMaxKeys);
  if (!expertwise && !ranks) return fail(ACE_ERR_INVALID_ARG, "group_rank is NULL");
  if (!std::isfinite(alpha)) return fail(ACE_ERR_INVALID_ARG, "alpha is not finite");
  if (!rt) return fail(ACE_ERR_INVALID_ARG, "routing is NULL");
  // row_pair has P + 1 entries: its last one (the pair count) exists at T = 0 too
  if (!rt->offsets || !rt->counts || !rt->row_pair)
    return fail(ACE_ERR_INVALID_ARG, "routing arrays are NULL");
  if (T > 0 && (!rt->row_token || !rt->row_slots || !rt->pair_list))
    return fail(ACE_ERR_INVALID_ARG, "routing arrays are NULL");
  if (rt->T != T || rt->k != k)
    return fail(ACE_ERR_INVALID_ARG, "routing was built for T=%d k=%d, call has T=%d k=%d", rt->T,
                rt->k, T, k);
  if (rt->n_keys != n_keys)
    return fail(ACE_ERR_INVALID_ARG, "routing has %d keys, call has %d", rt->n_keys, n_keys);
  if (any_rows) {
    if (rt->mode == ACE_ROWS_GROUP_DEDUP && im != ACE_INPUT_SHARED)
      return fail(ACE_ERR_INVALID_ARG, "ACE_ROWS_GROUP_DEDUP adapter rows need ACE_INPUT_SHARED");
    if (rt->mode != ACE_ROWS_GROUP_DEDUP && rt->mode != ACE_ROWS_GROUP_PAIRS &&
        rt->mode != ACE_ROWS_EXPERT)
      return fail(ACE_ERR_INVALID_ARG, "adapter routing has an unknown row mode %d", rt->mode);
  } else if (expertwise) {
    if (rt->mode != ACE_ROWS_EXPERT)
      return fail(ACE_ERR_INVALID_ARG, "expert-wise calls need ACE_ROWS_EXPERT routing");
  } else {
    if (rt->mode == ACE_ROWS_GROUP_DEDUP) {
      if (im == ACE_INPUT_PER_PAIR)
        return fail(ACE_ERR_INVALID_ARG,
                    "ACE_ROWS_GROUP_DEDUP needs ACE_INPUT_SHARED or ACE_INPUT_COMBINED");
    } else if (rt->mode != ACE_ROWS_GROUP_PAIRS) {
      return fail(ACE_ERR_INVALID_ARG, "grouped calls need group-keyed routing");
    }
  }
  if (!A || !B) return fail(ACE_ERR_INVALID_ARG, "A or B is NULL");
  if (T > 0 && !x) return fail(ACE_ERR_INVALID_ARG, "x is NULL");
  if (!aligned(A, 16) || !aligned(B, 16) || !aligned(x, 16))
    return fail(ACE_ERR_INVALID_ARG, "x, A and B must be 16-byte aligned");
  if (!aligned(pair_w, 4)) return fail(ACE_ERR_INVALID_ARG, "pair_w misaligned");
  p.keys = KeyTable{};
  p.keys.n_keys = n_keys;
  int R = 0, rmax = 0;
  for (int q = 0; q < n_keys; ++q) {
    const int r = expertwise ? uniform_rank : ranks[q];
    if (r < 1 || r > kMaxRank)
      return fail(ACE_ERR_UNSUPPORTED, "rank %d of key %d outside [1, %d]", r, q, kMaxRank);
    p.keys.rank[q] = r;
    p.keys.roff[q] = R;
    R += r;
    rmax = r > rmax ? r : rmax;
  }
  p.keys.roff[n_keys] = R;
  p.keys.R = R;
  p.r_max = rmax;
  p.dtype = dtype;
  p.per_pair = im == ACE_INPUT_PER_PAIR;
  p.combined = im == ACE_INPUT_COMBINED;
  p.T = T;
  p.k = k;
  p.d_in = d_in;
  p.d_out = d_out;
  p.alpha = alpha;
  p.x = x;
  p.A = A;
  p.B = B;
  p.pair_w = pair_w;
  p.rt = rt;
  return ok();
}

ace_status run_fwd(const Problem& p, void* y, void* ws, size_t ws_bytes, void* stream) {
  if (p.T > 0 && !y) return fail(ACE_ERR_INVALID_ARG, "y is NULL");
  if (!aligned(y, 16)) return fail(ACE_ERR_INVALID_ARG, "y must be 16-byte aligned");
  const size_t need = p.combined
                          ? fwd_combined_ws_bytes(p.T, p.k, p.d_out, p.keys.n_keys, p.r_max)
                          : fwd_ws_bytes(p.T, p.k, p.r_max);
  if (need > 0 && (!ws || ws_bytes < need))
    return fail(ACE_ERR_WORKSPACE, "forward needs %zu workspace bytes, got %zu", need,
                ws ? ws_bytes : (size_t)0);
  if (!aligned(ws, 256)) return fail(ACE_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (p.T == 0) return ok();
  const hipStream_t st = static_cast<hipStream_t>(stream);
  return hip_status(p.combined ? launch_fwd_combined(p, y, ws, st) : launch_fwd(p, y, ws, st),
                    "forward launch");
}

ace_status run_bwd(Problem& p, const void* h_fwd, const void* dy, void* dx, float* dA, float* dB,
                   void* ws, size_t ws_bytes, void* stream) {
  if (p.T > 0 && (!dy || !dx)) return fail(ACE_ERR_INVALID_ARG, "dy or dx is NULL");
  if (h_fwd && !aligned(h_fwd, 256))
    return fail(ACE_ERR_INVALID_ARG, "h_fwd must be a forward workspace (256-byte aligned)");
  p.h_fwd = h_fwd;
  if (!dA || !dB) return fail(ACE_ERR_INVALID_ARG, "dA or dB is NULL");
  if (!aligned(dy, 16) || !aligned(dx, 16))
    return fail(ACE_ERR_INVALID_ARG, "dy and dx must be 16-byte aligned");
  if (!aligned(dA, 4) || !aligned(dB, 4)) return fail(ACE_ERR_INVALID_ARG, "dA/dB misaligned");
  const size_t need =
      p.combined ? bwd_combined_ws_bytes(p.T, p.k, p.d_in, p.d_out, p.keys.n_keys, p.r_max)
                 : bwd_ws_bytes(p.T, p.k, p.d_in, p.d_out, p.keys.n_keys, p.keys.R, p.r_max);
  if (!ws || ws_bytes < need)
    return fail(ACE_ERR_WORKSPACE, "backward needs %zu workspace bytes, got %zu", need,
                ws ? ws_bytes : (size_t)0);
  if (!aligned(ws, 256)) return fail(ACE_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  const hipStream_t st = static_cast<hipStream_t>(stream);
  return hip_status(p.combined ? launch_bwd_combined(p, dy, dx, dA, dB, ws, st)
                               : launch_bwd(p, dy, dx, dA, dB, ws, st),
                    "backward launch");
}

ace_status run_moe_fwd(ace_dtype dtype, ace_input_mode im, int32_t T, int32_t k, int32_t d_in,
                       int32_t d_out, int32_t E, const void* x, const void* W,
                       const ace_routing* ert, int32_t n_keys, const int32_t* key_rank,
                       const int32_t* expert_key, float alpha, const void* A, const void* B,
                       const ace_routing* art, void* y, void* ws, size_t ws_bytes, void* stream) {
  if (dtype != ACE_F32 && dtype != ACE_BF16) return fail(ACE_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
  if (im != ACE_INPUT_SHARED && im != ACE_INPUT_PER_PAIR)
    return fail(ACE_ERR_INVALID_ARG, "input mode must be ACE_INPUT_SHARED or ACE_INPUT_PER_PAIR");
  if (T < 0) return fail(ACE_ERR_INVALID_ARG, "T = %d < 0", T);
  if (k < 1 || k > kMaxK) return fail(ACE_ERR_UNSUPPORTED, "k = %d outside [1, %d]", k, kMaxK);
  if ((int64_t)T * k >= (int64_t)1 << 31) return fail(ACE_ERR_UNSUPPORTED, "T*k >= 2^31");
  const int vec = dtype == ACE_BF16 ? 8 : 4;
  if (d_in < 1 || d_out < 1) return fail(ACE_ERR_INVALID_ARG, "d_in = %d, d_out = %d", d_in, d_out);
  if (d_in % vec || d_out % vec)
    return fail(ACE_ERR_UNSUPPORTED, "d_in (%d) and d_out (%d) must be multiples of %d", d_in,
                d_out, vec);
  if (E < 1 || E > kMaxKeys) return fail(ACE_ERR_UNSUPPORTED, "E = %d outside [1, %d]", E, kMaxKeys);
  if ((int64_t)E * d_out * d_in >= (int64_t)1 << 40)
    return fail(ACE_ERR_UNSUPPORTED, "expert weights too large");
  if (!ert || !ert->offsets || (T > 0 && (!ert->row_token || !ert->row_slots)))
    return fail(ACE_ERR_INVALID_ARG, "expert routing is NULL");
  if (ert->mode != ACE_ROWS_EXPERT || ert->n_keys != E)
    return fail(ACE_ERR_INVALID_ARG, "expert_rt must be ACE_ROWS_EXPERT routing over %d experts", E);
  if (ert->T != T || ert->k != k)
    return fail(ACE_ERR_INVALID_ARG, "expert routing was built for T=%d k=%d, call has T=%d k=%d",
                ert->T, ert->k, T, k);
  if (T > 0 && (!x || !W || !y)) return fail(ACE_ERR_INVALID_ARG, "x, W or y is NULL");
  if (!aligned(x, 16) || !aligned(W, 16) || !aligned(y, 16))
    return fail(ACE_ERR_INVALID_ARG, "x, W and y must be 16-byte aligned");
  if (n_keys < 0) return fail(ACE_ERR_INVALID_ARG, "n_keys = %d < 0", n_keys);
  MoeArgs a{};
  Problem p{};
  if (n_keys > 0) {
    if (!key_rank || !expert_key) return fail(ACE_ERR_INVALID_ARG, "key_rank or expert_key is NULL");
    ace_status s = check_problem(p, dtype, im, T, k, d_in, d_out, n_keys, key_rank, 0, alpha, x,
                                 A, B, nullptr, art, false, true);
    if (s != ACE_OK) return s;
    for (int e = 0; e < E; ++e) {
      const int q = expert_key[e];
      if (q < 0 || q >= n_keys)
        return fail(ACE_ERR_INVALID_ARG, "expert_key[%d] = %d outside [0, %d)", e, q, n_keys);
      if (art->mode == ACE_ROWS_EXPERT && q != e)
        return fail(ACE_ERR_INVALID_ARG, "expert-keyed adapter rows need expert_key[e] == e");
      a.key_of[e] = (uint8_t)q;
    }
    if (T > 0 && !art->pair_row) return fail(ACE_ERR_INVALID_ARG, "adapter routing arrays are NULL");
    const size_t need = fwd_ws_bytes(T, k, p.r_max);
    if (!ws || ws_bytes < need)
      return fail(ACE_ERR_WORKSPACE, "forward needs %zu workspace bytes, got %zu", need,
                  ws ? ws_bytes : (size_t)0);
    if (!aligned(ws, 256)) return fail(ACE_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  }
  if (T == 0) return ok();
  const hipStream_t st = static_cast<hipStream_t>(stream);
  a.x = x;
  a.W = W;
  a.offsets = ert->offsets;
  a.row_token = ert->row_token;
  a.row_slots = ert->row_slots;
  a.E = E;
  a.k = k;
  a.d_in = d_in;
  a.d_out = d_out;
  a.per_pair = im == ACE_INPUT_PER_PAIR;
  a.y = y;
  if (n_keys > 0) {
    hipError_t e = launch_shrink(p, ws, st);
    if (e != hipSuccess) return hip_status(e, "shrink launch");
    a.H = ws;
    a.rpad = rank_pad(dtype, p.r_max);
    a.h_row = art->pair_row;
    a.B = B;
    a.keys = p.keys;
  }
  return hip_status(launch_moe_gemm(dtype, a, (long)T * k, st), "expert GEMM launch");
}

}  // namespace

int device_cu_count() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

}  // namespace ace

using namespace ace;

extern "C" {

ace_status ace_group_permute(const int32_t* topk_ids, int32_t T, int32_t k, int32_t E,
                             const int32_t* expert_to_group, int32_t G, ace_row_mode mode,
                             ace_routing* rt, void* ws, size_t ws_bytes, void* stream) {
  if (!rt) return fail(ACE_ERR_INVALID_ARG, "routing is NULL");
  if (mode != ACE_ROWS_GROUP_DEDUP && mode != ACE_ROWS_GROUP_PAIRS && mode != ACE_ROWS_EXPERT)
    return fail(ACE_ERR_INVALID_ARG, "unknown row mode %d", (int)mode);
  if (T < 0) return fail(ACE_ERR_INVALID_ARG, "T = %d < 0", T);
  if (k < 1 || k > kMaxK) return fail(ACE_ERR_UNSUPPORTED, "k = %d outside [1, %d]", k, kMaxK);
  if ((int64_t)T * k >= (int64_t)1 << 31) return fail(ACE_ERR_UNSUPPORTED, "T*k >= 2^31");
  if (E < 1 || E > kMaxKeys) return fail(ACE_ERR_UNSUPPORTED, "E = %d outside [1, %d]", E, kMaxKeys);
  int n_keys = E;
  if (mode != ACE_ROWS_EXPERT) {
    if (G < 1 || G > kMaxKeys) return fail(ACE_ERR_UNSUPPORTED, "G = %d outside [1, %d]", G, kMaxKeys);
    if (!expert_to_group) return fail(ACE_ERR_INVALID_ARG, "expert_to_group is NULL");
    n_keys = G;
  }
  if (T > 0 && !topk_ids) return fail(ACE_ERR_INVALID_ARG, "topk_ids is NULL");
  // row_pair has P + 1 entries: the permutation writes its last one (the
  // pair count) at T = 0 too
  if (!rt->counts || !rt->offsets || !rt->n_dropped || !rt->row_pair)
    return fail(ACE_ERR_INVALID_ARG, "routing arrays are NULL");
  if (T > 0 && (!rt->row_token || !rt->row_slots || !rt->pair_row || !rt->pair_list))
    return fail(ACE_ERR_INVALID_ARG, "routing arrays are NULL");
  const size_t need = permute_ws_bytes(T, k, n_keys);
  if (need > 0 && (!ws || ws_bytes < need))
    return fail(ACE_ERR_WORKSPACE, "permute needs %zu workspace bytes, got %zu", need,
                ws ? ws_bytes : (size_t)0);
  if (!aligned(ws, 4)) return fail(ACE_ERR_WORKSPACE, "workspace misaligned");
  rt->n_keys = n_keys;
  rt->mode = mode;
  rt->T = T;
  rt->k = k;
  const PermuteOut out{(int)mode, n_keys, rt, ws};
  return hip_status(launch_permute(topk_ids, T, k, E, expert_to_group, G, 1, &out,
                                   static_cast<hipStream_t>(stream)),
                    "permute launch");
}

ace_status ace_group_permute_noalloc(const int32_t* topk_ids, int32_t T, int32_t k, int32_t E,
                                     const int32_t* expert_to_group, int32_t G, ace_row_mode mode,
                                     ace_routing* rt, void* stream) {
  // size check first (host only); ace_group_permute validates the rest
  if (T >= 0 && k >= 1 && k <= kMaxK && (int64_t)T * k < ((int64_t)1 << 31)) {
    const int n_keys = mode == ACE_ROWS_EXPERT ? E : G;
    if (n_keys >= 1 && n_keys <= kMaxKeys) {
      const size_t need = permute_ws_bytes(T, k, n_keys);
      if (need > kNoAllocScratchBytes)
        return fail(ACE_ERR_UNSUPPORTED,
                    "permutation of %d x %d pairs over %d keys needs %zu scratch bytes, the "
                    "static scratch holds %zu",
                    T, k, n_keys, need, kNoAllocScratchBytes);
    }
  }
  ace_status st = ACE_OK;
  void* ptr = device_scratch(&st);
  if (!ptr) return st;
  return ace_group_permute(topk_ids, T, k, E, expert_to_group, G, mode, rt, ptr,
                           kNoAllocScratchBytes, stream);
}

ace_status ace_group_expert_permute(const int32_t* topk_ids, int32_t T, int32_t k, int32_t E,
                                    const int32_t* expert_to_group, int32_t G,
                                    ace_row_mode group_mode, ace_routing* group_rt,
                                    ace_routing* expert_rt, void* ws, size_t ws_bytes,
                                    void* stream) {
  if (!group_rt || !expert_rt) return fail(ACE_ERR_INVALID_ARG, "routing is NULL");
  if (group_rt == expert_rt) return fail(ACE_ERR_INVALID_ARG, "the two routings are the same struct");
  if (group_mode != ACE_ROWS_GROUP_DEDUP && group_mode != ACE_ROWS_GROUP_PAIRS)
    return fail(ACE_ERR_INVALID_ARG, "group mode %d is not a group-keyed mode", (int)group_mode);
  if (T < 0) return fail(ACE_ERR_INVALID_ARG, "T = %d < 0", T);
  if (k < 1 || k > kMaxK) return fail(ACE_ERR_UNSUPPORTED, "k = %d outside [1, %d]", k, kMaxK);
  if ((int64_t)T * k >= (int64_t)1 << 31) return fail(ACE_ERR_UNSUPPORTED, "T*k >= 2^31");
  if (E < 1 || E > kMaxKeys) return fail(ACE_ERR_UNSUPPORTED, "E = %d outside [1, %d]", E, kMaxKeys);
  if (G < 1 || G > kMaxKeys) return fail(ACE_ERR_UNSUPPORTED, "G = %d outside [1, %d]", G, kMaxKeys);
  if (!expert_to_group) return fail(ACE_ERR_INVALID_ARG, "expert_to_group is NULL");
  if (T > 0 && !topk_ids) return fail(ACE_ERR_INVALID_ARG, "topk_ids is NULL");
  for (const ace_routing* rt : {(const ace_routing*)group_rt, (const ace_routing*)expert_rt}) {
    if (!rt->counts || !rt->offsets || !rt->n_dropped || !rt->row_pair)
      return fail(ACE_ERR_INVALID_ARG, "routing arrays are NULL");
    if (T > 0 && (!rt->row_token || !rt->row_slots || !rt->pair_row || !rt->pair_list))
      return fail(ACE_ERR_INVALID_ARG, "routing arrays are NULL");
  }
  // the group routing's cell tables first, the expert routing's after them
  const size_t need_g = round256(permute_ws_bytes(T, k, G));
  const size_t need = need_g + round256(permute_ws_bytes(T, k, E));
  if (!ws || ws_bytes < need)
    return fail(ACE_ERR_WORKSPACE, "permute needs %zu workspace bytes, got %zu", need,
                ws ? ws_bytes : (size_t)0);
  if (!aligned(ws, 4)) return fail(ACE_ERR_WORKSPACE, "workspace misaligned");
  group_rt->n_keys = G;
  group_rt->mode = group_mode;
  expert_rt->n_keys = E;
  expert_rt->mode = ACE_ROWS_EXPERT;
  for (ace_routing* rt : {group_rt, expert_rt}) {
    rt->T = T;
    rt->k = k;
  }
  const PermuteOut outs[2] = {{(int)group_mode, G, group_rt, ws},
                              {ACE_ROWS_EXPERT, E, expert_rt, static_cast<char*>(ws) + need_g}};
  return hip_status(launch_permute(topk_ids, T, k, E, expert_to_group, G, 2, outs,
                                   static_cast<hipStream_t>(stream)),
                    "permute launch");
}

ace_status ace_grouped_lora_fwd(ace_dtype dtype, ace_input_mode input_mode, int32_t T,
                                int32_t k, int32_t d_in, int32_t d_out, int32_t G,
                                const int32_t* group_rank, float alpha, const void* x,
                                const void* A, const void* B, const float* pair_w,
                                const ace_routing* rt, void* y, void* ws, size_t ws_bytes,
                                void* stream) {
  Problem p;
  ace_status s = check_problem(p, dtype, input_mode, T, k, d_in, d_out, G, group_rank, 0, alpha,
                               x, A, B, pair_w, rt, false);
  if (s != ACE_OK) return s;
  return run_fwd(p, y, ws, ws_bytes, stream);
}

ace_status ace_moe_lora_fwd(ace_dtype dtype, ace_input_mode input_mode, int32_t T, int32_t k,
                            int32_t d_in, int32_t d_out, int32_t E, const void* x, const void* W,
                            const ace_routing* expert_rt, int32_t n_keys, const int32_t* key_rank,
                            const int32_t* expert_key, float alpha, const void* A, const void* B,
                            const ace_routing* adapter_rt, void* y, void* ws, size_t ws_bytes,
                            void* stream) {
  return run_moe_fwd(dtype, input_mode, T, k, d_in, d_out, E, x, W, expert_rt, n_keys, key_rank,
                     expert_key, alpha, A, B, adapter_rt, y, ws, ws_bytes, stream);
}

ace_status ace_grouped_lora_bwd(ace_dtype dtype, ace_input_mode input_mode, int32_t T,
                                int32_t k, int32_t d_in, int32_t d_out, int32_t G,
                                const int32_t* group_rank, float alpha, const void* x,
                                const void* A, const void* B, const float* pair_w,
                                const ace_routing* rt, const void* h_fwd, const void* dy,
                                void* dx, float* dA, float* dB, void* ws, size_t ws_bytes,
                                void* stream) {
  Problem p;
  ace_status s = check_problem(p, dtype, input_mode, T, k, d_in, d_out, G, group_rank, 0, alpha,
                               x, A, B, pair_w, rt, false);
  if (s != ACE_OK) return s;
  return run_bwd(p, h_fwd, dy, dx, dA, dB, ws, ws_bytes, stream);
}

ace_status ace_expertwise_lora_fwd(ace_dtype dtype, ace_input_mode input_mode, int32_t T,
                                   int32_t k, int32_t d_in, int32_t d_out, int32_t E,
                                   int32_t rank, float alpha, const void* x, const void* A,
                                   const void* B, const float* pair_w, const ace_routing* rt,
                                   void* y, void* ws, size_t ws_bytes, void* stream) {
  Problem p;
  ace_status s = check_problem(p, dtype, input_mode, T, k, d_in, d_out, E, nullptr, rank, alpha,
                               x, A, B, pair_w, rt, true);
  if (s != ACE_OK) return s;
  return run_fwd(p, y, ws, ws_bytes, stream);
}

ace_status ace_expertwise_lora_bwd(ace_dtype dtype, ace_input_mode input_mode, int32_t T,
                                   int32_t k, int32_t d_in, int32_t d_out, int32_t E,
                                   int32_t rank, float alpha, const void* x, const void* A,
                                   const void* B, const float* pair_w, const ace_routing* rt,
                                   const void* h_fwd, const void* dy, void* dx, float* dA,
                                   float* dB, void* ws, size_t ws_bytes, void* stream) {
  Problem p;
  ace_status s = check_problem(p, dtype, input_mode, T, k, d_in, d_out, E, nullptr, rank, alpha,
                               x, A, B, pair_w, rt, true);
  if (s != ACE_OK) return s;
  return run_bwd(p, h_fwd, dy, dx, dA, dB, ws, ws_bytes, stream);
}

ace_status ace_pairwise_cka(ace_dtype dtype, int32_t N, int32_t d_in, int32_t d_out, int32_t E,
                            int32_t rank, const void* X, const void* A, const void* B, float* S,
                            void* ws, size_t ws_bytes, void* stream) {
  if (dtype != ACE_F32 && dtype != ACE_BF16) return fail(ACE_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
  if (N < 0) return fail(ACE_ERR_INVALID_ARG, "N = %d < 0", N);
  const int vec = dtype == ACE_BF16 ? 8 : 4;
  if (d_in < 1 || d_out < 1) return fail(ACE_ERR_INVALID_ARG, "d_in = %d, d_out = %d", d_in, d_out);
  if (d_in % vec) return fail(ACE_ERR_UNSUPPORTED, "d_in (%d) must be a multiple of %d", d_in, vec);
  if (E < 1 || E > kMaxKeys) return fail(ACE_ERR_UNSUPPORTED, "expert count %d outside [1, %d]", E, kMaxKeys);
  if (rank < 1 || rank > 64) return fail(ACE_ERR_UNSUPPORTED, "rank %d outside [1, 64]", rank);
  if ((int64_t)N * E * rank >= (int64_t)1 << 40) return fail(ACE_ERR_UNSUPPORTED, "probe too large");
  if (!A || !B || !S || (N > 0 && !X)) return fail(ACE_ERR_INVALID_ARG, "NULL argument");
  if (!aligned(X, 16) || !aligned(A, 16)) return fail(ACE_ERR_INVALID_ARG, "X and A must be 16-byte aligned");
  if (!aligned(S, 4) || !aligned(B, dtype == ACE_BF16 ? 2 : 4)) return fail(ACE_ERR_INVALID_ARG, "B or S misaligned");
  const size_t need = cka_ws_bytes(N, d_out, E, rank);
  if (!ws || ws_bytes < need)
    return fail(ACE_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", ws_bytes, need);
  CkaProblem p{};
  p.dtype = dtype;
  p.N = N;
  p.d_in = d_in;
  p.d_out = d_out;
  p.E = E;
  p.r = rank;
  p.X = X;
  p.A = A;
  p.B = B;
  p.S = S;
  return hip_status(launch_cka(p, ws, static_cast<hipStream_t>(stream)), "pairwise cka launch");
}

ace_status ace_similarity_graph(const float* S, int32_t E, double* W) {
  if (E < 1 || E > kMaxKeys) return fail(ACE_ERR_UNSUPPORTED, "expert count %d outside [1, %d]", E, kMaxKeys);
  if (!S || !W) return fail(ACE_ERR_INVALID_ARG, "NULL argument");
  for (int64_t i = 0; i < (int64_t)E * E; ++i)
    if (!std::isfinite(S[i])) return fail(ACE_ERR_INVALID_ARG, "S[%lld] is not finite", (long long)i);
  similarity_graph(S, E, W);
  return ok();
}

ace_status ace_louvain(const double* W, int32_t E, double gamma, int32_t* groups,
                       int32_t* n_groups) {
  if (E < 1 || E > kMaxKeys) return fail(ACE_ERR_UNSUPPORTED, "expert count %d outside [1, %d]", E, kMaxKeys);
  if (!W || !groups || !n_groups) return fail(ACE_ERR_INVALID_ARG, "NULL argument");
  if (!std::isfinite(gamma) || gamma < 0.0) return fail(ACE_ERR_INVALID_ARG, "gamma must be finite and >= 0");
  for (int i = 0; i < E; ++i)
    for (int j = 0; j < E; ++j) {
      const double w = W[(size_t)i * E + j];
      if (!std::isfinite(w) || w < 0.0 || w != W[(size_t)j * E + i])
        return fail(ACE_ERR_INVALID_ARG, "W must be finite, non-negative and symmetric (entry %d,%d)", i, j);
    }
  *n_groups = louvain(W, E, gamma, groups);
  return ok();
}

static ace_status check_groups(int32_t E, const int32_t* e2g, int32_t G) {
  if (E < 1 || E > kMaxKeys) return fail(ACE_ERR_UNSUPPORTED, "expert count %d outside [1, %d]", E, kMaxKeys);
  if (!e2g) return fail(ACE_ERR_INVALID_ARG, "expert_to_group is NULL");
  if (G < 1 || G > E) return fail(ACE_ERR_INVALID_ARG, "group count %d outside [1, %d]", G, E);
  std::vector<int> size(G, 0);
  for (int e = 0; e < E; ++e) {
    if (e2g[e] < 0 || e2g[e] >= G) return fail(ACE_ERR_INVALID_ARG, "group %d of expert %d outside [0, %d)", e2g[e], e, G);
    ++size[e2g[e]];
  }
  for (int g = 0; g < G; ++g)
    if (!size[g]) return fail(ACE_ERR_INVALID_ARG, "group %d has no expert", g);
  return ok();
}

ace_status ace_group_anchors(const float* S, int32_t E, const int32_t* expert_to_group, int32_t G,
                             int32_t* anchors) {
  ace_status s = check_groups(E, expert_to_group, G);
  if (s != ACE_OK) return s;
  if (!S || !anchors) return fail(ACE_ERR_INVALID_ARG, "NULL argument");
  group_anchors(S, E, expert_to_group, G, anchors);
  return ok();
}

ace_status ace_consolidate_adapters(ace_dtype dtype, int32_t d_in, int32_t d_out, int32_t E,
                                    int32_t rank, const void* A, const void* B,
                                    const int32_t* expert_to_group, int32_t G,
                                    const int32_t* anchors, const void* A_init, void* A_g,
                                    void* B_g, int32_t* group_rank, void* stream) {
  if (dtype != ACE_F32 && dtype != ACE_BF16) return fail(ACE_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
  ace_status s = check_groups(E, expert_to_group, G);
  if (s != ACE_OK) return s;
  const int vec = dtype == ACE_BF16 ? 8 : 4;
  if (d_in < 1 || d_out < 1) return fail(ACE_ERR_INVALID_ARG, "d_in = %d, d_out = %d", d_in, d_out);
  if (d_in % vec) return fail(ACE_ERR_UNSUPPORTED, "d_in (%d) must be a multiple of %d", d_in, vec);
  if (rank < 1 || rank > kMaxRank) return fail(ACE_ERR_UNSUPPORTED, "rank %d outside [1, %d]", rank, kMaxRank);
  if (!A || !B || !A_g || !B_g || !anchors || (G < E && !A_init))
    return fail(ACE_ERR_INVALID_ARG, "NULL argument");
  if (!aligned(A, 16) || !aligned(A_g, 16) || !aligned(A_init, 16))
    return fail(ACE_ERR_INVALID_ARG, "A, A_init and A_g must be 16-byte aligned");
  ConsolidateProblem p{};
  p.d_in = d_in;
  p.d_out = d_out;
  p.r = rank;
  p.A = A;
  p.B = B;
  p.A_init = A_init;
  p.Ag = A_g;
  p.Bg = B_g;
  p.anchor = anchors;
  p.keys.n_keys = G;
  std::vector<int> size(G, 0);
  for (int e = 0; e < E; ++e) ++size[expert_to_group[e]];
  int R = 0;
  for (int g = 0; g < G; ++g) {
    if (anchors[g] < 0 || anchors[g] >= E || expert_to_group[anchors[g]] != g)
      return fail(ACE_ERR_INVALID_ARG, "anchor %d of group %d is not one of its experts", anchors[g], g);
    p.keys.rank[g] = size[g] * rank;
    p.keys.roff[g] = R;
    R += size[g] * rank;
  }
  p.keys.roff[G] = R;
  p.keys.R = R;
  if (group_rank)
    for (int g = 0; g < G; ++g) group_rank[g] = p.keys.rank[g];
  return hip_status(launch_consolidate(dtype, p, static_cast<hipStream_t>(stream)),
                    "consolidate launch");
}

size_t ace_workspace_bytes(ace_op op, int32_t T, int32_t k, int32_t d_in, int32_t d_out,
                           int32_t n_keys, int32_t r_max) {
  if (T < 0 || k < 1 || k > kMaxK || n_keys < 1 || n_keys > kMaxKeys) {
    fail(ACE_ERR_INVALID_ARG, "invalid workspace query");
    return (size_t)-1;
  }
  switch (op) {
    case ACE_OP_PERMUTE:
      return round256(permute_ws_bytes(T, k, n_keys));
    case ACE_OP_FWD:
      if (r_max < 1 || r_max > kMaxRank) {
        fail(ACE_ERR_INVALID_ARG, "invalid workspace query");
        return (size_t)-1;
      }
      {
        // covers every input mode (the pre-combined one also needs d_out)
        const size_t a = fwd_ws_bytes(T, k, r_max);
        const size_t b = fwd_combined_ws_bytes(T, k, d_out > 0 ? d_out : 0, n_keys, r_max);
        return round256(a > b ? a : b);
      }
    case ACE_OP_BWD:
      if (d_in < 1 || d_out < 1 || r_max < 1 || r_max > kMaxRank) {
        fail(ACE_ERR_INVALID_ARG, "invalid workspace query");
        return (size_t)-1;
      }
      {
        const size_t a = bwd_ws_bytes(T, k, d_in, d_out, n_keys, n_keys * r_max, r_max);
        const size_t b = bwd_combined_ws_bytes(T, k, d_in, d_out, n_keys, r_max);
        return round256(a > b ? a : b);
      }
    case ACE_OP_CKA:
      if (d_in < 1 || d_out < 1 || r_max < 1 || r_max > 64) {
        fail(ACE_ERR_INVALID_ARG, "invalid workspace query");
        return (size_t)-1;
      }
      return round256(cka_ws_bytes(T, d_out, n_keys, r_max));
  }
  fail(ACE_ERR_INVALID_ARG, "unknown op %d", (int)op);
  return (size_t)-1;
}

ace_status ace_routing_check(const ace_routing* rt, int32_t* n_dropped, void* stream) {
  if (!rt || !rt->n_dropped || !n_dropped) return fail(ACE_ERR_INVALID_ARG, "NULL argument");
  hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_status(e, "stream synchronize");
  return hip_status(hipMemcpy(n_dropped, rt->n_dropped, sizeof(int32_t), hipMemcpyDeviceToHost),
                    "copy n_dropped");
}

const char* ace_last_error(void) { return g_err.c_str(); }

}  // extern "C"
