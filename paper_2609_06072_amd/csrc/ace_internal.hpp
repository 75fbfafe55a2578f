// Host-side declarations shared by the C-ABI layer and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/ace.h"
#include "ace_device.hpp"

namespace ace {

// One adapted projection as the kernels see it.
struct Problem {
  int dtype;       // ACE_F32 / ACE_BF16
  int per_pair;    // ACE_INPUT_PER_PAIR
  int combined;    // ACE_INPUT_COMBINED: per-pair input, output combined per token
  int T, k, d_in, d_out;
  float alpha;
  const void* x;
  const void* A;
  const void* B;
  const float* pair_w;
  const ace_routing* rt;
  KeyTable keys;   // ranks and rank offsets of the n_keys adapters
  int r_max;
  const void* h_fwd = nullptr;  // backward: h per row from the forward workspace, or null
};

int permute_tokens_per_block(int k);
size_t permute_ws_bytes(int T, int k, int n_keys);
// One routing written by a permutation launch sequence: its row mode, key
// count, output arrays and workspace (permute_ws_bytes(T, k, n_keys)).
struct PermuteOut {
  int mode, n_keys;
  const ace_routing* rt;
  void* ws;
};
constexpr int kMaxPermPasses = 2;
hipError_t launch_permute(const int32_t* ids, int T, int k, int E, const int32_t* e2g, int G,
                          int npass, const PermuteOut* outs, hipStream_t stream);

// Source of the rows of a rank contraction.
constexpr int kSrcShared = 0;    // src[row_token[u]]
constexpr int kSrcPerPair = 1;   // src[t*k + j] (the row's single slot)
constexpr int kSrcPairList = 2;  // src[plist[u]], u a pair position (segments from ppos)

struct ContractArgs {
  const void* src;            // x or dY, rows of length K
  const void* W;              // weight row (roff_q + r) at W + (roff_q + r) * ldw
  int32_t ldw, K, src_mode, k;
  float alpha;
  const float* pair_w;
  int32_t out_w;              // multiply a single-pair row's result by its pair weight
  const int32_t* plist;       // kSrcPairList: pair at each position
  const int32_t* offsets;
  const int32_t* row_token;
  const uint32_t* row_slots;
  void* out_row;              // [U][rpad] or null
  int32_t rpad;
  void* out_t;                // [R][ldh] (column u - offsets[q]) or null
  long ldh;
  int32_t out_t_pairs;        // out_t holds one column per pair (times its weight):
                              //   column = pair position - first position of the key
  const int32_t* ppos;        // [U+1] first pair position of each row, or null (one per row)
  void* out_dense;            // [T * kslots][R] or null
  int32_t kslots;
  // row_sum (bf16, kSrcPairList): tiles hold whole rows; the results of a
  // row's pairs, times their weights, are summed in the epilogue and stored
  // per row (out_t column u - offsets[q], out_dense) -- dH_u = s B^T G_u
  int32_t row_sum;
  const int32_t* pair_row;    // row_sum: row serving each pair
  KeyTable keys;
};

struct ExpandArgs {
  const void* H;              // [U][rpad], scaled, zero beyond r_q
  int32_t rpad;
  const void* W;              // key q's rows start at W + w_key_mul * roff_q
  int32_t w_key_mul;
  int32_t w_stride_is_rank;   // row stride r_q (B_q) or R (A^T)
  const int32_t* offsets;
  const int32_t* row_token;
  const uint32_t* row_slots;
  int32_t k, n_out;
  void* out;                  // [T*k][n_out], accumulated
  const float* pair_w;        // or null (weight 1)
  int32_t multi_slot;         // rows may serve several slots (row-deduplicated grouping)
  int32_t nch;                // set by the launcher
  KeyTable keys;
};

int rank_blocks(int r_max);
int rank_pad(int dtype, int r_max);
hipError_t launch_contract(int dtype, const ContractArgs& a, int r_max, long P,
                           hipStream_t stream);
hipError_t launch_expand(int dtype, const ExpandArgs& a, int r_max, long P, hipStream_t stream);

size_t fwd_ws_bytes(int T, int k, int r_max);
hipError_t launch_fwd(const Problem& p, void* y, void* ws, hipStream_t stream);

// Shrink h = (alpha / r_q) A_q xin once per row of p.rt, into h [U][rpad]
// (the first launch of the forward).
hipError_t launch_shrink(const Problem& p, void* h, hipStream_t stream);

// Expert projection with the adapter update in its epilogue:
//   y[t*k + j] = W_e xin(t, j) + h[h_row[t*k + j]] B_q^T   (q = key_of[e])
struct MoeArgs {
  const void* x;              // [T][d_in] (shared) or [T*k][d_in] (per pair)
  const void* W;              // [E][d_out][d_in]
  const int32_t* offsets;     // expert routing (ACE_ROWS_EXPERT)
  const int32_t* row_token;
  const uint32_t* row_slots;
  int32_t E, k, d_in, d_out, per_pair;
  const void* H;              // [U'][rpad] scaled shrink per adapter row, or null (no adapter)
  int32_t rpad;
  const int32_t* h_row;       // adapter row of each pair (the adapter routing's pair_row)
  const void* B;              // key q: [d_out][r_q] at d_out * roff_q
  void* y;                    // [T*k][d_out], written
  int32_t nt;                 // column tiles (set by the launcher)
  KeyTable keys;              // adapter keys
  uint8_t key_of[kMaxKeys];   // adapter key of each expert
};
hipError_t launch_moe_gemm(int dtype, const MoeArgs& a, long P, hipStream_t stream);

// Backward helpers shared with the pre-combined mode.
//   prep: A^T [d_in][R] into At and B_q^T rows [R][d_out] into Bt (each
//         skipped when null), and zero_bytes of zeros at `zero` (16-byte
//         multiple inside a 256-byte padded region).
//   combine: h_u = sum over the pairs of row u of w_p hp[pos] (hp row-major
//         [P][rpad] per pair position), written to Ht [R][ldh] (column
//         u - offsets[q]) and/or Hd [T][R] (dense per token); either may be null.
hipError_t launch_prep(const Problem& p, void* At, void* Bt, void* zero, long zero_bytes,
                       hipStream_t stream);
hipError_t launch_combine(const Problem& p, const void* hp, int rpad, void* Ht, long ldh,
                          void* Hd, hipStream_t stream);

// Pre-combined input mode (ACE_INPUT_COMBINED).
size_t fwd_combined_ws_bytes(int T, int k, int d_out, int n_keys, int r_max);
size_t bwd_combined_ws_bytes(int T, int k, int d_in, int d_out, int n_keys, int r_max);
hipError_t launch_fwd_combined(const Problem& p, void* y, void* ws, hipStream_t stream);
hipError_t launch_bwd_combined(const Problem& p, const void* dy, void* dx, float* dA, float* dB,
                               void* ws, hipStream_t stream);

// Weight gradients dB_q = sum_p dY[p] Hw_p^T over the pairs of key q and
// dA_q = sum_u dH_u x_u^T over its rows (split over chunks, reduced in order).
struct GradArgs {
  const void* x;              // [T][d_in] (shared) or [T*k][d_in] (per pair)
  const void* dy;             // [T*k][d_out]
  const void* Hw;             // w_p s A x per pair: rank row roff_q + r at Hw + (roff_q + r) * ldh,
                              //   column = pair position - first pair position of key q
  const void* dHt;            // dH per row: same layout, column = u - offsets[q]
  long ldh;
  float* dA;                  // [R][d_in]
  float* dB;                  // key q: [d_out][r_q] at dB + d_out * roff_q
  void* part;                 // split partials
  const int32_t* offsets;
  const int32_t* row_token;
  const uint32_t* row_slots;
  const int32_t* ppos;        // [U+1] first pair position of each row, or null (one pair per row)
  const int32_t* plist;       // [P] pair (t*k + j) at each position, or null
  int32_t k, d_in, d_out, per_pair;
  int32_t combined;           // pre-combined input mode: dB runs over the rows (dy row =
                              //   token, Hw = h per row), dA over the pairs (x row = plist,
                              //   dHt = w dH per pair position)
  int32_t nbB, nbA;           // column blocks of dB / dA (set by the launcher)
  int32_t split;              // contraction indices per item: 0 (1024), 1024 or 2048
  int32_t split_b;            // the same for the dB items: 0 (= split), or a multiple of 64
                              //   from 512 to 4096
  int32_t* itab;              // item table written by the gradient launch for the reduce
                              //   (set by the launcher, after the partials)
  // phase 0: dB and dA items.  phase 1 (bf16, r_max <= 16): dB items only, each
  // also contracting its dY columns against B^T into dHp; phase 2: dA items only
  // (dH complete).  The split reduce runs after phases 0 and 2.
  int32_t phase;
  float* dHp;                 // phase 1: [nbB][npos][dhs] fp32, B_q^T dY per pair
                              //   position, the 128 columns of one dB column block
                              //   (wide items: [npos][nbW][64], 512 columns)
  long npos;
  int32_t dhs;                // rank stride of dHp (8 or 16; 64 for wide items)
  const void* Bt;             // phase 1: B^T [R][d_out], storage type
  KeyTable keys;
};

// dH per row from the phase-1 partials (bf16):
//   dH_u[r] = sum over the row's pairs p, in position order, of
//             (s_q * sum_cb dHp[cb][p][r]) * w_p
// stored per key as [r][u - offsets[q]] (dHt), and row-major [u][rpad] with
// zeros past r_q (dHrow) or in dense per-token rows (dHf), either may be null.
struct DhReduceArgs {
  const float* dHp;           // [nbB][npos][dhs], or [npos][nbB][64] with pos_major
  long npos;
  int32_t dhs, nbB;
  int32_t pos_major;          // partials of the wide items (pair-major runs)
  const int32_t* offsets;
  const int32_t* row_token;
  const uint32_t* row_slots;
  const int32_t* ppos;        // [U+1] first pair position of each row, or null (position = row)
  const int32_t* plist;       // pair at each position (weights of multi-pair rows)
  const float* pair_w;
  int32_t k;
  float alpha;
  void* dHt;
  long ldh;
  void* dHrow;
  int32_t rpad;
  void* dHf;                  // [T * kslots][R]: row tok * kslots + (kslots > 1 ? slot : 0)
  int32_t kslots;
  KeyTable keys;
};

// dx[t][c] += sum_K dHf[t][K] At[c][K mod R], K < KR (shared input).
struct DxArgs {
  const void* dHf;            // [T][KR]
  const void* At;             // [d_in][R]
  const void* A;              // [R][d_in]
  void* dx;                   // [T][d_in]
  int32_t T, d_in, R, KR;
};

size_t grads_part_bytes(int T, int k, int d_in, int d_out, int n_keys, int r_max);
hipError_t launch_grads(int dtype, GradArgs g, int r_max, long P, hipStream_t stream);
hipError_t launch_dh_reduce(const DhReduceArgs& d, long U, hipStream_t stream);
// Columns per dB column block (the dH partials of phase 1 are per block).
constexpr int kGradColBlk = 128;
// Phase 1 at ranks 33..64 with shared input and wide outputs (bf16): dB items
// of kWideCols dY columns whose dH partials ([nbW][npos][64] fp32, nbW =
// ceil(d_out / kWideCols)) replace the dH contraction; phase 2 and the
// split reduce as usual.
constexpr int kWideCols = 512;
hipError_t launch_grads_wide(GradArgs g, long P, hipStream_t stream);
hipError_t launch_dx_gemm(int dtype, const DxArgs& d, hipStream_t stream);

size_t bwd_ws_bytes(int T, int k, int d_in, int d_out, int n_keys, int R, int r_max);
hipError_t launch_bwd(const Problem& p, const void* dy, void* dx, float* dA, float* dB, void* ws,
                      hipStream_t stream);

// Pairwise linear CKA of expert adapters (ace_pairwise_cka).
struct CkaProblem {
  int dtype;
  int N, d_in, d_out, E, r;
  const void* X;   // [N][d_in]
  const void* A;   // [E*r][d_in]
  const void* B;   // expert e: [d_out][r] at d_out * r * e
  float* S;        // [E][E]
};
size_t cka_ws_bytes(int N, int d_out, int E, int r);
hipError_t launch_cka(const CkaProblem& p, void* ws, hipStream_t stream);

// Expert grouping (host) and adapter consolidation (device).
void similarity_graph(const float* S, int E, double* W);
int louvain(const double* W, int E, double gamma, int32_t* groups);  // returns G
void group_anchors(const float* S, int E, const int32_t* e2g, int G, int32_t* anchors);
struct ConsolidateProblem {
  int d_in, d_out, r;
  const void* A;
  const void* B;
  const void* A_init;
  void* Ag;
  void* Bg;
  KeyTable keys;            // group ranks r_g = |G_g| r and offsets
  const int32_t* anchor;    // host [G]
};
hipError_t launch_consolidate(int dtype, const ConsolidateProblem& p, hipStream_t stream);

// Number of compute units of the current device (cached per device).
int device_cu_count();

}  // namespace ace
