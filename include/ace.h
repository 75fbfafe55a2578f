/*
 * ace.h -- C-ABI of libace, grouped adapter execution for MoE LoRA on MI355X.
 *
 * Method: ACE (Adapter Consolidation across Experts, arXiv 2609.06072).
 *   Sec. 3.1    expert-wise LoRA: a routed expert e adds p_e * B_e A_e x.
 *   Sec. 3.3    rank consolidation: a group G_g shares B_g A_g, with
 *               A_g in R^{r_g x d_in}, B_g in R^{d_out x r_g},
 *               r_g = sum of its members' ranks (same parameter budget).
 *   Sec. 3.4    shared adapter updates: expert e uses the adapter of g(e).
 *   Sec. 3.5    grouped adapter execution: for the active groups
 *               A(x) = { g(e) : e in R(x) } of a token, c_g(x) = B_g A_g x is
 *               computed once and handed to every routed expert of g.
 *   Appendix "Implementation Details": gate/up projections share the token
 *               input x (grouped execution applies); the down projection
 *               takes an expert-specific input per routed pair.
 *
 * Conventions for every call
 *   - Pointers marked "device" are HIP device pointers owned by the caller;
 *     "host" pointers are read during the call only.  The library keeps no
 *     pointer after it returns and allocates no device memory.
 *   - Every call that launches work is asynchronous on `stream` (a
 *     hipStream_t passed as void*, NULL = the null stream) and does not
 *     synchronise, except ace_routing_check.
 *   - Errors: arguments are validated on the host before anything is
 *     launched; a rejected call returns a negative ace_status, writes
 *     nothing, and ace_last_error() describes why.  A failed launch returns
 *     ACE_ERR_HIP.  Faults inside kernels surface at the caller's next sync.
 *   - Element types: ACE_F32 (float) or ACE_BF16 (bfloat16, RNE).  Matrix
 *     products accumulate in fp32 on the matrix cores.
 *   - Row alignment: d_in and d_out must be multiples of 8 (bf16) or 4
 *     (f32), and x, A, y, dy, dx must be 16-byte aligned.
 *   - Limits: 1 <= k <= 32, number of keys (experts or groups) <= 256,
 *     1 <= rank <= 256 per key, T*k < 2^31.
 *
 * Parameter layout (the caller's adapter tensors)
 *   Keys q = 0..n_keys-1 (groups for the grouped calls, experts for the
 *   expert-wise calls) with ranks r_q and rank offsets roff_q = sum_{q'<q} r_q',
 *   R = sum_q r_q:
 *     A  : [R, d_in] row-major; rows roff_q .. roff_q + r_q - 1 are A_q.
 *     B  : R * d_out elements; key q's block B_q in R^{d_out x r_q}, row-major,
 *          starts at element d_out * roff_q.
 *   Gradients dA, dB use the same layouts, in fp32.
 *   The LoRA scale of key q is s_q = alpha / r_q.
 *
 * Outputs of the forward (Sec. 3.4 with the router weight optional):
 *   y[t*k + j, :] += w[t, j] * s_q * B_q (A_q xin(t, j))   for every routed
 *   pair (t, j) with q = the key of expert topk_ids[t, j];
 *   xin(t, j) = x[t] (ACE_INPUT_SHARED) or x[t*k + j] (ACE_INPUT_PER_PAIR);
 *   w = 1 when pair_w is NULL.  With ACE_INPUT_COMBINED the same sum lands in
 *   y[t, :] (input x[t*k + j]), see ace_input_mode.
 */
#ifndef ACE_H_
#define ACE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ACE_OK = 0,
  ACE_ERR_INVALID_ARG = -1,  /* bad pointer, size, mode or range            */
  ACE_ERR_UNSUPPORTED = -2,  /* valid but outside the supported limits      */
  ACE_ERR_WORKSPACE = -3,    /* workspace missing or smaller than required  */
  ACE_ERR_HIP = -4           /* a HIP runtime call failed                   */
} ace_status;

typedef enum { ACE_F32 = 0, ACE_BF16 = 1 } ace_dtype;

typedef enum {
  /* one row per (token, active group): Sec. 3.5 grouped execution            */
  ACE_ROWS_GROUP_DEDUP = 0,
  /* one row per routed pair, keyed by its group: shared adapters run with the
     expert-wise execution pattern (the paper's "w/o grouped execution")      */
  ACE_ROWS_GROUP_PAIRS = 1,
  /* one row per routed pair, keyed by its expert: expert-wise LoRA, Sec. 3.1 */
  ACE_ROWS_EXPERT = 2
} ace_row_mode;

typedef enum {
  ACE_INPUT_SHARED = 0,   /* x is [T, d_in]; every routed expert sees x[t]        */
  ACE_INPUT_PER_PAIR = 1, /* x is [T*k, d_in]; pair (t,j) has its own row t*k+j   */
  /* x is [T*k, d_in] as for ACE_INPUT_PER_PAIR, but the output is combined per
     token with the routing weights: y is [T, d_out] and
       y[t] += sum_j w[t, j] * s_q * B_q (A_q x[t*k + j]).
     This is the down projection of an MoE layer whose expert outputs are
     summed with the weights p_e (Sec. 3.1): since that sum is linear, a
     (token, group) row evaluates its adapter once on the weighted sum of its
     pairs' inputs (Sec. 3.5 applied to the down projection).  dy and dx of
     the backward are [T, d_out] and [T*k, d_in].                              */
  ACE_INPUT_COMBINED = 2
} ace_input_mode;

typedef enum {
  ACE_OP_PERMUTE = 0,
  ACE_OP_FWD = 1,
  ACE_OP_BWD = 2,
  ACE_OP_CKA = 3   /* ace_pairwise_cka: T = probe rows N, k = 1, n_keys = E, r_max = rank */
} ace_op;

/*
 * Routing rows produced by ace_group_permute.  The caller allocates the
 * device arrays (sizes below, P = T*k) and keeps the struct alive while the
 * forward/backward calls that read it are in flight.  The host fields are
 * written by ace_group_permute and checked by the other calls.
 *
 * Rows are sorted by key, then token, then slot.  Row u serves token
 * row_token[u]; bit j of row_slots[u] is set for every slot j it serves.
 * The routed pairs sorted by (key, token, slot) are listed in pair_list; the
 * pairs of row u sit at positions row_pair[u] .. row_pair[u+1] (one per row
 * except in ACE_ROWS_GROUP_DEDUP mode, where a row serves every slot of its
 * token whose expert is in the group).
 * offsets[q] .. offsets[q+1] is key q's segment; offsets[n_keys] = U, the
 * number of rows (U <= P; in ACE_ROWS_GROUP_DEDUP mode U is the number of
 * distinct (token, group) pairs, Sec. 3.5).
 */
typedef struct ace_routing {
  int32_t* counts;     /* device [n_keys]    rows per key                           */
  int32_t* offsets;    /* device [n_keys+1]  exclusive prefix of counts             */
  int32_t* row_token;  /* device [P]         token of each row (entries >= U unused)*/
  uint32_t* row_slots; /* device [P]         slot mask of each row                  */
  int32_t* pair_row;   /* device [P]         row that serves pair t*k+j, -1 if dropped */
  int32_t* n_dropped;  /* device [1]         pairs dropped (id out of range or repeated) */
  int32_t* row_pair;   /* device [P+1]       position of row u's first pair in pair
                                             order (key, token, slot); [U] = number
                                             of routed pairs                          */
  int32_t* pair_list;  /* device [P]         pair t*k+j at each position in pair order */
  int32_t n_keys;      /* host: set by ace_group_permute                            */
  int32_t mode;        /* host: ace_row_mode used                                   */
  int32_t T, k;        /* host: problem size used                                   */
} ace_routing;

/*
 * Route expansion and permutation (Sec. 3.5, the active group set A(x)).
 *   topk_ids        device int32 [T, k]: routed expert of slot j of token t.
 *                   An id outside [0, E), or whose group is outside [0, G),
 *                   drops the pair (counted in rt->n_dropped).  The routed
 *                   experts of a token are a set (Sec. 3.1): an id equal to
 *                   one at a lower slot of the same token drops the pair too
 *                   (counted likewise), in every mode.
 *   expert_to_group device int32 [E]: g(e); may be NULL iff mode == ACE_ROWS_EXPERT.
 *   mode            row mode; n_keys = G for the group modes, E for ACE_ROWS_EXPERT.
 *   ws, ws_bytes    device scratch, at least
 *                   ace_workspace_bytes(ACE_OP_PERMUTE, T, k, 0, 0, n_keys, 0);
 *                   needs no initialisation.
 * Output arrays of rt are overwritten.  Bit-exact and deterministic.
 */
ace_status ace_group_permute(const int32_t* topk_ids, int32_t T, int32_t k, int32_t E,
                             const int32_t* expert_to_group, int32_t G, ace_row_mode mode,
                             ace_routing* rt, void* ws, size_t ws_bytes, void* stream);

/*
 * ace_group_permute for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): no workspace argument.  The permutation's scratch (its count
 * tables, ace_workspace_bytes(ACE_OP_PERMUTE, T, k, 0, 0, n_keys, 0) bytes)
 * is a static device array of ACE_PERMUTE_SCRATCH_BYTES in the library, one
 * per GPU, held until the process ends; its address is looked up on the
 * first call on each device.  Nothing is allocated and nothing needs
 * clearing (the tables are fully written before they are read).
 *   Arguments, outputs and errors as for ace_group_permute; a problem whose
 *   scratch exceeds ACE_PERMUTE_SCRATCH_BYTES returns ACE_ERR_UNSUPPORTED
 *   before anything is launched (4 MiB holds, e.g., T*k = 1M pairs over 64
 *   keys or 500K pairs over 256 keys).
 *   Calls on one GPU share its array: calls that overlap in time on the same
 *   GPU (different streams or threads) race and must not be issued.
 */
#define ACE_PERMUTE_SCRATCH_BYTES (4u << 20)
ace_status ace_group_permute_noalloc(const int32_t* topk_ids, int32_t T, int32_t k, int32_t E,
                                     const int32_t* expert_to_group, int32_t G,
                                     ace_row_mode mode, ace_routing* rt, void* stream);

/*
 * Both routings an ACE layer needs from one top-k routing (Sec. 3.5 for the
 * grouped gate/up projections; the down projection stays expert-wise, App. L):
 * group_rt in group_mode (ACE_ROWS_GROUP_DEDUP or ACE_ROWS_GROUP_PAIRS,
 * n_keys = G) and expert_rt in ACE_ROWS_EXPERT (n_keys = E), from one pass over
 * topk_ids.  The outputs are bit-identical to two ace_group_permute calls.
 *   group_rt, expert_rt  distinct structs with distinct device arrays.
 *   ws, ws_bytes         device scratch, at least
 *                        ace_workspace_bytes(ACE_OP_PERMUTE, T, k, 0, 0, G, 0) +
 *                        ace_workspace_bytes(ACE_OP_PERMUTE, T, k, 0, 0, E, 0);
 *                        4-byte aligned; needs no initialisation.
 * Other arguments and errors as for ace_group_permute.
 */
ace_status ace_group_expert_permute(const int32_t* topk_ids, int32_t T, int32_t k, int32_t E,
                                    const int32_t* expert_to_group, int32_t G,
                                    ace_row_mode group_mode, ace_routing* group_rt,
                                    ace_routing* expert_rt, void* ws, size_t ws_bytes,
                                    void* stream);

/*
 * Grouped LoRA forward (Sec. 3.4 output, Sec. 3.5 execution).
 *   group_rank  host int32 [G]: r_g, the consolidated rank of each group.
 *   alpha       LoRA scaling numerator (s_g = alpha / r_g).
 *   x           device [T, d_in] (shared) or [T*k, d_in] (per pair, combined), dtype.
 *   A, B        device, packed as described at the top, dtype.
 *   pair_w      device fp32 [T, k] or NULL (weight 1).
 *   rt          rows from ace_group_permute in ACE_ROWS_GROUP_DEDUP (requires
 *               ACE_INPUT_SHARED or ACE_INPUT_COMBINED) or ACE_ROWS_GROUP_PAIRS
 *               mode, with n_keys == G.
 *   y           device [T*k, d_out] ([T, d_out] for ACE_INPUT_COMBINED), dtype:
 *               accumulated (+=).
 *   ws          device scratch of at least
 *               ace_workspace_bytes(ACE_OP_FWD, T, k, d_in, d_out, G, max r_g)
 *               (it holds h = (alpha/r_g) A_g x per row, per routed pair for
 *               ACE_INPUT_COMBINED); no initialisation.
 * Two launches: the shrink h once per row of the permutation, then the
 * expand B_g h added into every slot the row serves.  ACE_INPUT_COMBINED:
 * h per routed pair, its weighted sum per row into dense per-token rows
 * [T, R], and y += those rows times B^T (a GEMM over K = R).
 */
ace_status ace_grouped_lora_fwd(ace_dtype dtype, ace_input_mode input_mode, int32_t T,
                                int32_t k, int32_t d_in, int32_t d_out, int32_t G,
                                const int32_t* group_rank, float alpha, const void* x,
                                const void* A, const void* B, const float* pair_w,
                                const ace_routing* rt, void* y, void* ws, size_t ws_bytes,
                                void* stream);

/*
 * Grouped LoRA backward: gradients of L = <dy, y_out> for the forward above
 * (Sec. 3.1.2 / 3.4: a shared adapter collects every routed pair of its group).
 *   h_fwd       NULL, or the workspace of the forward call made with the same
 *               arguments (it still holds h = (alpha/r_g) A_g x per row); the
 *               backward then reads h from it instead of recomputing it.
 *               Read only; must not be overwritten in between.
 *   dy          device [T*k, d_out] ([T, d_out] for ACE_INPUT_COMBINED), dtype.
 *   dx          device, shape of x, dtype: accumulated (+=).
 *   dA          device fp32 [R, d_in]: overwritten (a group with no rows gets 0).
 *   dB          device fp32, layout of B: overwritten.
 *   ws          device scratch of at least
 *               ace_workspace_bytes(ACE_OP_BWD, T, k, d_in, d_out, G, max r_g);
 *               needs no initialisation.
 * Deterministic: every output element is reduced in a fixed order.
 */
ace_status ace_grouped_lora_bwd(ace_dtype dtype, ace_input_mode input_mode, int32_t T,
                                int32_t k, int32_t d_in, int32_t d_out, int32_t G,
                                const int32_t* group_rank, float alpha, const void* x,
                                const void* A, const void* B, const float* pair_w,
                                const ace_routing* rt, const void* h_fwd, const void* dy,
                                void* dx, float* dA, float* dB, void* ws, size_t ws_bytes,
                                void* stream);

/*
 * Expert-wise LoRA (Sec. 3.1), the baseline that grouped execution replaces:
 * every expert owns a rank-`rank` adapter (s = alpha / rank), one row per
 * routed pair.  Arguments as for the grouped calls with n_keys = E; rt must
 * come from ace_group_permute in ACE_ROWS_EXPERT mode.
 */
ace_status ace_expertwise_lora_fwd(ace_dtype dtype, ace_input_mode input_mode, int32_t T,
                                   int32_t k, int32_t d_in, int32_t d_out, int32_t E,
                                   int32_t rank, float alpha, const void* x, const void* A,
                                   const void* B, const float* pair_w, const ace_routing* rt,
                                   void* y, void* ws, size_t ws_bytes, void* stream);

ace_status ace_expertwise_lora_bwd(ace_dtype dtype, ace_input_mode input_mode, int32_t T,
                                   int32_t k, int32_t d_in, int32_t d_out, int32_t E,
                                   int32_t rank, float alpha, const void* x, const void* A,
                                   const void* B, const float* pair_w, const ace_routing* rt,
                                   const void* h_fwd, const void* dy, void* dx, float* dA,
                                   float* dB, void* ws, size_t ws_bytes, void* stream);

/*
 * Adapted expert projection: the frozen expert GEMM of an MoE layer with the
 * adapter update added in its epilogue (Sec. 3.1 base projection plus the
 * Sec. 3.4 shared-adapter update, the adapter part evaluated as in Sec. 3.5):
 *   y[t*k + j, :] = W_e xin(t, j) + s_q B_q (A_q xin(t, j))
 * for every routed pair, e = topk_ids[t, j], q = expert_key[e], s_q =
 * alpha / r_q, xin as for the LoRA calls.  No router weight (gate and up
 * projections, and the down projection ahead of the weighted combine).
 * y is written, not accumulated: the separate adapter forward's
 * read-modify-write of y disappears.
 *   input_mode  ACE_INPUT_SHARED (x [T, d_in]) or ACE_INPUT_PER_PAIR
 *               (x [T*k, d_in]).
 *   W           device [E, d_out, d_in], dtype: expert e's frozen weight.
 *   expert_rt   rows from ace_group_permute in ACE_ROWS_EXPERT mode over E
 *               experts: the GEMM's row tiles (one expert per tile).
 *   n_keys      number of adapters; 0 runs the plain expert projection
 *               y = W_e xin (key_rank, expert_key, A, B, adapter_rt and ws
 *               are then ignored and may be NULL).
 *   key_rank    host int32 [n_keys]: rank r_q of each adapter.
 *   expert_key  host int32 [E]: adapter of each expert (its group g(e) for
 *               consolidated adapters, e itself for expert-wise LoRA).
 *   A, B        device, adapters in the packed layout at the top, dtype.
 *   adapter_rt  rows of the adapter's shrink h = s_q A_q xin, from
 *               ace_group_permute on the same topk_ids with expert_to_group
 *               = expert_key: ACE_ROWS_GROUP_DEDUP (grouped execution, once
 *               per (token, active group); needs ACE_INPUT_SHARED),
 *               ACE_ROWS_GROUP_PAIRS, or ACE_ROWS_EXPERT (expert-wise; then
 *               expert_key[e] == e; expert_rt itself may be passed).
 *               n_keys == adapter_rt->n_keys.
 *   y           device [T*k, d_out], dtype: the rows of routed pairs are
 *               written; rows of dropped pairs are left untouched.
 *   ws          device scratch of at least
 *               ace_workspace_bytes(ACE_OP_FWD, T, k, d_in, d_out, n_keys,
 *               max r_q) (h per adapter row); no initialisation.
 * Two launches: the shrink once per adapter row, then the expert GEMM whose
 * K loop runs over d_in (x against W_e) and then over r_q (h against B_q)
 * into the same fp32 accumulators; each output element is rounded once.
 * Deterministic.
 */
ace_status ace_moe_lora_fwd(ace_dtype dtype, ace_input_mode input_mode, int32_t T, int32_t k,
                            int32_t d_in, int32_t d_out, int32_t E, const void* x, const void* W,
                            const ace_routing* expert_rt, int32_t n_keys, const int32_t* key_rank,
                            const int32_t* expert_key, float alpha, const void* A, const void* B,
                            const ace_routing* adapter_rt, void* y, void* ws, size_t ws_bytes,
                            void* stream);

/*
 * Pairwise linear CKA of the expert adapters of one layer on a shared probe
 * set (Sec. 3.3, rank consolidation): the similarity that groups experts.
 * Every probe row goes through every adapter regardless of routing; with
 * Z_e the N x d_out matrix of rows (B_e A_e x_n)^T, centred over the probe
 * rows (Zc_e = H Z_e, H = I - 11^T/N),
 *   S[i][j] = ||Zc_i^T Zc_j||_F^2 / (||Zc_i^T Zc_i||_F ||Zc_j^T Zc_j||_F).
 * The LoRA scale is common to the experts of a layer and CKA is invariant to
 * it, so B_e A_e is used unscaled.  An expert whose centred output is
 * identically zero (B_e = 0, N < 2, ...) gets S = 0 in its row and column.
 *   X       device [N, d_in], dtype: the probe hidden states.
 *   A, B    device, the expert adapters in the packed layout at the top with
 *           E keys of rank `rank` (1 <= rank <= 64), dtype.
 *   S       device fp32 [E, E]: overwritten (symmetric, diagonal 1).
 *   ws      device scratch of at least
 *           ace_workspace_bytes(ACE_OP_CKA, N, 1, d_in, d_out, E, rank);
 *           no initialisation.
 * Evaluated through the rank-r identity
 *   ||Zc_i^T Zc_j||_F^2 = <G_i M_ij, M_ij G_j>_F,  M = Pc^T Pc,
 *   Pc = centred X A^T (N x E*rank),  G_e = B_e^T B_e,
 * which is exact up to rounding: X A^T on the matrix cores (fp32
 * accumulation), M in fp32, no N x d_out matrix formed.  Deterministic.
 */
ace_status ace_pairwise_cka(ace_dtype dtype, int32_t N, int32_t d_in, int32_t d_out, int32_t E,
                            int32_t rank, const void* X, const void* A, const void* B, float* S,
                            void* ws, size_t ws_bytes, void* stream);

/*
 * Expert grouping from the CKA matrix (appendices "Layer-wise graph
 * construction" and "Layer-wise grouping with the Louvain method").  Host
 * computations on host arrays; E <= 256.
 *
 * ace_similarity_graph: W[i][j] = max(0, (S[i][j] + S[j][i])/2 - b) for
 *   i != j, W[i][i] = 0, with b the median of the off-diagonal entries of
 *   (S + S^T)/2 (the mean of the two middle ones for an even count).
 *   S host fp32 [E, E]; W host fp64 [E, E] (overwritten).
 *
 * ace_louvain: groups the nodes of W by greedy modularity optimisation,
 *   Q = (1/2m) sum_ij (W_ij - gamma k_i k_j / 2m) [z_i == z_j]
 *   (k_i = sum_j W_ij, 2m = sum_ij W_ij; the paper uses gamma = 0.8).  Node i,
 *   in index order, leaves its community and joins the candidate (a community
 *   holding one of its neighbours, or its own) with the largest gain
 *   k_i,in(C) - gamma k_i tot(C) / 2m (ties to the lowest community id) when
 *   that gain beats staying; sweeps repeat until none moves, the communities
 *   become super-nodes and the next level starts; a level with no move ends
 *   it.  Sums run in index order, so the result is reproducible bit for bit.
 *   W host fp64 [E, E], symmetric, non-negative; groups host int32 [E]
 *   (out): numbered in order of their lowest expert; *n_groups (out) = G.
 *   A graph without edges leaves every expert alone (G = E).
 *
 * ace_group_anchors: the CKA centre of every group, the member with the
 *   largest summed similarity S[i][j] to the other members (ties to the
 *   lowest expert).  expert_to_group host int32 [E] with values in [0, G),
 *   every group non-empty; anchors host int32 [G] (out).
 */
ace_status ace_similarity_graph(const float* S, int32_t E, double* W);
ace_status ace_louvain(const double* W, int32_t E, double gamma, int32_t* groups,
                       int32_t* n_groups);
ace_status ace_group_anchors(const float* S, int32_t E, const int32_t* expert_to_group, int32_t G,
                             int32_t* anchors);

/*
 * Consolidated group adapters from the expert adapters (Sec. 3.3 rank
 * consolidation; group-anchor appendix).  Group g has rank
 * r_g = |G_g| * rank (the budget is unchanged) and its adapter starts from
 * its anchor expert a = anchors[g]:
 *   A_g rows 0 .. rank-1     = A_a
 *   A_g rows rank .. r_g-1   = the next r_g - rank rows of A_init (the
 *                              standard LoRA draw of the extra rank, group
 *                              by group in group order)
 *   B_g columns 0 .. rank-1  = (r_g / rank) * B_a, so that the group adapter
 *                              at scale alpha / r_g reproduces the anchor's
 *                              update at alpha / rank
 *   B_g other columns        = 0
 *   A, B      device, expert adapters (E keys of rank `rank`, packed layout
 *             above), dtype.
 *   expert_to_group, anchors  host int32 [E], [G] (every group non-empty, its
 *             anchor one of its members).
 *   A_init    device [(E - G) * rank, d_in], dtype; may be NULL when G == E.
 *   A_g, B_g  device, packed layout above with G keys of ranks r_g (the
 *             group blocks in group order), dtype: overwritten.  Their total
 *             rank is E * rank (the budget is unchanged).
 *   group_rank host int32 [G] (out) or NULL: r_g of every group, the ranks
 *             to pass to the grouped calls with A_g, B_g.
 * Asynchronous on `stream`; A_g and B_g must not overlap the inputs.
 * group_rank is written before the call returns.
 */
ace_status ace_consolidate_adapters(ace_dtype dtype, int32_t d_in, int32_t d_out, int32_t E,
                                    int32_t rank, const void* A, const void* B,
                                    const int32_t* expert_to_group, int32_t G,
                                    const int32_t* anchors, const void* A_init, void* A_g,
                                    void* B_g, int32_t* group_rank, void* stream);

/*
 * Device scratch needed by an op (bytes, rounded up to 256).  n_keys and
 * r_max bound the packed rank R <= n_keys * r_max; dtype-independent (sized
 * for fp32).  Pure host computation; (size_t)-1 for invalid arguments.
 */
size_t ace_workspace_bytes(ace_op op, int32_t T, int32_t k, int32_t d_in, int32_t d_out,
                           int32_t n_keys, int32_t r_max);

/*
 * Copies rt->n_dropped to *n_dropped after synchronising `stream`.  For
 * tests and debugging; the only call that blocks.
 */
ace_status ace_routing_check(const ace_routing* rt, int32_t* n_dropped, void* stream);

/* Message of the last failed call on this thread ("" if none). */
const char* ace_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ACE_H_ */
