"""Plain, slow, fp64 CPU oracle for ACE grouped adapter execution.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or run
this module: it exists so that tests/, the smoke check and the bench's CPU
baseline can check and time the HIP library against an independent statement
of what the method computes.  It shares no code with the library.

What it follows (arXiv 2609.06072):
  * Sec. 3.1, problem statement: an MoE layer routes input x to the expert set
    R(x) with router probabilities p_e(x); with expert-wise LoRA each routed
    expert adds  p_e(x) * Delta W_e x,  Delta W_e = B_e A_e  (rank r_e).
  * Sec. 3.1.1: the layer budget is sum_e (d_in + d_out) r_e.
  * Sec. 3.1.2: an adapter's gradient only collects routed tokens.
  * Sec. 3.3, rank consolidation: a group G_g shares Delta W_g = B_g A_g with
    A_g in R^{r_g x d_in}, B_g in R^{d_out x r_g}, r_g = sum_{e in G_g} r_e.
  * Sec. 3.4, shared adapter updates: expert e uses Delta W_{g(e)}.
  * Sec. 3.5, grouped adapter execution: for the active group set
    A(x) = { g(e) : e in R(x) }, c_g(x) = Delta W_g x is evaluated once per
    active group and reused by every routed expert of that group.
  * Appendix "Implementation Details": gate and up projections share the
    input x (grouped execution applies); the down projection takes the
    expert-specific h_e (one input row per routed pair).
  * Down projection, pre-combined form: the layer output combines the expert
    outputs linearly with p_e (Sec. 3.1), so the adapter part of the combined
    output is sum_{g in A(t)} s_g B_g A_g (sum_{j: g(e_tj) = g} p_tj h_tj):
    one input combination and one adapter evaluation per (token, active
    group).  The paper keeps down expert-wise; this identity is a reading of
    Sec. 3.1 and 3.5 together (its steps: precombined_delta).

Readings where the paper is silent (each is restated in the design notes):
  * LoRA scale s = alpha / r for each adapter (alpha = 16, the paper's
    "scaling factor"); a group adapter uses alpha / r_g.
  * The op adds Delta to a per-(token, slot) output Y[t*k + j]; an optional
    per-pair weight w[t, j] multiplies it (p_e of Sec. 3.1); default w = 1.
  * Backward is the derivative of L = <dY, Y_out>.  Y and dx accumulate,
    dA and dB are returned whole.
  * Row order of the permutation: by key, then token, then slot (ascending).
  * Routed ids outside [0, E) (and group ids outside [0, G)) drop the pair;
    so does an id that repeats one at a lower slot of the same token (R(x)
    is a set of experts).

Parameter layout (shared with the C-ABI, a convention of this project):
  A: [R, d_in], key q's block is rows roff_q .. roff_q + r_q  (A_q).
  B: flat, key q's block B_q in R^{d_out x r_q} row-major starts at d_out*roff_q.
  roff_q = sum_{q' < q} r_{q'}.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

ROWS_GROUP_DEDUP = 0
ROWS_GROUP_PAIRS = 1
ROWS_EXPERT = 2
INPUT_SHARED = 0
INPUT_PER_PAIR = 1
INPUT_COMBINED = 2   # per-pair input, output combined per token: [T, d_out]


# ---------------------------------------------------------------------------
# routing: which adapter serves each routed pair (Sec. 3.4), and the rows of
# grouped execution (Sec. 3.5)
# ---------------------------------------------------------------------------

def repeated_id(topk_ids, t: int, j: int) -> bool:
    """True when slot j of token t repeats an expert id listed at a lower
    slot of the same token.  The routed experts R(x) of Sec. 3.1 are a set,
    so such a pair is not part of the routing and is dropped."""
    e = int(topk_ids[t][j])
    return any(int(topk_ids[t][jj]) == e for jj in range(j))


def pair_keys(topk_ids: np.ndarray, E: int, expert_to_group: Optional[np.ndarray],
              G: int) -> np.ndarray:
    """Adapter key of every routed pair: g(e) for group keys, e itself for
    expert keys (expert_to_group None).  -1 marks a dropped pair (an id out
    of range, a group out of range, or an id repeated within the token)."""
    T, k = topk_ids.shape
    keys = np.full((T, k), -1, dtype=np.int64)
    for t in range(T):
        for j in range(k):
            e = int(topk_ids[t, j])
            if not 0 <= e < E or repeated_id(topk_ids, t, j):
                continue
            if expert_to_group is None:
                keys[t, j] = e
            else:
                g = int(expert_to_group[e])
                if 0 <= g < G:
                    keys[t, j] = g
    return keys


def permute(topk_ids: np.ndarray, E: int, expert_to_group: Optional[np.ndarray],
            G: int, mode: int) -> Dict[str, np.ndarray]:
    """Rows of the permuted problem.

    GROUP_DEDUP: one row per (token t, active group g in A(x_t)) -- Sec. 3.5's
      "once per active group"; its slot mask holds every j with g(e_tj) = g.
    GROUP_PAIRS / EXPERT: one row per routed pair (t, j), keyed by g(e_tj) or
      e_tj; mask = {j}.
    Rows are sorted by (key, token, slot).  Built by listing the rows and
    sorting them, not by histogram/scan.  Also lists the routed pairs in
    (key, token, slot) order (pair_list) and the position of each row's first
    pair in that list (row_pair, with row_pair[U] = number of pairs).
    """
    T, k = topk_ids.shape
    n_keys = E if mode == ROWS_EXPERT else G
    keys = pair_keys(topk_ids, E, None if mode == ROWS_EXPERT else expert_to_group, G)
    rows: List[Tuple[int, int, int, int]] = []   # (key, token, first slot, mask)
    for t in range(T):
        if mode == ROWS_GROUP_DEDUP:
            active: Dict[int, List[int]] = {}
            for j in range(k):
                q = int(keys[t, j])
                if q < 0:
                    continue
                if q not in active:
                    active[q] = [j, 0]
                active[q][1] |= 1 << j
            for q, (j0, m) in active.items():
                rows.append((q, t, j0, m))
        else:
            for j in range(k):
                q = int(keys[t, j])
                if q >= 0:
                    rows.append((q, t, j, 1 << j))
    rows.sort(key=lambda r: (r[0], r[1], r[2]))
    U = len(rows)
    counts = np.zeros(n_keys, dtype=np.int64)
    row_token = np.zeros(U, dtype=np.int64)
    row_slots = np.zeros(U, dtype=np.int64)
    pair_row = np.full(T * k, -1, dtype=np.int64)
    for u, (q, t, _j0, m) in enumerate(rows):
        counts[q] += 1
        row_token[u] = t
        row_slots[u] = m
        for j in range(k):
            if (m >> j) & 1:
                pair_row[t * k + j] = u
    offsets = np.zeros(n_keys + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    # The routed pairs themselves in (key, token, slot) order, listed and
    # sorted on their own; row_pair[u] = position of row u's first pair.
    pairs = sorted((int(keys[t, j]), t, j) for t in range(T) for j in range(k) if keys[t, j] >= 0)
    pair_list = np.array([t * k + j for (_q, t, j) in pairs], dtype=np.int64)
    position = {(q, t, j): i for i, (q, t, j) in enumerate(pairs)}
    row_pair = np.zeros(U + 1, dtype=np.int64)
    for u, (q, t, j0, _m) in enumerate(rows):
        row_pair[u] = position[(q, t, j0)]
    row_pair[U] = len(pairs)
    return {"counts": counts, "offsets": offsets, "row_token": row_token,
            "row_slots": row_slots, "pair_row": pair_row, "U": U,
            "row_pair": row_pair, "pair_list": pair_list}


# ---------------------------------------------------------------------------
# parameters
# ---------------------------------------------------------------------------

def rank_offsets(ranks: Sequence[int]) -> np.ndarray:
    r = np.asarray(ranks, dtype=np.int64)
    off = np.zeros(r.shape[0] + 1, dtype=np.int64)
    off[1:] = np.cumsum(r)
    return off


def unpack(A: np.ndarray, B: np.ndarray, ranks: Sequence[int], d_out: int
           ) -> Tuple[List[np.ndarray], List[np.ndarray]]:
    """Split packed parameters into A_q [r_q, d_in] and B_q [d_out, r_q]."""
    off = rank_offsets(ranks)
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64).reshape(-1)
    As, Bs = [], []
    for q, r in enumerate(ranks):
        r = int(r)
        As.append(A[off[q]:off[q] + r, :])
        Bs.append(B[d_out * off[q]: d_out * (off[q] + r)].reshape(d_out, r))
    return As, Bs


def pack_B(Bs: Sequence[np.ndarray]) -> np.ndarray:
    return np.concatenate([np.asarray(b, dtype=np.float64).reshape(-1) for b in Bs])


# ---------------------------------------------------------------------------
# forward / backward by definition (Sec. 3.1 and 3.4): one adapter
# application per routed pair, vectorised per adapter key with fp64 matmul
# ---------------------------------------------------------------------------

def _pairs_by_key(keys: np.ndarray, n_keys: int) -> List[np.ndarray]:
    flat = keys.reshape(-1)
    return [np.nonzero(flat == q)[0] for q in range(n_keys)]


def _inputs(x: np.ndarray, pairs: np.ndarray, k: int, input_mode: int) -> np.ndarray:
    return x[pairs // k] if input_mode == INPUT_SHARED else x[pairs]


def lora_delta(x, A, B, ranks, alpha, topk_ids, E, expert_to_group, G,
               input_mode=INPUT_SHARED, pair_w=None) -> np.ndarray:
    """Delta[t*k + j] = w_tj * (alpha / r_q) * B_q (A_q xin(t, j)),  q = key of
    the pair (g(e) for groups, e for experts).  Returns fp64 [T*k, d_out]; with
    INPUT_COMBINED (per-pair input) the per-token sum over the slots,
    sum_j Delta[t*k + j], as fp64 [T, d_out]."""
    x = np.asarray(x, dtype=np.float64)
    T, k = topk_ids.shape
    n_keys = len(ranks)
    d_out = int(np.asarray(B).size // max(1, int(np.sum(ranks))))
    As, Bs = unpack(A, B, ranks, d_out)
    keys = pair_keys(topk_ids, E, expert_to_group, G)
    w = np.ones(T * k) if pair_w is None else np.asarray(pair_w, np.float64).reshape(-1)
    out = np.zeros((T * k, d_out))
    for q, pairs in enumerate(_pairs_by_key(keys, n_keys)):
        if pairs.size == 0:
            continue
        s = alpha / float(ranks[q])
        xin = _inputs(x, pairs, k, input_mode)
        h = xin @ As[q].T                 # h = A_q x          (Sec. 3.1.3)
        c = h @ Bs[q].T                   # Delta W_q x = B_q h
        out[pairs] = (w[pairs] * s)[:, None] * c
    if input_mode == INPUT_COMBINED:
        return out.reshape(T, k, d_out).sum(axis=1)
    return out


def lora_grads(x, A, B, ranks, alpha, topk_ids, E, expert_to_group, G, dy,
               input_mode=INPUT_SHARED, pair_w=None):
    """Gradients of L = sum_{t,j} <dY[t*k+j], Delta[t*k+j]>.

    Per pair with key q, coefficient c = w * alpha / r_q and h = A_q xin:
      dB_q  += c * dY h^T                 [d_out, r_q]
      dA_q  += c * (B_q^T dY) xin^T       [r_q, d_in]
      dxin  += c * A_q^T B_q^T dY         (shared input: summed over slots)
    Only routed pairs contribute (Sec. 3.1.2).  With INPUT_COMBINED, dY is the
    gradient of the combined output [T, d_out], so every pair of token t sees
    dY[t].  Returns fp64 dx (shape of x), dA [R, d_in] and dB packed like B.
    """
    x = np.asarray(x, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    T, k = topk_ids.shape
    n_keys = len(ranks)
    d_out = dy.shape[1]
    As, Bs = unpack(A, B, ranks, d_out)
    keys = pair_keys(topk_ids, E, expert_to_group, G)
    w = np.ones(T * k) if pair_w is None else np.asarray(pair_w, np.float64).reshape(-1)
    dx = np.zeros_like(x)
    dAs = [np.zeros_like(a) for a in As]
    dBs = [np.zeros_like(b) for b in Bs]
    for q, pairs in enumerate(_pairs_by_key(keys, n_keys)):
        if pairs.size == 0:
            continue
        c = (w[pairs] * (alpha / float(ranks[q])))[:, None]
        xin = _inputs(x, pairs, k, input_mode)
        dyp = dy[pairs // k] if input_mode == INPUT_COMBINED else dy[pairs]
        g = c * dyp                        # weighted output gradient per pair
        h = xin @ As[q].T
        dBs[q] = g.T @ h
        dh = g @ Bs[q]
        dAs[q] = dh.T @ xin
        contrib = dh @ As[q]
        rows = pairs // k if input_mode == INPUT_SHARED else pairs
        np.add.at(dx, rows, contrib)
    dA = np.concatenate(dAs, axis=0) if dAs else np.zeros((0, x.shape[1]))
    return dx, dA, pack_B(dBs)


# ---------------------------------------------------------------------------
# grouped adapter execution, in the paper's steps (Sec. 3.5): form A(x),
# evaluate c_g(x) once per active group, hand it to every routed expert of g
# ---------------------------------------------------------------------------

def grouped_execution_delta(x, A, B, ranks, alpha, topk_ids, E, expert_to_group, G,
                            pair_w=None) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    T, k = topk_ids.shape
    d_out = int(np.asarray(B).size // max(1, int(np.sum(ranks))))
    As, Bs = unpack(A, B, ranks, d_out)
    rt = permute(topk_ids, E, expert_to_group, G, ROWS_GROUP_DEDUP)
    w = np.ones(T * k) if pair_w is None else np.asarray(pair_w, np.float64).reshape(-1)
    out = np.zeros((T * k, d_out))
    for g in range(G):
        lo, hi = int(rt["offsets"][g]), int(rt["offsets"][g + 1])
        if hi == lo:
            continue
        toks = rt["row_token"][lo:hi]
        cg = (x[toks] @ As[g].T) @ Bs[g].T * (alpha / float(ranks[g]))   # c_g once
        for i, u in enumerate(range(lo, hi)):
            m = int(rt["row_slots"][u])
            for j in range(k):
                if (m >> j) & 1:
                    p = int(toks[i]) * k + j
                    out[p] = w[p] * cg[i]
    return out


def precombined_delta(x, A, B, ranks, alpha, topk_ids, E, expert_to_group, G,
                      pair_w=None) -> np.ndarray:
    """Down projection with the combine moved in front of the adapter: for
    every (token, active group) row, z = sum over its slots j of w_tj h_tj
    (h = the per-pair input x[t*k + j]), then out[t] += s_g B_g (A_g z).
    Returns fp64 [T, d_out]."""
    x = np.asarray(x, dtype=np.float64)
    T, k = topk_ids.shape
    d_out = int(np.asarray(B).size // max(1, int(np.sum(ranks))))
    As, Bs = unpack(A, B, ranks, d_out)
    rt = permute(topk_ids, E, expert_to_group, G, ROWS_GROUP_DEDUP)
    w = np.ones(T * k) if pair_w is None else np.asarray(pair_w, np.float64).reshape(-1)
    out = np.zeros((T, d_out))
    for g in range(G):
        lo, hi = int(rt["offsets"][g]), int(rt["offsets"][g + 1])
        for u in range(lo, hi):
            t, m = int(rt["row_token"][u]), int(rt["row_slots"][u])
            z = np.zeros(x.shape[1])
            for j in range(k):
                if (m >> j) & 1:
                    z += w[t * k + j] * x[t * k + j]
            out[t] += (alpha / float(ranks[g])) * (Bs[g] @ (As[g] @ z))
    return out


# ---------------------------------------------------------------------------
# the adapted expert projection (Sec. 3.1): the frozen expert weight and the
# adapter update applied to the same input, y = (W_e + s_q B_q A_q) xin
# ---------------------------------------------------------------------------

def expert_projection(x, W, topk_ids, E, input_mode=INPUT_SHARED) -> np.ndarray:
    """Y[t*k + j] = W_e xin(t, j) with e = topk_ids[t, j] and W [E, d_out, d_in]
    (the frozen per-expert projection of Sec. 3.1).  Rows of dropped pairs
    (id outside [0, E) or repeated within the token) are zero.  Returns fp64 [T*k, d_out]."""
    x = np.asarray(x, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    T, k = topk_ids.shape
    out = np.zeros((T * k, W.shape[1]))
    ids = np.asarray(topk_ids).astype(np.int64).reshape(-1).copy()
    for t in range(T):
        for j in range(k):
            if repeated_id(topk_ids, t, j):
                ids[t * k + j] = -1
    for e in range(E):
        pairs = np.nonzero(ids == e)[0]
        if pairs.size:
            out[pairs] = _inputs(x, pairs, k, input_mode) @ W[e].T
    return out


def adapted_projection(x, W, A, B, ranks, alpha, topk_ids, E, expert_to_group, G,
                       input_mode=INPUT_SHARED) -> np.ndarray:
    """Y[t*k + j] = W_e xin(t, j) + (alpha / r_q) B_q (A_q xin(t, j)): the
    expert's frozen projection plus its adapter update (the adapter of the
    expert's group, or its own with expert keys), no router weight (gate and
    up projections, and the down projection before the combine).  Rows of
    dropped pairs are zero.  Returns fp64 [T*k, d_out]."""
    base = expert_projection(x, W, topk_ids, E, input_mode)
    return base + lora_delta(x, A, B, ranks, alpha, topk_ids, E, expert_to_group, G,
                             input_mode=input_mode)


# ---------------------------------------------------------------------------
# brute force: scalar Python loops straight from the definition (tiny inputs)
# ---------------------------------------------------------------------------

def brute_delta(x, A, B, ranks, alpha, topk_ids, E, expert_to_group, G,
                input_mode=INPUT_SHARED, pair_w=None):
    T, k = topk_ids.shape
    R = int(sum(ranks))
    d_out = len(B) // R
    d_in = len(A[0])
    off = [0]
    for r in ranks:
        off.append(off[-1] + int(r))
    combined = input_mode == INPUT_COMBINED
    out = [[0.0] * d_out for _ in range(T if combined else T * k)]
    for t in range(T):
        for j in range(k):
            e = int(topk_ids[t][j])
            if not 0 <= e < E or repeated_id(topk_ids, t, j):
                continue
            q = e if expert_to_group is None else int(expert_to_group[e])
            if not 0 <= q < len(ranks):
                continue
            r = int(ranks[q])
            xin = x[t] if input_mode == INPUT_SHARED else x[t * k + j]
            w = 1.0 if pair_w is None else float(pair_w[t][j])
            s = alpha / r
            h = [sum(float(A[off[q] + a][i]) * float(xin[i]) for i in range(d_in))
                 for a in range(r)]
            for n in range(d_out):
                acc = 0.0
                for a in range(r):
                    acc += float(B[d_out * off[q] + n * r + a]) * h[a]
                if combined:
                    out[t][n] += w * s * acc
                else:
                    out[t * k + j][n] = w * s * acc
    return np.array(out, dtype=np.float64)


def brute_adapted_projection(x, W, A, B, ranks, alpha, topk_ids, E, expert_to_group, G,
                             input_mode=INPUT_SHARED):
    """Scalar loops over the merged weight: y[n] = sum_i (W_e[n][i] +
    s_q sum_a B_q[n][a] A_q[a][i]) xin[i] (the adapter folded into the
    expert weight, as LoRA is merged for inference)."""
    T, k = topk_ids.shape
    d_out, d_in = len(W[0]), len(W[0][0])
    off = [0]
    for r in ranks:
        off.append(off[-1] + int(r))
    out = [[0.0] * d_out for _ in range(T * k)]
    for t in range(T):
        for j in range(k):
            e = int(topk_ids[t][j])
            if not 0 <= e < E or repeated_id(topk_ids, t, j):
                continue
            q = e if expert_to_group is None else int(expert_to_group[e])
            r = int(ranks[q])
            s = alpha / r
            xin = x[t] if input_mode == INPUT_SHARED else x[t * k + j]
            for n in range(d_out):
                acc = 0.0
                for i in range(d_in):
                    m = float(W[e][n][i])
                    for a in range(r):
                        m += s * float(B[d_out * off[q] + n * r + a]) * float(A[off[q] + a][i])
                    acc += m * float(xin[i])
                out[t * k + j][n] = acc
    return np.array(out, dtype=np.float64)


def brute_grads(x, A, B, ranks, alpha, topk_ids, E, expert_to_group, G, dy,
                input_mode=INPUT_SHARED, pair_w=None):
    T, k = topk_ids.shape
    R = int(sum(ranks))
    d_out = len(B) // R
    d_in = len(A[0])
    off = [0]
    for r in ranks:
        off.append(off[-1] + int(r))
    dx = [[0.0] * d_in for _ in range(len(x))]
    dA = [[0.0] * d_in for _ in range(R)]
    dB = [0.0] * (d_out * R)
    for t in range(T):
        for j in range(k):
            e = int(topk_ids[t][j])
            if not 0 <= e < E or repeated_id(topk_ids, t, j):
                continue
            q = e if expert_to_group is None else int(expert_to_group[e])
            if not 0 <= q < len(ranks):
                continue
            r = int(ranks[q])
            xr = t if input_mode == INPUT_SHARED else t * k + j
            w = 1.0 if pair_w is None else float(pair_w[t][j])
            c = w * alpha / r
            g = [float(v) for v in dy[t if input_mode == INPUT_COMBINED else t * k + j]]
            h = [sum(float(A[off[q] + a][i]) * float(x[xr][i]) for i in range(d_in))
                 for a in range(r)]
            bg = [sum(float(B[d_out * off[q] + n * r + a]) * g[n] for n in range(d_out))
                  for a in range(r)]
            for n in range(d_out):
                for a in range(r):
                    dB[d_out * off[q] + n * r + a] += c * g[n] * h[a]
            for a in range(r):
                for i in range(d_in):
                    dA[off[q] + a][i] += c * bg[a] * float(x[xr][i])
            for i in range(d_in):
                dx[xr][i] += c * sum(float(A[off[q] + a][i]) * bg[a] for a in range(r))
    return (np.array(dx, dtype=np.float64), np.array(dA, dtype=np.float64),
            np.array(dB, dtype=np.float64))


def rel_l2(a, ref) -> float:
    """||a - ref||_2 / ||ref||_2 over the whole tensor; inf if ref = 0 and a != 0."""
    a = np.asarray(a, dtype=np.float64).ravel()
    ref = np.asarray(ref, dtype=np.float64).ravel()
    nr = float(np.linalg.norm(ref))
    nd = float(np.linalg.norm(a - ref))
    if nr == 0.0:
        return 0.0 if nd == 0.0 else float("inf")
    return nd / nr
