"""Plain fp64 CPU oracle for ACE's consolidation pipeline.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or run
this module: it exists so that tests/, the smoke check and the bench's CPU
baseline can check and time the library against an independent statement of
what the method computes.  It shares no code with the library.

What it follows (arXiv 2609.06072):
  * Sec. 3.3, rank consolidation: the same probe inputs x_1 .. x_N go through
    every expert adapter of a layer regardless of routing; expert e's
    adapter-induced representation is Z_e, the N x d_out matrix whose row n is
    (Delta W_e x_n)^T, Delta W_e = B_e A_e.  Z_e is mean-centred over the
    probe rows (H Z_e with H = I - 11^T / N), and two experts are compared with
    linear CKA:
        s_ij = ||Zc_i^T Zc_j||_F^2 / (||Zc_i^T Zc_i||_F ||Zc_j^T Zc_j||_F).
  * Appendix "Layer-wise graph construction": S is symmetrised, its diagonal
    set to zero, and W_ij = max(0, S_ij - b) with b the median of the
    off-diagonal entries.
  * Appendix "Layer-wise grouping with the Louvain method": greedy local
    moves on the weighted modularity
        Q = (1/2m) sum_ij (W_ij - gamma k_i k_j / 2m) [z_i == z_j]
    with gain  k_i,in(C) - gamma k_i tot(C) / 2m  for moving node i into C,
    then coarsening into super-nodes, repeated; gamma = 0.8 in the paper.
  * Sec. 3.3 and the appendix on group anchors: a group adapter has rank
    r_g = sum of its members' ranks; it is initialised from the CKA-centre
    expert of the group (the member most similar to the others), the
    remaining rank dimensions take standard LoRA initialisation.

Readings where the paper is silent (each is restated in the design notes):
  * The LoRA scale of the expert adapters (alpha / r, equal for every expert of
    the layer) multiplies every Z_e alike; CKA is invariant to it, so Z_e
    uses B_e A_e without the scale.
  * An expert whose centred output is identically zero has no defined CKA:
    its row and column of S are 0, the diagonal included.
  * Louvain order: nodes are visited in index order; after removing node i
    from its community, every community holding a neighbour of i and i's own
    community are candidates; the candidate with the largest gain wins (ties
    to the lowest community id), and i moves only if that gain is strictly
    larger than the gain of staying.  Sweeps repeat until one moves nothing;
    the communities then become super-nodes (numbered by their lowest
    member) and the next level starts; the algorithm ends at a level with no
    move.  Final groups are numbered in order of their lowest expert.
    Degrees, 2m, k_i,in and the coarse weights are summed in index order
    (the gain comparisons decide the partition, so the order is fixed).
  * The CKA centre of a group is the member with the largest sum of CKA
    similarities to the other members (ties to the lowest index).
  * The group adapter keeps the anchor's update exactly: rank rows 0 .. r-1 of
    A_g are A_anchor, columns 0 .. r-1 of B_g are (r_g / r) B_anchor (so that
    (alpha / r_g) B_g A_g = (alpha / r) B_anchor A_anchor), the other rows of
    A_g come from a standard LoRA draw supplied by the caller and the other
    columns of B_g are zero.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np


# ---------------------------------------------------------------------------
# Sec. 3.3: adapter-induced representations and linear CKA
# ---------------------------------------------------------------------------

def adapter_outputs(X: np.ndarray, A: np.ndarray, B: np.ndarray, E: int, r: int) -> List[np.ndarray]:
    """Z_e (N x d_out) for every expert: row n is (B_e A_e x_n)^T.
    A is [E*r, d_in] (expert e's rows e*r ..), B holds expert e's B_e
    (d_out x r, row-major) at element d_out*r*e."""
    X = np.asarray(X, dtype=np.float64)
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64).ravel()
    d_out = B.size // (E * r)
    Z = []
    for e in range(E):
        Ae = A[e * r:(e + 1) * r]
        Be = B[d_out * r * e:d_out * r * (e + 1)].reshape(d_out, r)
        dW = Be @ Ae                       # Delta W_e, d_out x d_in
        Z.append(X @ dW.T)                 # rows (Delta W_e x_n)^T
    return Z


def center(Z: np.ndarray) -> np.ndarray:
    """H Z with H = I - 11^T / N, evaluated as Z - 1 (1^T Z / N): every row
    minus the mean over the probe rows."""
    return Z - Z.sum(axis=0, keepdims=True) / Z.shape[0]


def cka_matrix(X: np.ndarray, A: np.ndarray, B: np.ndarray, E: int, r: int) -> np.ndarray:
    """Pairwise linear CKA s_ij of Sec. 3.3 on the materialised, centred Z_e."""
    Zc = [center(Z) for Z in adapter_outputs(X, A, B, E, r)]
    self_norm = [np.linalg.norm(Z.T @ Z, "fro") for Z in Zc]
    S = np.zeros((E, E))
    for i in range(E):
        for j in range(E):
            den = self_norm[i] * self_norm[j]
            if den > 0.0:
                S[i, j] = np.linalg.norm(Zc[i].T @ Zc[j], "fro") ** 2 / den
    return S


# ---------------------------------------------------------------------------
# Appendix: similarity graph and Louvain grouping
# ---------------------------------------------------------------------------

def similarity_graph(S: np.ndarray) -> np.ndarray:
    """W_ij = max(0, S_ij - b) on the symmetrised S with zero diagonal; b is
    the median of the off-diagonal entries."""
    S = np.asarray(S, dtype=np.float64)
    E = S.shape[0]
    Ssym = (S + S.T) / 2.0
    np.fill_diagonal(Ssym, 0.0)
    if E < 2:
        return np.zeros((E, E))
    off = Ssym[~np.eye(E, dtype=bool)]
    b = float(np.median(off))
    W = np.maximum(0.0, Ssym - b)
    np.fill_diagonal(W, 0.0)
    return W


def modularity(W: np.ndarray, labels: Sequence[int], gamma: float) -> float:
    """Q = (1/2m) sum_ij (W_ij - gamma k_i k_j / 2m) [z_i == z_j]."""
    W = np.asarray(W, dtype=np.float64)
    k = W.sum(axis=1)
    two_m = W.sum()
    if two_m <= 0.0:
        return 0.0
    z = np.asarray(labels)
    same = z[:, None] == z[None, :]
    return float(((W - gamma * np.outer(k, k) / two_m) * same).sum() / two_m)


def _degrees(W: np.ndarray) -> Tuple[List[float], float]:
    """k_i = sum_j W_ij and 2m = sum_i k_i, each summed in index order."""
    n = W.shape[0]
    k = []
    for i in range(n):
        s = 0.0
        for j in range(n):
            s += float(W[i, j])
        k.append(s)
    two_m = 0.0
    for i in range(n):
        two_m += k[i]
    return k, two_m


def _local_moves(W: np.ndarray, gamma: float) -> Tuple[np.ndarray, bool]:
    """One level of greedy local moves from singletons (the reading of the
    visiting order in the module notes).  Returns community ids (not yet
    renumbered) and whether any node moved."""
    n = W.shape[0]
    k, two_m = _degrees(W)
    comm = np.arange(n)
    tot = list(k)                       # sum of degrees per community
    moved_any = False
    if two_m <= 0.0:
        return comm, False
    while True:
        moved = False
        for i in range(n):
            ci = int(comm[i])
            tot[ci] -= k[i]             # remove i from its community
            # k_i,in(C): weight from i to the members of C (self-loop excluded),
            # summed in index order
            kin = {}
            for j in range(n):
                if j != i and W[i, j] > 0.0:
                    c = int(comm[j])
                    kin[c] = kin.get(c, 0.0) + float(W[i, j])
            cands = set(kin) | {ci}

            def gain(c):
                return kin.get(c, 0.0) - gamma * k[i] * tot[c] / two_m
            best = min(cands, key=lambda c: (-gain(c), c))
            if best != ci and gain(best) > gain(ci):
                comm[i] = best
                moved = True
                moved_any = True
            tot[int(comm[i])] += k[i]
        if not moved:
            break
    return comm, moved_any


def _renumber(labels: np.ndarray) -> np.ndarray:
    """Community ids in order of their lowest member."""
    out = np.empty_like(labels)
    seen = {}
    for i, c in enumerate(labels):
        if c not in seen:
            seen[c] = len(seen)
        out[i] = seen[c]
    return out


def louvain(W: np.ndarray, gamma: float = 0.8) -> np.ndarray:
    """Louvain grouping of the experts (nodes of W); returns the group of each
    expert, groups numbered in order of their lowest expert."""
    W = np.asarray(W, dtype=np.float64)
    n = W.shape[0]
    node_of = np.arange(n)              # super-node of every original node
    Wl = W.copy()
    while True:
        comm, moved = _local_moves(Wl, gamma)
        if not moved:
            break
        comm = _renumber(comm)
        nc = int(comm.max()) + 1
        # coarsen: W'_ab = sum over members i of a and j of b of W_ij,
        # accumulated with (i, j) in row-major order
        Wc = np.zeros((nc, nc))
        for i in range(Wl.shape[0]):
            for j in range(Wl.shape[0]):
                Wc[comm[i], comm[j]] += Wl[i, j]
        Wl = Wc
        node_of = comm[node_of]
    return _renumber(node_of)


# ---------------------------------------------------------------------------
# Sec. 3.3 / anchor appendix: consolidated group adapters
# ---------------------------------------------------------------------------

def cka_anchors(S: np.ndarray, expert_to_group: Sequence[int], G: int) -> np.ndarray:
    """CKA centre of each group: the member with the largest summed
    similarity to the other members (ties to the lowest expert)."""
    S = np.asarray(S, dtype=np.float64)
    anchors = np.full(G, -1, dtype=np.int64)
    for g in range(G):
        members = [e for e in range(len(expert_to_group)) if expert_to_group[e] == g]
        best, best_score = -1, None
        for i in members:
            score = sum(S[i, j] for j in members if j != i)
            if best_score is None or score > best_score:
                best, best_score = i, score
        anchors[g] = best
    return anchors


def group_ranks(expert_to_group: Sequence[int], G: int, r: int) -> np.ndarray:
    """r_g = sum of the members' ranks (every expert has rank r)."""
    return np.array([r * sum(1 for e in expert_to_group if e == g) for g in range(G)],
                    dtype=np.int64)


def consolidate(A: np.ndarray, B: np.ndarray, E: int, r: int, expert_to_group: Sequence[int],
                G: int, anchors: Sequence[int], A_init: np.ndarray
                ) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Group adapters from the expert adapters (readings in the module notes).
    A [E*r, d_in] and B (expert e's [d_out, r] block at d_out*r*e) are the
    expert-wise adapters; A_init [(E - G) * r, d_in] holds the standard LoRA
    draw of the extra rank rows, group by group in group order.  Returns
    (A_g packed [R, d_in], B_g packed flat, ranks)."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64).ravel()
    A_init = np.asarray(A_init, dtype=np.float64)
    d_in = A.shape[1]
    d_out = B.size // (E * r)
    ranks = group_ranks(expert_to_group, G, r)
    Ag, Bg = [], []
    extra = 0
    for g in range(G):
        rg = int(ranks[g])
        a = int(anchors[g])
        Ablk = np.zeros((rg, d_in))
        Ablk[:r] = A[a * r:(a + 1) * r]
        Ablk[r:] = A_init[extra:extra + rg - r]
        extra += rg - r
        Bblk = np.zeros((d_out, rg))
        Bblk[:, :r] = (rg / r) * B[d_out * r * a:d_out * r * (a + 1)].reshape(d_out, r)
        Ag.append(Ablk)
        Bg.append(Bblk.ravel())
    return np.concatenate(Ag, axis=0), np.concatenate(Bg), ranks
