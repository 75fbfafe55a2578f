"""Pins of the consolidation oracle (CKA, similarity graph, Louvain, anchors,
consolidated initialisation) against what the paper and the mathematics fix.

Each check is chosen so that a plausible slip in the oracle (a dropped
centring, a transposed operand, a wrong norm, a missing symmetrisation, an
inverted gain) fails one of them.
"""
import json
import os

import numpy as np

from oracle import ace_oracle as O
from oracle import consolidation_oracle as C

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "consolidation_examples.json")


def _adapters(rng, E, r, d_in, d_out):
    A = rng.standard_normal((E * r, d_in)) / np.sqrt(d_in)
    B = rng.standard_normal(E * r * d_out) * 0.02
    return A, B


# ---------------------------------------------------------------- CKA

def test_cka_equals_kernel_form():
    """Linear CKA in its sample-Gram (HSIC) form: with K_e = Zc_e Zc_e^T,
    ||Zc_i^T Zc_j||_F^2 = tr(K_i K_j)."""
    rng = np.random.default_rng(1)
    E, r, d_in, d_out, N = 5, 3, 7, 6, 11
    X = rng.standard_normal((N, d_in)) + 3.0
    A, B = _adapters(rng, E, r, d_in, d_out)
    S = C.cka_matrix(X, A, B, E, r)
    K = []
    for e in range(E):
        Ae = A[e * r:(e + 1) * r]
        Be = B[d_out * r * e:d_out * r * (e + 1)].reshape(d_out, r)
        Z = np.array([[sum(Be[o, q] * sum(Ae[q, i] * X[n, i] for i in range(d_in)) for q in range(r))
                       for o in range(d_out)] for n in range(N)])
        mu = Z.sum(axis=0) / N
        Zc = Z - mu
        K.append(Zc @ Zc.T)
    for i in range(E):
        for j in range(E):
            ref = np.trace(K[i] @ K[j]) / np.sqrt(np.trace(K[i] @ K[i]) * np.trace(K[j] @ K[j]))
            assert abs(S[i, j] - ref) <= 1e-12 * max(1.0, abs(ref))


def test_cka_scalar_output_is_squared_pearson():
    """d_out = r = 1: Z_e is one column, and linear CKA is the squared Pearson
    correlation of the two columns."""
    rng = np.random.default_rng(2)
    E, N, d_in = 4, 50, 6
    X = rng.standard_normal((N, d_in))
    A, B = _adapters(rng, E, 1, d_in, 1)
    S = C.cka_matrix(X, A, B, E, 1)
    z = np.stack([X @ A[e] * B[e] for e in range(E)])
    rho = np.corrcoef(z)
    np.testing.assert_allclose(S, rho ** 2, rtol=1e-12, atol=1e-14)


def test_cka_invariances_and_range():
    rng = np.random.default_rng(3)
    E, r, d_in, d_out, N = 6, 2, 9, 5, 40
    X = rng.standard_normal((N, d_in))
    A, B = _adapters(rng, E, r, d_in, d_out)
    S = C.cka_matrix(X, A, B, E, r)
    np.testing.assert_allclose(np.diag(S), 1.0, rtol=1e-12)
    np.testing.assert_allclose(S, S.T, rtol=1e-12, atol=1e-15)
    assert S.min() >= 0.0 and S.max() <= 1.0 + 1e-12
    # a per-expert output scale (e.g. the LoRA scale) does not change S
    B2 = B.copy()
    B2[d_out * r * 2:d_out * r * 3] *= -7.5
    np.testing.assert_allclose(C.cka_matrix(X, A, B2, E, r), S, rtol=1e-10, atol=1e-14)
    # an orthogonal map of one expert's output space does not change S
    Q, _ = np.linalg.qr(rng.standard_normal((d_out, d_out)))
    B3 = B.copy()
    B3[d_out * r:2 * d_out * r] = (Q @ B[d_out * r:2 * d_out * r].reshape(d_out, r)).ravel()
    np.testing.assert_allclose(C.cka_matrix(X, A, B3, E, r), S, rtol=1e-10, atol=1e-14)
    # shifting every probe row by the same vector does not change S (centring)
    np.testing.assert_allclose(C.cka_matrix(X + rng.standard_normal(d_in), A, B, E, r), S,
                               rtol=1e-9, atol=1e-13)


def test_cka_special_cases():
    rng = np.random.default_rng(4)
    r, d_in, d_out, N = 2, 4, 3, 8
    # probe of four Walsh columns: each has zero mean and they are mutually
    # orthogonal, so the centred probe Gram X^T X is diagonal
    X = np.array([[(-1) ** bin(n & m).count("1") for m in (1, 2, 4, 7)] for n in range(N)], dtype=float)
    Xc = X - X.mean(axis=0)
    G = Xc.T @ Xc
    assert np.allclose(G - np.diag(np.diag(G)), 0)
    A = np.zeros((3 * r, d_in))
    A[0:r, 0] = [1.0, 0.5]          # expert 0 reads input coordinate 0
    A[r:2 * r, 1] = [2.0, -1.0]     # expert 1 reads coordinate 1: orthogonal to expert 0
    A[2 * r:3 * r] = A[0:r]         # expert 2 equals expert 0 up to a scale of B
    B = rng.standard_normal(3 * r * d_out)
    B[2 * r * d_out:] = 3.0 * B[:r * d_out]
    S = C.cka_matrix(X, A, B, 3, r)
    assert abs(S[0, 1]) < 1e-14 and abs(S[1, 0]) < 1e-14
    assert abs(S[0, 2] - 1.0) < 1e-12
    # an all-zero adapter has no defined CKA: its row and column are 0
    B0 = B.copy()
    B0[r * d_out:2 * r * d_out] = 0.0
    S0 = C.cka_matrix(X, A, B0, 3, r)
    assert np.all(S0[1] == 0.0) and np.all(S0[:, 1] == 0.0)


def test_cka_low_rank_identity():
    """The identity the library evaluates: with P = Xc A^T (all experts),
    M = P^T P and G_e = B_e^T B_e,
      ||Zc_i^T Zc_j||_F^2 = <G_i M_ij, M_ij G_j>_F."""
    rng = np.random.default_rng(5)
    E, r, d_in, d_out, N = 5, 3, 10, 7, 30
    X = rng.standard_normal((N, d_in)) * 2 + 1
    A, B = _adapters(rng, E, r, d_in, d_out)
    Xc = X - X.mean(axis=0)
    P = Xc @ A.T
    M = P.T @ P
    Gm = [B[d_out * r * e:d_out * r * (e + 1)].reshape(d_out, r) for e in range(E)]
    Gm = [b.T @ b for b in Gm]
    num = np.array([[np.sum((Gm[i] @ M[i * r:(i + 1) * r, j * r:(j + 1) * r]) *
                            (M[i * r:(i + 1) * r, j * r:(j + 1) * r] @ Gm[j]))
                     for j in range(E)] for i in range(E)])
    S = num / np.sqrt(np.outer(np.diag(num), np.diag(num)))
    np.testing.assert_allclose(S, C.cka_matrix(X, A, B, E, r), rtol=1e-11)


# ---------------------------------------------------------------- graph

def test_similarity_graph_hand_example():
    g = json.load(open(GOLDEN))["graph"]
    W = C.similarity_graph(np.array(g["S"]))
    np.testing.assert_allclose(W, np.array(g["W"]), atol=1e-12)


def test_similarity_graph_properties():
    rng = np.random.default_rng(6)
    S = rng.uniform(0, 1, (9, 9))
    W = C.similarity_graph(S)
    Ss = (S + S.T) / 2
    off = Ss[~np.eye(9, dtype=bool)]
    b = np.median(off)
    assert np.all(np.diag(W) == 0) and np.allclose(W, W.T) and W.min() >= 0
    # an edge survives exactly when its symmetrised similarity exceeds the median
    mask = ~np.eye(9, dtype=bool)
    assert np.array_equal((W > 0)[mask], (Ss > b)[mask])
    # about half of the off-diagonal entries survive
    assert abs(int((W[mask] > 0).sum()) - mask.sum() // 2) <= 2


# ---------------------------------------------------------------- Louvain

def _components(W):
    n = W.shape[0]
    lab = -np.ones(n, dtype=int)
    c = 0
    for s in range(n):
        if lab[s] >= 0:
            continue
        stack = [s]
        lab[s] = c
        while stack:
            i = stack.pop()
            for j in range(n):
                if W[i, j] > 0 and lab[j] < 0:
                    lab[j] = c
                    stack.append(j)
        c += 1
    return lab


def _same_partition(a, b):
    a, b = np.asarray(a), np.asarray(b)
    return np.array_equal(a[:, None] == a[None, :], b[:, None] == b[None, :])


def test_modularity_hand_values():
    """Q of fixed partitions of the 4-node example at gamma = 0.8 (and one at
    gamma = 1), every value worked out by hand from the modularity formula of
    the Louvain appendix.  A dropped gamma, a wrong 2m normaliser or a
    missing degree term changes at least one of them.  The hand values are
    decimal, so the comparison allows binary rounding (1e-12)."""
    g = json.load(open(GOLDEN))["modularity"]
    W = np.array(g["W"], dtype=np.float64)
    for case in g["cases"]:
        Q = C.modularity(W, case["labels"], case["gamma"])
        assert abs(Q - case["Q"]) <= 1e-12, (case["labels"], case["gamma"], Q, case["Q"])


def test_louvain_two_cliques():
    W = np.zeros((8, 8))
    for blk in ([0, 2, 4, 6], [1, 3, 5, 7]):
        for i in blk:
            for j in blk:
                if i != j:
                    W[i, j] = 1.0
    W[0, 1] = W[1, 0] = 0.1     # a weak bridge
    z = C.louvain(W, 0.8)
    assert list(z) == [0, 1, 0, 1, 0, 1, 0, 1]


def test_louvain_gamma_zero_merges_components():
    """With gamma = 0 every move toward a neighbour gains, so the groups are
    the connected components of the graph."""
    rng = np.random.default_rng(7)
    for trial in range(5):
        n = 12
        W = np.zeros((n, n))
        for _ in range(10):
            i, j = rng.integers(0, n, 2)
            if i != j:
                W[i, j] = W[j, i] = rng.uniform(0.1, 1)
        assert _same_partition(C.louvain(W, 0.0), _components(W))


def test_louvain_local_optimum_and_gain():
    """No single expert can be moved to another group (or to a group of its
    own) to increase Q, and Q does not fall below the singletons'."""
    rng = np.random.default_rng(8)
    for trial in range(6):
        n = 10
        S = rng.uniform(0, 1, (n, n))
        W = C.similarity_graph(S)
        z = C.louvain(W, 0.8)
        q = C.modularity(W, z, 0.8)
        assert q >= C.modularity(W, np.arange(n), 0.8) - 1e-12
        for i in range(n):
            for c in list(set(z)) + [n + 1]:
                z2 = z.copy()
                z2[i] = c
                assert C.modularity(W, z2, 0.8) <= q + 1e-12


def _partitions(items):
    if not items:
        yield []
        return
    first, rest = items[0], items[1:]
    for p in _partitions(rest):
        for i in range(len(p)):
            yield p[:i] + [[first] + p[i]] + p[i + 1:]
        yield [[first]] + p


def test_louvain_finds_planted_optimum():
    """Planted, well separated groups on 7 nodes: Louvain reaches the
    partition with the largest Q over all 877 partitions."""
    rng = np.random.default_rng(9)
    planted = [0, 0, 1, 1, 1, 2, 2]
    n = len(planted)
    for trial in range(3):
        W = np.zeros((n, n))
        for i in range(n):
            for j in range(i + 1, n):
                w = rng.uniform(0.6, 1.0) if planted[i] == planted[j] else rng.uniform(0, 0.05)
                W[i, j] = W[j, i] = w
        best, bestq = None, -np.inf
        for p in _partitions(list(range(n))):
            z = np.zeros(n, dtype=int)
            for c, blk in enumerate(p):
                z[blk] = c
            q = C.modularity(W, z, 0.8)
            if q > bestq:
                best, bestq = z, q
        z = C.louvain(W, 0.8)
        assert _same_partition(z, best) and _same_partition(z, planted)


def test_louvain_degenerate():
    assert list(C.louvain(np.zeros((4, 4)), 0.8)) == [0, 1, 2, 3]
    assert list(C.louvain(np.zeros((1, 1)), 0.8)) == [0]
    g = json.load(open(GOLDEN))["louvain"]
    assert list(C.louvain(np.array(g["W"]), g["gamma"])) == g["groups"]


# ---------------------------------------------------------------- anchors / consolidation

def test_anchor_hand_example():
    g = json.load(open(GOLDEN))["anchors"]
    a = C.cka_anchors(np.array(g["S"]), g["groups"], g["G"])
    assert list(a) == g["anchors"]


def test_consolidated_adapter_keeps_anchor_update():
    """Every routed expert of a group sees exactly its anchor's expert-wise
    update right after consolidation; the budget is unchanged."""
    rng = np.random.default_rng(10)
    E, r, d_in, d_out, T, k, alpha = 6, 2, 8, 5, 9, 2, 16.0
    A, B = _adapters(rng, E, r, d_in, d_out)
    e2g = np.array([0, 1, 0, 2, 1, 0])
    G = 3
    anchors = np.array([2, 4, 3])
    A_init = rng.standard_normal(((E - G) * r, d_in))
    Ag, Bg, ranks = C.consolidate(A, B, E, r, e2g, G, anchors, A_init)
    assert list(ranks) == [6, 4, 2]
    assert sum(ranks) * (d_in + d_out) == E * r * (d_in + d_out)
    x = rng.standard_normal((T, d_in))
    ids = np.array([rng.choice(E, k, replace=False) for _ in range(T)])
    grouped = O.lora_delta(x, Ag, Bg, list(ranks), alpha, ids, E, e2g, G)
    # expert-wise reference: expert e uses its group anchor's adapter
    Aa = np.concatenate([A[anchors[e2g[e]] * r:(anchors[e2g[e]] + 1) * r] for e in range(E)])
    Ba = np.concatenate([B[d_out * r * anchors[e2g[e]]:d_out * r * (anchors[e2g[e]] + 1)]
                         for e in range(E)])
    ref = O.lora_delta(x, Aa, Ba, [r] * E, alpha, ids, E, None, E)
    np.testing.assert_allclose(grouped, ref, rtol=1e-12, atol=1e-15)
    # the extra rank rows carry the standard draw, the extra B columns are zero
    np.testing.assert_array_equal(Ag[r:6], A_init[0:4])
    assert np.all(Bg[:d_out * 6].reshape(d_out, 6)[:, r:] == 0)
