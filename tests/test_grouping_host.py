"""The library's host-side grouping (similarity graph, Louvain, anchors)
against the consolidation oracle, on the CPU.

The partition is an integer result decided by floating-point gain
comparisons; both sides sum in index order in fp64, so graphs, groups and
anchors must agree exactly.
"""
import json
import os

import numpy as np
import pytest

from oracle import consolidation_oracle as C

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "consolidation_examples.json")


@pytest.fixture(scope="module")
def ace():
    from paper_2609_06072_amd import ace as mod
    return mod


def _planted_S(rng, E, sizes, within=(0.5, 0.9), across=(0.0, 0.2)):
    lab = np.repeat(np.arange(len(sizes)), sizes)[rng.permutation(E)]
    S = np.where(lab[:, None] == lab[None, :], rng.uniform(*within, (E, E)), rng.uniform(*across, (E, E)))
    np.fill_diagonal(S, 1.0)
    return S.astype(np.float32), lab


def test_similarity_graph_matches_oracle(ace):
    rng = np.random.default_rng(0)
    for E in (1, 2, 3, 8, 60, 64, 256):
        S = rng.uniform(0, 1, (E, E)).astype(np.float32)
        W = ace.ace_similarity_graph(S)
        assert np.array_equal(W, C.similarity_graph(S.astype(np.float64))), E


def test_louvain_matches_oracle(ace):
    rng = np.random.default_rng(1)
    cases = []
    for E in (2, 5, 16, 64):
        cases.append(C.similarity_graph(rng.uniform(0, 1, (E, E))))
    for E, sizes in ((64, [4] * 16), (60, [4] * 15), (64, [2, 4, 8, 8, 4, 2, 8, 4, 8, 8, 8])):
        S, _ = _planted_S(rng, E, sizes)
        cases.append(C.similarity_graph(S.astype(np.float64)))
    for W in cases:
        for gamma in (0.8, 0.0, 1.5):
            z, G = ace.ace_louvain(W, gamma)
            ref = C.louvain(W, gamma)
            assert list(z) == list(ref) and G == int(ref.max()) + 1


def test_louvain_recovers_planted_groups(ace):
    rng = np.random.default_rng(2)
    for E, sizes in ((64, [4] * 16), (64, [2, 4, 8, 8, 4, 2, 8, 4, 8, 8, 8])):
        S, lab = _planted_S(rng, E, sizes, within=(0.6, 0.9), across=(0.0, 0.05))
        z, G = ace.ace_louvain(ace.ace_similarity_graph(S), 0.8)
        assert G == len(sizes)
        assert np.array_equal(lab[:, None] == lab[None, :], z[:, None] == z[None, :])


def test_golden_examples(ace):
    g = json.load(open(GOLDEN))
    W = ace.ace_similarity_graph(np.array(g["graph"]["S"], dtype=np.float32))
    np.testing.assert_allclose(W, np.array(g["graph"]["W"]), atol=1e-6)
    z, G = ace.ace_louvain(np.array(g["louvain"]["W"]), g["louvain"]["gamma"])
    assert list(z) == g["louvain"]["groups"] and G == 2
    a = ace.ace_group_anchors(np.array(g["anchors"]["S"], dtype=np.float32), g["anchors"]["groups"],
                              g["anchors"]["G"])
    assert list(a) == g["anchors"]["anchors"]


def test_anchors_match_oracle(ace):
    rng = np.random.default_rng(3)
    for E, sizes in ((64, [4] * 16), (12, [5, 1, 6])):
        S, lab = _planted_S(rng, E, sizes)
        z = np.unique(lab, return_inverse=True)[1].astype(np.int32)
        G = int(z.max()) + 1
        a = ace.ace_group_anchors(S, z, G)
        assert list(a) == list(C.cka_anchors(S.astype(np.float64), z, G))
        for g in range(G):
            assert z[a[g]] == g


def test_grouping_rejects_bad_arguments(ace):
    W = np.zeros((4, 4))
    W[0, 1] = 1.0           # not symmetric
    with pytest.raises(ace.AceError):
        ace.ace_louvain(W, 0.8)
    with pytest.raises(ace.AceError):
        ace.ace_louvain(np.zeros((4, 4)), -1.0)
    S = np.eye(4, dtype=np.float32)
    with pytest.raises(ace.AceError):
        ace.ace_group_anchors(S, [0, 0, 2, 2], 3)     # group 1 empty
    with pytest.raises(ace.AceError):
        ace.ace_group_anchors(S, [0, 0, 1, 5], 2)     # id out of range
    S[1, 2] = np.nan
    with pytest.raises(ace.AceError):
        ace.ace_similarity_graph(S)
