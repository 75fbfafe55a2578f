"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each test ties the oracle to something other than itself: hand-worked values
(tests/golden/hand_examples.json), special cases that reduce to a textbook
matmul, invariants of the method (Sec. 3.3 budget, Sec. 3.5 compute-once
reuse, G = E reducing to expert-wise LoRA), finite differences, and brute
force on tiny inputs.
"""
import json
import os

import numpy as np
import pytest

from oracle import ace_oracle as O
from paper_2609_06072_amd import workloads as W

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))


def _np(a, dt=np.float64):
    return np.asarray(a, dtype=dt)


# ---------------------------------------------------------------- hand-worked

def test_hand_grouped_forward():
    g = GOLD["grouped"]
    ids = _np(g["topk_ids"], np.int64)
    args = (_np(g["x"]), _np(g["A"]), _np(g["B"]), g["group_rank"], g["alpha"], ids,
            g["E"], _np(g["expert_to_group"], np.int64), g["G"])
    assert np.array_equal(O.lora_delta(*args), _np(g["delta"]))
    assert np.array_equal(O.grouped_execution_delta(*args), _np(g["delta"]))
    assert np.array_equal(O.brute_delta(*args), _np(g["delta"]))
    w = _np(g["pair_w"])
    assert np.array_equal(O.lora_delta(*args, pair_w=w), _np(g["delta_weighted"]))
    assert np.array_equal(O.grouped_execution_delta(*args, pair_w=w), _np(g["delta_weighted"]))


def test_hand_grouped_backward():
    g = GOLD["grouped"]
    ids = _np(g["topk_ids"], np.int64)
    args = (_np(g["x"]), _np(g["A"]), _np(g["B"]), g["group_rank"], g["alpha"], ids,
            g["E"], _np(g["expert_to_group"], np.int64), g["G"], _np(g["dy"]))
    for fn in (O.lora_grads, O.brute_grads):
        dx, dA, dB = fn(*args)
        assert np.array_equal(dx, _np(g["dx"]))
        assert np.array_equal(dA, _np(g["dA"]))
        assert np.array_equal(dB, _np(g["dB"]))


@pytest.mark.parametrize("mode,name", [(O.ROWS_GROUP_DEDUP, "group_dedup"),
                                       (O.ROWS_GROUP_PAIRS, "group_pairs"),
                                       (O.ROWS_EXPERT, "expert")])
def test_hand_permutation(mode, name):
    g = GOLD["grouped"]
    rt = O.permute(_np(g["topk_ids"], np.int64), g["E"], _np(g["expert_to_group"], np.int64),
                   g["G"], mode)
    exp = g["permute"][name]
    for key in ("counts", "offsets", "row_token", "row_slots", "pair_row", "row_pair", "pair_list"):
        assert list(rt[key]) == exp[key], key


def test_hand_per_pair_expertwise():
    g = GOLD["per_pair"]
    ids = _np(g["topk_ids"], np.int64)
    args = (_np(g["x"]), _np(g["A"]), _np(g["B"]), g["expert_rank"], g["alpha"], ids,
            g["E"], None, g["E"])
    d = O.lora_delta(*args, input_mode=O.INPUT_PER_PAIR)
    assert np.array_equal(d, _np(g["delta"]))
    assert np.array_equal(O.brute_delta(*args, input_mode=O.INPUT_PER_PAIR), _np(g["delta"]))
    rt = O.permute(ids, g["E"], None, g["E"], O.ROWS_EXPERT)
    for key, v in g["permute_expert"].items():
        assert list(rt[key]) == v, key


# ------------------------------------------------------------------ helpers

def tiny_problem(seed, T=5, k=3, E=6, G=3, d_in=7, d_out=5, r_e=2, input_mode=O.INPUT_SHARED,
                 expert_keys=False, drop=False):
    rng = np.random.default_rng(seed)
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int64)
    if drop:
        ids[0, 0] = E + 3          # out-of-range id: the pair is dropped
    e2g = None
    if expert_keys:
        ranks = [r_e] * E
        n_keys = E
    else:
        e2g = rng.permutation(np.arange(E) % G).astype(np.int64)
        ranks = [int(r_e * np.sum(e2g == g)) for g in range(G)]
        n_keys = G
    R = sum(ranks)
    rows = T if input_mode == O.INPUT_SHARED else T * k
    x = rng.normal(size=(rows, d_in))
    A = rng.normal(size=(R, d_in))
    B = rng.normal(size=(d_out * R,))
    dy = rng.normal(size=(T if input_mode == O.INPUT_COMBINED else T * k, d_out))
    w = rng.uniform(0.1, 1.0, size=(T, k))
    return dict(x=x, A=A, B=B, ranks=ranks, ids=ids, E=E, e2g=e2g, n_keys=n_keys, dy=dy, w=w,
                im=input_mode)


def fwd(p, **kw):
    return O.lora_delta(p["x"], p["A"], p["B"], p["ranks"], 16.0, p["ids"], p["E"], p["e2g"],
                        p["n_keys"], input_mode=p["im"], **kw)


def grads(p, **kw):
    return O.lora_grads(p["x"], p["A"], p["B"], p["ranks"], 16.0, p["ids"], p["E"], p["e2g"],
                        p["n_keys"], p["dy"], input_mode=p["im"], **kw)


# ------------------------------------------------------------- brute force

@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("im", [O.INPUT_SHARED, O.INPUT_PER_PAIR, O.INPUT_COMBINED])
@pytest.mark.parametrize("expert_keys", [False, True])
def test_brute_force_matches(seed, im, expert_keys):
    p = tiny_problem(seed, input_mode=im, expert_keys=expert_keys, drop=(seed == 3))
    a = (p["x"], p["A"], p["B"], p["ranks"], 16.0, p["ids"], p["E"], p["e2g"], p["n_keys"])
    for w in (None, p["w"]):
        d0 = O.brute_delta(*a, input_mode=im, pair_w=w)
        d1 = fwd(p, pair_w=w)
        assert O.rel_l2(d1, d0) < 1e-12
        g0 = O.brute_grads(*a, p["dy"], input_mode=im, pair_w=w)
        g1 = grads(p, pair_w=w)
        for u, v in zip(g1, g0):
            assert O.rel_l2(u, v) < 1e-12


# --------------------------------------------------- Sec. 3.5 compute-once

@pytest.mark.parametrize("seed", range(3))
def test_grouped_execution_equals_per_pair_definition(seed):
    p = tiny_problem(seed, T=9, k=4, E=8, G=3)
    a = (p["x"], p["A"], p["B"], p["ranks"], 16.0, p["ids"], p["E"], p["e2g"], p["n_keys"])
    for w in (None, p["w"]):
        assert O.rel_l2(O.grouped_execution_delta(*a, pair_w=w), fwd(p, pair_w=w)) < 1e-13


def test_hand_combined():
    """Pre-combined down projection, worked by hand (forward and backward)."""
    g, c = GOLD["grouped"], GOLD["combined"]
    ids = _np(g["topk_ids"], np.int64)
    args = (_np(c["x"]), _np(g["A"]), _np(g["B"]), g["group_rank"], g["alpha"], ids,
            g["E"], _np(g["expert_to_group"], np.int64), g["G"])
    w = _np(c["pair_w"])
    for d in (O.lora_delta(*args, input_mode=O.INPUT_COMBINED, pair_w=w),
              O.precombined_delta(*args, pair_w=w),
              O.brute_delta(*args, input_mode=O.INPUT_COMBINED, pair_w=w)):
        assert np.array_equal(d, _np(c["out"]))
    for fn in (O.lora_grads, O.brute_grads):
        dx, dA, dB = fn(*args, _np(c["dy"]), input_mode=O.INPUT_COMBINED, pair_w=w)
        assert np.array_equal(dx, _np(c["dx"]))
        assert np.array_equal(dA, _np(c["dA"]))
        assert np.array_equal(dB, _np(c["dB"]))


@pytest.mark.parametrize("seed", range(3))
def test_precombine_equals_per_pair_then_combine(seed):
    """Combining the per-pair inputs before the group adapter (one evaluation
    per active group) equals the per-pair down delta followed by the weighted
    combine over the token's slots."""
    p = tiny_problem(seed, T=9, k=4, E=8, G=3, input_mode=O.INPUT_PER_PAIR, drop=(seed == 2))
    a = (p["x"], p["A"], p["B"], p["ranks"], 16.0, p["ids"], p["E"], p["e2g"], p["n_keys"])
    T, k = p["ids"].shape
    for w in (None, p["w"]):
        per_pair = O.lora_delta(*a, input_mode=O.INPUT_PER_PAIR, pair_w=w)
        combined = per_pair.reshape(T, k, -1).sum(axis=1)
        assert O.rel_l2(O.precombined_delta(*a, pair_w=w), combined) < 1e-13


# -------------------------------------------- G = E reduces to expert-wise

@pytest.mark.parametrize("permuted", [False, True])
def test_group_per_expert_is_expertwise(permuted):
    rng = np.random.default_rng(11)
    T, k, E, d_in, d_out, r = 7, 3, 5, 6, 4, 3
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int64)
    x = rng.normal(size=(T, d_in))
    A = rng.normal(size=(E * r, d_in))
    B = rng.normal(size=(d_out * E * r,))
    dy = rng.normal(size=(T * k, d_out))
    ew = O.lora_delta(x, A, B, [r] * E, 16.0, ids, E, None, E)
    ewg = O.lora_grads(x, A, B, [r] * E, 16.0, ids, E, None, E, dy)
    perm = rng.permutation(E) if permuted else np.arange(E)   # expert e -> group perm[e]
    # group perm[e] carries expert e's adapter
    Ag = np.zeros_like(A)
    Bg = np.zeros_like(B)
    for e in range(E):
        g = perm[e]
        Ag[g * r:(g + 1) * r] = A[e * r:(e + 1) * r]
        Bg[d_out * g * r: d_out * (g + 1) * r] = B[d_out * e * r: d_out * (e + 1) * r]
    gr = O.lora_delta(x, Ag, Bg, [r] * E, 16.0, ids, E, perm, E)
    assert np.array_equal(gr, ew)
    ded = O.grouped_execution_delta(x, Ag, Bg, [r] * E, 16.0, ids, E, perm, E)
    assert np.array_equal(ded, ew)
    dx, dA, dB = O.lora_grads(x, Ag, Bg, [r] * E, 16.0, ids, E, perm, E, dy)
    assert np.array_equal(dx, ewg[0])
    for e in range(E):
        g = perm[e]
        assert np.array_equal(dA[g * r:(g + 1) * r], ewg[1][e * r:(e + 1) * r])
        assert np.array_equal(dB[d_out * g * r: d_out * (g + 1) * r],
                              ewg[2][d_out * e * r: d_out * (e + 1) * r])


# --------------------------------------- G = 1 full merge is dense LoRA

def test_full_merge_is_dense_lora():
    rng = np.random.default_rng(5)
    T, k, E, d_in, d_out, r = 6, 2, 4, 5, 3, 4
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int64)
    x = rng.normal(size=(T, d_in))
    A = rng.normal(size=(r, d_in))
    Bm = rng.normal(size=(d_out, r))
    d = O.lora_delta(x, A, Bm.reshape(-1), [r], 16.0, ids, E, np.zeros(E, np.int64), 1)
    dense = (16.0 / r) * np.matmul(np.matmul(x, A.T), Bm.T)     # textbook LoRA
    assert O.rel_l2(d, np.repeat(dense, k, axis=0)) < 1e-14
    rt = O.permute(ids, E, np.zeros(E, np.int64), 1, O.ROWS_GROUP_DEDUP)
    assert rt["U"] == T and all(m == (1 << k) - 1 for m in rt["row_slots"])


# ------------------------------------------- zero adapters, linearity

def test_zero_B_and_zero_A():
    p = tiny_problem(2)
    p0 = dict(p, B=np.zeros_like(p["B"]))
    assert np.array_equal(fwd(p0), np.zeros_like(fwd(p)))
    dx, dA, dB = grads(p0)
    assert not dx.any() and not dA.any() and np.abs(dB).sum() > 0   # LoRA init case
    p1 = dict(p, A=np.zeros_like(p["A"]))
    dx, dA, dB = grads(p1)
    assert not dB.any() and not dx.any() and np.abs(dA).sum() > 0


def test_linearity():
    p = tiny_problem(3)
    rng = np.random.default_rng(9)
    x2 = rng.normal(size=p["x"].shape)
    d1, d2 = fwd(p), fwd(dict(p, x=x2))
    assert O.rel_l2(fwd(dict(p, x=p["x"] + 2.5 * x2)), d1 + 2.5 * d2) < 1e-13
    assert O.rel_l2(O.lora_delta(p["x"], p["A"], p["B"], p["ranks"], 8.0, p["ids"], p["E"],
                                 p["e2g"], p["n_keys"]), 0.5 * d1) < 1e-15
    w = p["w"]
    dw = fwd(p, pair_w=w)
    assert O.rel_l2(dw, d1 * w.reshape(-1, 1)) < 1e-15


# ------------------- Sec. 3.3: a group of concatenated adapters, scaled

def test_concatenated_group_adapter_scale():
    """With A_g = [A_e; ...] and B_g = [B_e, ...], Delta W_g = sum_e B_e A_e, so
    (alpha/r_g) Delta W_g x = (r_e / r_g) sum_e (alpha/r_e) B_e A_e x."""
    rng = np.random.default_rng(21)
    E, d_in, d_out, r = 3, 6, 5, 2
    x = rng.normal(size=(1, d_in))
    As = [rng.normal(size=(r, d_in)) for _ in range(E)]
    Bs = [rng.normal(size=(d_out, r)) for _ in range(E)]
    total = np.zeros(d_out)
    for e in range(E):
        ids = np.array([[e]])
        total += O.lora_delta(x, np.concatenate(As), O.pack_B(Bs), [r] * E, 16.0, ids, E, None, E)[0]
    Ag = np.concatenate(As)
    Bg = np.concatenate(Bs, axis=1)
    ids = np.array([[0]])
    grp = O.lora_delta(x, Ag, Bg.reshape(-1), [E * r], 16.0, ids, E, np.zeros(E, np.int64), 1)[0]
    assert O.rel_l2(grp, total * (r / (E * r))) < 1e-14


# ------------------------------------------------ finite differences

@pytest.mark.parametrize("im", [O.INPUT_SHARED, O.INPUT_PER_PAIR, O.INPUT_COMBINED])
def test_finite_differences(im):
    p = tiny_problem(4, T=4, k=2, E=4, G=2, d_in=3, d_out=4, r_e=1, input_mode=im)
    w = p["w"]

    def L(pp):
        return float(np.sum(p["dy"] * fwd(pp, pair_w=w)))

    dx, dA, dB = grads(p, pair_w=w)
    h = 1e-3
    for name, g in (("x", dx), ("A", dA), ("B", dB)):
        base = p[name]
        num = np.zeros_like(base)
        it = np.nditer(base, flags=["multi_index"])
        for _ in it:
            i = it.multi_index
            a, b = base.copy(), base.copy()
            a[i] += h
            b[i] -= h
            num[i] = (L(dict(p, **{name: a})) - L(dict(p, **{name: b}))) / (2 * h)
        assert O.rel_l2(g, num) < 1e-9, name


# --------------------------------------------- gradient support (Sec 3.1.2)

def test_empty_group_and_dropped_pairs():
    rng = np.random.default_rng(8)
    T, k, E, G, d_in, d_out = 6, 2, 6, 3, 4, 3
    e2g = np.array([0, 0, 1, 1, 2, 2])
    ids = np.stack([rng.choice([0, 1, 4, 5], size=k, replace=False) for _ in range(T)])
    ids[2, :] = [-1, 99]        # token 2: both pairs dropped
    ranks = [4, 4, 4]
    x = rng.normal(size=(T, d_in))
    A = rng.normal(size=(12, d_in))
    B = rng.normal(size=(d_out * 12,))
    dy = rng.normal(size=(T * k, d_out))
    dx, dA, dB = O.lora_grads(x, A, B, ranks, 16.0, ids, E, e2g, G, dy)
    assert not dA[4:8].any() and not dB[d_out * 4: d_out * 8].any()     # group 1 never routed
    assert not dx[2].any()
    d = O.lora_delta(x, A, B, ranks, 16.0, ids, E, e2g, G)
    assert not d[4:6].any()


def test_repeated_id_within_a_token_is_dropped():
    """The routed experts R(x) of a token are a set (Sec. 3.1): a slot that
    repeats an expert id listed at a lower slot of the same token is not a
    routed pair.  Every oracle path treats it exactly like an id out of range."""
    rng = np.random.default_rng(11)
    T, k, E, G, d_in, d_out = 3, 3, 4, 2, 5, 4
    e2g = np.array([0, 0, 1, 1])
    ids = np.array([[2, 2, 0], [1, 3, 1], [0, 1, 2]])
    gone = ids.copy()
    gone[0, 1] = gone[1, 2] = -1              # the repeats, dropped by hand
    x = rng.normal(size=(T, d_in))
    xp = rng.normal(size=(T * k, d_in))
    dy = rng.normal(size=(T * k, d_out))
    for e2g_, n_keys, ranks in ((e2g, G, [4, 4]), (None, E, [2, 2, 2, 2])):
        A = rng.normal(size=(sum(ranks), d_in))
        B = rng.normal(size=(d_out * sum(ranks),))
        for im, xin in ((O.INPUT_SHARED, x), (O.INPUT_PER_PAIR, xp)):
            a = (xin, A, B, ranks, 16.0)
            d = O.lora_delta(*a, ids, E, e2g_, n_keys, input_mode=im)
            assert not d[1].any() and not d[5].any()
            assert np.array_equal(d, O.lora_delta(*a, gone, E, e2g_, n_keys, input_mode=im))
            assert np.allclose(O.brute_delta(*a, ids, E, e2g_, n_keys, input_mode=im), d,
                               rtol=1e-12, atol=1e-12)
            g1 = O.lora_grads(*a, ids, E, e2g_, n_keys, dy, input_mode=im)
            g0 = O.lora_grads(*a, gone, E, e2g_, n_keys, dy, input_mode=im)
            for u, v in zip(g1, g0):
                assert np.array_equal(u, v)
    for mode in (O.ROWS_GROUP_DEDUP, O.ROWS_GROUP_PAIRS, O.ROWS_EXPERT):
        r1 = O.permute(ids, E, e2g, G, mode)
        r0 = O.permute(gone, E, e2g, G, mode)
        for key in ("counts", "offsets", "row_token", "row_slots", "pair_row", "row_pair",
                    "pair_list"):
            assert np.array_equal(r1[key], r0[key]), (mode, key)
        assert r1["pair_row"][1] == -1 and r1["pair_row"][5] == -1
    # token 0 in group mode: slots 0 and 2 (experts 2 and 0) are in different
    # groups, so the repeat leaves one row per group with one slot each
    r = O.permute(ids, E, e2g, G, O.ROWS_GROUP_DEDUP)
    assert sorted(int(m) for m, t in zip(r["row_slots"], r["row_token"]) if t == 0) == [1, 4]


# ---------------------------------------------- permutation invariants

@pytest.mark.parametrize("mode", [O.ROWS_GROUP_DEDUP, O.ROWS_GROUP_PAIRS, O.ROWS_EXPERT])
def test_permutation_invariants(mode):
    cfg = W.CONFIGS["olmoe_bf16"].scaled(T=200)
    rt = W.make_routing(cfg, seed=1)
    ids = rt.topk_ids.astype(np.int64)
    res = O.permute(ids, cfg.E, rt.expert_to_group, rt.G, mode)
    U = res["U"]
    assert res["counts"].sum() == U and res["offsets"][-1] == U
    assert np.all(np.diff(res["offsets"]) >= 0)
    pc = sum(bin(int(m)).count("1") for m in res["row_slots"])
    assert pc == cfg.P
    for q in range(len(res["counts"])):
        toks = res["row_token"][res["offsets"][q]:res["offsets"][q + 1]]
        assert np.all(np.diff(toks) > 0) if mode != O.ROWS_GROUP_PAIRS else np.all(np.diff(toks) >= 0)
    key = (lambda e: e) if mode == O.ROWS_EXPERT else (lambda e: rt.expert_to_group[e])
    for p in range(cfg.P):
        u = res["pair_row"][p]
        t, j = divmod(p, cfg.k)
        assert res["row_token"][u] == t and (res["row_slots"][u] >> j) & 1
        q = key(ids[t, j])
        assert res["offsets"][q] <= u < res["offsets"][q + 1]
    if mode == O.ROWS_GROUP_DEDUP:
        exp_U = sum(len({rt.expert_to_group[e] for e in ids[t]}) for t in range(cfg.T))
        assert U == exp_U
    else:
        assert U == cfg.P
    # pair order: every routed pair once, sorted by (key, token, slot); a
    # row's pairs are consecutive and start at row_pair[u]
    rp, pl = res["row_pair"], res["pair_list"]
    assert rp[U] == cfg.P and sorted(pl.tolist()) == list(range(cfg.P))
    keyed = [(key(ids[p // cfg.k, p % cfg.k]), p // cfg.k, p % cfg.k) for p in pl]
    assert keyed == sorted(keyed)
    for u in range(U):
        m = int(res["row_slots"][u])
        slots = [j for j in range(cfg.k) if (m >> j) & 1]
        assert rp[u + 1] - rp[u] == len(slots)
        t = res["row_token"][u]
        assert pl[rp[u]:rp[u + 1]].tolist() == [t * cfg.k + j for j in slots]
    if mode != O.ROWS_GROUP_DEDUP:
        assert np.array_equal(rp, np.arange(U + 1))


def test_k1_dedup_is_pairs():
    rng = np.random.default_rng(2)
    ids = rng.integers(0, 8, size=(30, 1))
    e2g = np.arange(8) // 2
    a = O.permute(ids, 8, e2g, 4, O.ROWS_GROUP_DEDUP)
    b = O.permute(ids, 8, e2g, 4, O.ROWS_GROUP_PAIRS)
    for key in ("counts", "offsets", "row_token", "row_slots", "pair_row", "row_pair", "pair_list"):
        assert np.array_equal(a[key], b[key])


def test_rel_l2():
    assert O.rel_l2([1.0, 0.0], [1.0, 0.0]) == 0.0
    assert O.rel_l2([0.0], [0.0]) == 0.0
    assert O.rel_l2([1e-30], [0.0]) == float("inf")
    assert abs(O.rel_l2([3.0, 4.0], [0.0, 4.0]) - 0.75) < 1e-15


# ----------------------------- adapted expert projection (frozen W_e + adapter)

def test_hand_adapted_projection():
    g, a = GOLD["grouped"], GOLD["adapted"]
    ids = _np(g["topk_ids"], np.int64)
    Wb = _np(a["W"])
    args = (_np(g["x"]), Wb, _np(g["A"]), _np(g["B"]), g["group_rank"], g["alpha"], ids,
            g["E"], _np(g["expert_to_group"], np.int64), g["G"])
    assert np.array_equal(O.expert_projection(_np(g["x"]), Wb, ids, g["E"]), _np(a["base"]))
    assert np.array_equal(O.adapted_projection(*args), _np(a["y"]))
    assert np.array_equal(O.brute_adapted_projection(*args), _np(a["y"]))


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("im", [O.INPUT_SHARED, O.INPUT_PER_PAIR])
@pytest.mark.parametrize("expert_keys", [False, True])
def test_adapted_projection_brute_force(seed, im, expert_keys):
    p = tiny_problem(seed, input_mode=im, expert_keys=expert_keys, drop=(seed == 2))
    rng = np.random.default_rng(100 + seed)
    Wb = rng.normal(size=(p["E"], 5, 7))
    a = (p["x"], Wb, p["A"], p["B"], p["ranks"], 16.0, p["ids"], p["E"], p["e2g"], p["n_keys"])
    y0 = O.brute_adapted_projection(*a, input_mode=im)
    y1 = O.adapted_projection(*a, input_mode=im)
    assert O.rel_l2(y1, y0) < 1e-12
    if seed == 2:   # the dropped pair's row stays zero
        assert not y1[0].any()


def test_adapted_projection_single_expert_is_merged_linear():
    """One expert, k = 1: every token goes through W + s B A, a plain matmul
    with the merged weight."""
    rng = np.random.default_rng(11)
    T, d_in, d_out, r = 9, 6, 4, 3
    x = rng.normal(size=(T, d_in))
    Wb = rng.normal(size=(1, d_out, d_in))
    A = rng.normal(size=(r, d_in))
    Bm = rng.normal(size=(d_out, r))
    ids = np.zeros((T, 1), np.int64)
    y = O.adapted_projection(x, Wb, A, Bm.reshape(-1), [r], 16.0, ids, 1, None, 1)
    merged = Wb[0] + (16.0 / r) * np.matmul(Bm, A)
    assert O.rel_l2(y, np.matmul(x, merged.T)) < 1e-14


def test_adapted_projection_zero_adapter_is_base():
    p = tiny_problem(1)
    rng = np.random.default_rng(12)
    Wb = rng.normal(size=(p["E"], 5, 7))
    y = O.adapted_projection(p["x"], Wb, p["A"], np.zeros_like(p["B"]), p["ranks"], 16.0,
                             p["ids"], p["E"], p["e2g"], p["n_keys"])
    base = np.zeros((p["ids"].size, 5))
    for t in range(p["ids"].shape[0]):          # per pair: x_t times W_e^T
        for j in range(p["ids"].shape[1]):
            base[t * p["ids"].shape[1] + j] = np.matmul(Wb[p["ids"][t, j]], p["x"][t])
    assert O.rel_l2(y, base) < 1e-14
