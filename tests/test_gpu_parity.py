"""Parity of the HIP library with the fp64 oracle on the same seeded inputs.

Integer outputs (the permutation) must match bit for bit; outputs and
gradients must match within relative L2 2e-2 (bf16 inputs) or 1e-5 (fp32).
Small cases compare every element; the full-size workloads compare sampled
tokens (forward, dx) and whole keys (dA, dB) that the oracle recomputes.
"""
import numpy as np
import pytest
import torch

from oracle import ace_oracle as O
from paper_2609_06072_amd import workloads as W

from gpu_harness import (PATHS, TOL, WEIGHTED, check_all, check_dB_rows, check_rel, f64,
                         make_case, oracle_args, oracle_bwd, oracle_fwd, run_gpu, say)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a HIP device")
    from paper_2609_06072_amd import ace  # noqa: F401  (fails loudly if libace.so is missing)


# Sizes the oracle finishes in seconds; still several 64-row tiles per key and
# ragged tails (d not a multiple of 64, T not a multiple of any block).
SMALL = {
    "tiny_fp32": W.CONFIGS["tiny_fp32"],
    "olmoe_bf16": W.CONFIGS["olmoe_bf16"].scaled(T=330, d_model=256, d_ffn=136),
    "qwen_bf16": W.CONFIGS["qwen_bf16"].scaled(T=301, d_model=264, d_ffn=176),
    "deepseek_bf16": W.CONFIGS["deepseek_bf16"].scaled(T=299, d_model=256, d_ffn=184),
    "mixtral_bf16": W.CONFIGS["mixtral_bf16"].scaled(T=517, d_model=256, d_ffn=456),
}


# ---------------------------------------------------------------- permute

def _perm_check(ids, E, e2g, G, mode):
    from paper_2609_06072_amd import ace
    dev = "cuda"
    rt = ace.ace_group_permute(torch.from_numpy(ids.astype(np.int32)).to(dev), E,
                               None if e2g is None else torch.from_numpy(e2g.astype(np.int32)).to(dev),
                               G, mode)
    return _perm_compare(rt, ids, E, e2g, G, mode)


def _perm_compare(rt, ids, E, e2g, G, mode):
    from paper_2609_06072_amd import ace
    T, k = ids.shape
    ref = O.permute(ids.astype(np.int64), E, None if mode == ace.ACE_ROWS_EXPERT else e2g, G, mode)
    U = ref["U"]
    torch.cuda.synchronize()
    assert np.array_equal(rt.counts.cpu().numpy(), ref["counts"])
    assert np.array_equal(rt.offsets.cpu().numpy(), ref["offsets"])
    if T * k > 0:
        assert np.array_equal(rt.row_token.cpu().numpy()[:U], ref["row_token"])
        assert np.array_equal(rt.row_slots.cpu().numpy().view(np.uint32)[:U], ref["row_slots"])
        assert np.array_equal(rt.pair_row.cpu().numpy(), ref["pair_row"])
        npairs = int(ref["row_pair"][U])
        assert np.array_equal(rt.row_pair.cpu().numpy()[:U + 1], ref["row_pair"])
        assert np.array_equal(rt.pair_list.cpu().numpy()[:npairs], ref["pair_list"])
    else:
        assert int(rt.row_pair.cpu().numpy()[0]) == 0
    dropped = int(np.sum(ref["pair_row"] < 0)) if mode != ace.ACE_ROWS_GROUP_DEDUP else None
    n = ace.ace_routing_check(rt)
    valid_pairs = sum(bin(int(m)).count("1") for m in ref["row_slots"])
    assert n == T * k - valid_pairs
    if dropped is not None:
        assert n == dropped
    return rt


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
@pytest.mark.parametrize("mode", [0, 1, 2])
def test_permute_bitexact_full_size(name, mode):
    cfg = W.CONFIGS[name]
    rt = W.make_routing(cfg)
    say(f"permute {name} mode={mode}")
    _perm_check(rt.topk_ids, cfg.E, rt.expert_to_group, rt.G, mode)


def _dual_check(ids, E, e2g, G, mode):
    """Both routings of one ace_group_expert_permute call against the oracle."""
    from paper_2609_06072_amd import ace
    dev = "cuda"
    grt, ert = ace.ace_group_expert_permute(torch.from_numpy(ids.astype(np.int32)).to(dev), E,
                                            torch.from_numpy(e2g.astype(np.int32)).to(dev), G,
                                            mode)
    assert (grt.c.mode, grt.c.n_keys, ert.c.mode, ert.c.n_keys) == (mode, G, ace.ACE_ROWS_EXPERT, E)
    _perm_compare(grt, ids, E, e2g, G, mode)
    _perm_compare(ert, ids, E, None, G, ace.ACE_ROWS_EXPERT)


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
@pytest.mark.parametrize("mode", [0, 1])
def test_group_expert_permute_bitexact_full_size(name, mode):
    cfg = W.CONFIGS[name]
    rt = W.make_routing(cfg)
    say(f"group+expert permute {name} mode={mode}")
    _dual_check(rt.topk_ids, cfg.E, rt.expert_to_group, rt.G, mode)


def test_group_expert_permute_edge_cases():
    rng = np.random.default_rng(5)
    say("group+expert permute edges")
    _dual_check(np.zeros((0, 4), np.int32), 8, np.arange(8) // 2, 4, 0)        # T = 0
    ids = rng.integers(0, 10, size=(203, 4))                                     # dropped pairs
    ids[::7, 1] = -1
    ids[::11, 2] = 99
    e2g = np.arange(10) // 3
    e2g[9] = 17
    _dual_check(ids, 10, e2g, 4, 0)
    _dual_check(ids, 10, e2g, 4, 1)
    ids = np.stack([rng.permutation(256)[:32] for _ in range(97)])              # k = 32, 256 keys
    _dual_check(ids, 256, rng.permutation(256) // 2, 128, 0)
    # a cell table too large for the scatter's own fold on the expert side
    # (the scan launch) while the group side folds
    ids = rng.integers(0, 64, size=(70001, 1))
    _dual_check(ids, 64, rng.permutation(64) // 4, 16, 0)


def test_permute_edge_cases():
    rng = np.random.default_rng(3)
    say("permute edges")
    # T = 0
    _perm_check(np.zeros((0, 4), np.int32), 8, np.arange(8) // 2, 4, 0)
    # k = 1, ragged T
    ids = rng.integers(0, 16, size=(1001, 1))
    _perm_check(ids, 16, np.arange(16) // 4, 4, 0)
    # G = 1 (full merge): U = T, every mask full
    ids = np.stack([rng.permutation(8)[:3] for _ in range(257)])
    rt = _perm_check(ids, 8, np.zeros(8, np.int64), 1, 0)
    assert int(rt.offsets[1]) == 257
    # k = 32 with E = G = 256 (identity groups)
    ids = np.stack([rng.permutation(256)[:32] for _ in range(97)])
    _perm_check(ids, 256, np.arange(256), 256, 0)
    _perm_check(ids, 256, None, 256, 2)
    # every token on one expert / one group
    ids = np.stack([[5, 1] for _ in range(300)])
    _perm_check(ids, 8, np.arange(8) // 4, 2, 0)
    # a cell table too large for the scatter's own fold (the scan launch)
    ids = rng.integers(0, 64, size=(70001, 1))
    _perm_check(ids, 64, None, 64, 2)
    # dropped pairs: out-of-range ids and a group id out of range
    ids = rng.integers(0, 10, size=(200, 4))
    ids[::7, 1] = -1
    ids[::11, 2] = 99
    e2g = np.arange(10) // 3
    e2g[9] = 17                                  # expert 9 maps outside [0, G)
    for mode in (0, 1, 2):
        _perm_check(ids, 10, e2g, 4, mode)


# ------------------------------------------------------- small full parity

@pytest.mark.parametrize("name", W.CONFIG_ORDER)
@pytest.mark.parametrize("path", list(PATHS))
def test_parity_small(name, path):
    cfg = SMALL[name]
    c = make_case(cfg, path, seed=1, with_w=(path in WEIGHTED))
    say(f"parity {name} {path} T={cfg.T} d_in={c.d_in} d_out={c.d_out} keys={c.n_keys}")
    out = run_gpu(c)
    tol = TOL[cfg.dtype]
    check_all("delta", f64(out["y"]), oracle_fwd(c), tol)
    dx, dA, dB = oracle_bwd(c)
    check_all("dx", f64(out["dx"]), dx, tol)
    check_all("dA", f64(out["dA"]), dA, tol)
    check_rel("dB", f64(out["dB"]), dB, tol)
    check_dB_rows("dB", f64(out["dB"]), dB, c.ranks, c.d_out, tol)


@pytest.mark.parametrize("name", ["tiny_fp32", "olmoe_bf16", "mixtral_bf16"])
@pytest.mark.parametrize("path", list(PATHS))
def test_parity_small_h_reused(name, path):
    """Backward that reads h from the forward's workspace: same gradients."""
    cfg = SMALL[name]
    c = make_case(cfg, path, seed=2, with_w=(path in WEIGHTED))
    say(f"parity (h reused) {name} {path} T={cfg.T} keys={c.n_keys}")
    out = run_gpu(c, reuse_h=True)
    tol = TOL[cfg.dtype]
    dx, dA, dB = oracle_bwd(c)
    check_rel("dx", f64(out["dx"]), dx, tol)
    check_rel("dA", f64(out["dA"]), dA, tol)
    check_rel("dB", f64(out["dB"]), dB, tol)
    ref = run_gpu(c, fwd=False)
    # only Hw differs (bf16: h rounded once more before the weight); dx and dA
    # do not read it
    assert torch.equal(out["dx"], ref["dx"]) and torch.equal(out["dA"], ref["dA"])
    if cfg.dtype == "f32":
        check_rel("dB vs recomputed h", f64(out["dB"]), f64(ref["dB"]), 1e-6)


# ------------------------------------------------ full size, sampled checks

def _sub_tokens(c, toks):
    """Oracle inputs restricted to the given tokens (per-pair definition, so
    every pair's value is unchanged)."""
    ids = c.rt.topk_ids[toks].astype(np.int64)
    k = c.cfg.k
    if c.input_mode == W.INPUT_SHARED:
        x = f64(c.x[torch.as_tensor(toks, device=c.x.device)])
    else:
        pairs = (np.asarray(toks)[:, None] * k + np.arange(k)[None, :]).ravel()
        x = f64(c.x[torch.as_tensor(pairs, device=c.x.device)])
    w = c.rt.topk_w[toks].astype(np.float64) if c.pair_w is not None else None
    return ids, x, w


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
@pytest.mark.parametrize("path", ["grouped", "expertwise", "down_expertwise", "combined",
                                  "pairs_shared", "pairs_per_pair"])
def test_parity_full_size_sampled(name, path):
    cfg = W.CONFIGS[name]
    if path in ("down_expertwise", "combined", "pairs_per_pair") and "down" not in cfg.projections:
        pytest.skip("this workload adapts the up projection only")
    # pair weights where the timed paths can carry them (per-row weights of
    # multi-slot rows on the grouped path)
    c = make_case(cfg, path, seed=0, with_w=(path in ("combined", "grouped", "pairs_per_pair")))
    say(f"full-size {name} {path} T={cfg.T} d_in={c.d_in} d_out={c.d_out}")
    out = run_gpu(c, reuse_h=True)   # as timed: the backward reuses the forward's h
    tol = TOL[cfg.dtype]
    k = cfg.k
    rng = np.random.default_rng(123)
    toks = np.sort(rng.choice(cfg.T, size=min(48, cfg.T), replace=False))
    ids, x, w = _sub_tokens(c, toks)
    a, _ = oracle_args(c, ids=ids, x=x)
    ref = O.lora_delta(*a, input_mode=c.input_mode, pair_w=w)
    rows = (toks[:, None] * k + np.arange(k)[None, :]).ravel()
    # output / output-gradient rows: per pair, or per token when combined
    orows = toks if c.input_mode == W.INPUT_COMBINED else rows
    check_all("delta(sampled tokens)", f64(out["y"][torch.as_tensor(orows, device="cuda")]), ref,
              tol)
    dy_sub = f64(c.dy[torch.as_tensor(orows, device="cuda")])
    dx_ref, _, _ = O.lora_grads(*a, dy_sub, input_mode=c.input_mode, pair_w=w)
    if c.input_mode == W.INPUT_SHARED:
        got = f64(out["dx"][torch.as_tensor(toks, device="cuda")])
    else:
        got = f64(out["dx"][torch.as_tensor(rows, device="cuda")])
    check_all("dx(sampled tokens)", got, dx_ref, tol)
    # dA/dB of the largest and the smallest non-empty key: every pair of the key
    keys = O.pair_keys(c.rt.topk_ids.astype(np.int64), cfg.E, c.e2g, c.n_keys)
    cnt = np.bincount(keys[keys >= 0].ravel(), minlength=c.n_keys)
    nz = np.nonzero(cnt)[0]
    off = np.concatenate([[0], np.cumsum(c.ranks)])
    for q in {int(nz[np.argmax(cnt[nz])]), int(nz[np.argmin(cnt[nz])])}:
        ids_q = c.rt.topk_ids.astype(np.int64).copy()
        ids_q[keys != q] = -1
        a, w = oracle_args(c, ids=ids_q)
        _, dA, dB = O.lora_grads(*a, f64(c.dy), input_mode=c.input_mode, pair_w=w)
        lo, hi = off[q], off[q + 1]
        check_all(f"dA[key {q}]", f64(out["dA"][lo:hi]), dA[lo:hi], tol)
        got_B, ref_B = f64(out["dB"][c.d_out * lo: c.d_out * hi]), dB[c.d_out * lo: c.d_out * hi]
        check_rel(f"dB[key {q}]", got_B, ref_B, tol)
        check_dB_rows(f"dB[key {q}]", got_B, ref_B, [c.ranks[q]], c.d_out, tol)


# ---------------------------------------------------------- invariants

@pytest.mark.parametrize("permuted", [False, True])
def test_group_per_expert_is_bitwise_expertwise(permuted):
    """G = E with one expert per group runs the same kernels on the same rows
    as expert-wise LoRA.  Every row's forward and every key's dA/dB must agree
    bit for bit; dx too when the map is the identity (a permuted map changes
    the order in which keys are summed into dx, so dx is checked to tolerance)."""
    cfg = SMALL["olmoe_bf16"]
    c = make_case(cfg, "expertwise", seed=2)
    ew = run_gpu(c)
    rng = np.random.default_rng(4)
    perm = rng.permutation(cfg.E) if permuted else np.arange(cfg.E)   # expert e -> group perm[e]
    r = cfg.r_e
    inv = torch.as_tensor(np.argsort(perm), device="cuda")            # group g holds expert inv[g]
    A = c.A.view(cfg.E, r, c.d_in)[inv].reshape(-1, c.d_in).contiguous()
    B = c.B.view(cfg.E, c.d_out * r)[inv].reshape(-1).contiguous()
    rt = W.Routing(c.rt.topk_ids, c.rt.topk_w, perm.astype(np.int32),
                   np.full(cfg.E, r, np.int32), r)
    g = make_case(cfg, "grouped", seed=2)
    g.rt, g.ranks, g.e2g, g.n_keys, g.A, g.B = rt, [r] * cfg.E, rt.expert_to_group, cfg.E, A, B
    g.x, g.dy = c.x, c.dy
    gr = run_gpu(g)
    assert torch.equal(gr["y"], ew["y"])
    dA = ew["dA"].view(cfg.E, r, c.d_in)[inv].reshape(-1, c.d_in)
    dB = ew["dB"].view(cfg.E, -1)[inv].reshape(-1)
    assert torch.equal(gr["dA"], dA) and torch.equal(gr["dB"], dB)
    if permuted:
        check_rel("dx", f64(gr["dx"]), f64(ew["dx"]), 1e-2)
    else:
        assert torch.equal(gr["dx"], ew["dx"])


@pytest.mark.parametrize("path", ["expertwise", "combined_expertwise", "grouped", "down_expertwise"])
def test_repeated_ids_are_dropped(path):
    """A token that lists an expert twice: the repeat is dropped (the routed
    experts of a token are a set) on every path, including the shared-input
    expert-wise backward, whose dense per-token dH rows would otherwise
    collide, and the combined expert-wise down projection."""
    from paper_2609_06072_amd import ace
    cfg = SMALL["olmoe_bf16"]
    c = make_case(cfg, path, seed=12, with_w=(path in WEIGHTED))
    ids = c.rt.topk_ids.copy()
    ids[::5, 1] = ids[::5, 0]
    ids[::7, 3] = ids[::7, 2]
    c.rt = W.Routing(ids.astype(np.int32), c.rt.topk_w, c.rt.expert_to_group, c.rt.group_rank,
                     c.rt.expert_rank)
    say(f"repeated ids {path}")
    out = run_gpu(c)
    n_rep = sum(1 for t in range(cfg.T) for j in range(cfg.k) if ids[t, j] in ids[t, :j])
    assert n_rep > 0
    assert ace.ace_routing_check(out["routing"]) == n_rep
    tol = TOL[cfg.dtype]
    check_all("delta", f64(out["y"]), oracle_fwd(c), tol)
    dx, dA, dB = oracle_bwd(c)
    check_all("dx", f64(out["dx"]), dx, tol)
    check_all("dA", f64(out["dA"]), dA, tol)
    check_dB_rows("dB", f64(out["dB"]), dB, c.ranks, c.d_out, tol)


@pytest.mark.parametrize("path", ["grouped", "down_expertwise", "pairs_shared"])
def test_deterministic(path):
    c = make_case(SMALL["qwen_bf16"], path, seed=3)
    a = run_gpu(c)
    b = run_gpu(c)
    for key in ("y", "dx", "dA", "dB"):
        assert torch.equal(a[key], b[key]), key
    for key in ("row_token", "row_slots", "pair_row", "offsets", "row_pair", "pair_list"):
        assert torch.equal(getattr(a["routing"], key), getattr(b["routing"], key))


def test_zero_B_gives_zero_update():
    c = make_case(SMALL["olmoe_bf16"], "grouped", seed=5)
    c.B = torch.zeros_like(c.B)
    out = run_gpu(c)
    assert not out["y"].any() and not out["dx"].any() and not out["dA"].any()
    dx, dA, dB = oracle_bwd(c)
    check_rel("dB(B=0)", f64(out["dB"]), dB, TOL["bf16"])


def test_empty_group_gets_exact_zero():
    cfg = SMALL["olmoe_bf16"]
    c = make_case(cfg, "grouped", seed=6)
    ids = c.rt.topk_ids.copy()
    gone = set(np.nonzero(c.rt.expert_to_group == 3)[0].tolist())
    keep = [e for e in range(cfg.E) if e not in gone]
    rng = np.random.default_rng(6)
    for t in range(ids.shape[0]):
        for j in range(ids.shape[1]):
            if ids[t, j] in gone:
                free = [e for e in keep if e not in ids[t]]
                ids[t, j] = free[rng.integers(len(free))]
    c.rt = W.Routing(ids.astype(np.int32), c.rt.topk_w, c.rt.expert_to_group, c.rt.group_rank, c.rt.expert_rank)
    out = run_gpu(c)
    off = np.concatenate([[0], np.cumsum(c.ranks)])
    lo, hi = off[3], off[4]
    assert not out["dA"][lo:hi].any() and not out["dB"][c.d_out * lo: c.d_out * hi].any()
    dx, dA, dB = oracle_bwd(c)
    check_rel("dA", f64(out["dA"]), dA, TOL["bf16"])


@pytest.mark.parametrize("path", ["grouped", "combined"])
def test_accumulates_into_existing_outputs(path):
    c = make_case(SMALL["deepseek_bf16"], path, seed=7, with_w=(path == "combined"))
    rows = c.cfg.T if path == "combined" else c.cfg.P
    y0 = W.draw_tensor((rows, c.d_out), 1.0, 7, "y_in", "bf16", "cuda")
    dx0 = W.draw_tensor(tuple(c.x.shape), 1.0, 7, "dx_in", "bf16", "cuda")
    out = run_gpu(c, y_in=y0, dx_in=dx0)
    ref = f64(y0) + oracle_fwd(c)
    check_rel("y_in + delta", f64(out["y"]), ref, TOL["bf16"])
    dx, _, _ = oracle_bwd(c)
    check_rel("dx_in + dx", f64(out["dx"]), f64(dx0) + dx, TOL["bf16"])


@pytest.mark.parametrize("name", ["mixtral_bf16", "qwen_bf16"])
def test_accumulates_full_size_weighted(name):
    """Full-size grouped forward with pair weights into y_in ~ N(0, 1) (rows
    that serve several slots add w * C once per slot).  Every sampled element
    of y_out must lie within half a bf16 ulp of fp64(y_in) + delta (the one
    rounding of the sum), plus 2% of the row's largest |delta| (the bf16
    rounding of h between the two contractions), and every row must pass the
    relative-L2 bound."""
    cfg = W.CONFIGS[name]
    c = make_case(cfg, "grouped", seed=3, with_w=True)
    y0 = W.draw_tensor((cfg.P, c.d_out), 1.0, 3, "y_in", "bf16", "cuda")
    say(f"full-size accumulate {name} T={cfg.T} d_out={c.d_out}")
    out = run_gpu(c, bwd=False, y_in=y0)
    rng = np.random.default_rng(5)
    toks = np.sort(rng.choice(cfg.T, size=32, replace=False))
    ids, x, w = _sub_tokens(c, toks)
    a, _ = oracle_args(c, ids=ids, x=x)
    delta = O.lora_delta(*a, input_mode=c.input_mode, pair_w=w)
    rows = torch.as_tensor((toks[:, None] * cfg.k + np.arange(cfg.k)[None, :]).ravel(), device="cuda")
    ref = f64(y0[rows]) + delta
    got = f64(out["y"][rows])
    check_all("y_in + delta (sampled tokens)", got, ref, TOL["bf16"])
    ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-30))) - 7)
    bound = 0.5 * ulp + 0.02 * np.abs(delta).max(axis=1, keepdims=True) + 1e-7
    worst = float(np.max(np.abs(got - ref) / bound))
    assert worst <= 1.0, f"an element is {worst:.2f}x the rounding bound"


@pytest.mark.parametrize("path", ["grouped", "combined"])
def test_empty_input(path):
    cfg = SMALL["olmoe_bf16"].scaled(T=0)
    c = make_case(cfg, path, seed=0)
    out = run_gpu(c)
    assert out["y"].numel() == 0
    assert not out["dA"].isnan().any() and not out["dA"].any() and not out["dB"].any()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("r_e", [1, 2, 3, 6])
def test_small_and_odd_ranks(dtype, r_e):
    """The paper trains with expert rank 2; ranks that are not multiples of
    4 or 16 exercise the masked operand paths."""
    cfg = W.CONFIGS["olmoe_bf16"].scaled(T=200, d_model=128, d_ffn=96, dtype=dtype, r_e=r_e)
    for path in ("grouped", "down_expertwise", "combined"):
        c = make_case(cfg, path, seed=8, with_w=True)
        out = run_gpu(c)
        tol = TOL[dtype]
        check_rel("delta", f64(out["y"]), oracle_fwd(c), tol)
        dx, dA, dB = oracle_bwd(c)
        check_rel("dx", f64(out["dx"]), dx, tol)
        check_rel("dA", f64(out["dA"]), dA, tol)
        check_rel("dB", f64(out["dB"]), dB, tol)


@pytest.mark.parametrize("path", ["expertwise", "grouped"])
def test_shared_single_read_backward(path):
    """Shared input at ranks up to 16 with an output of at least 1280
    columns: the dB pass forms the dH partials per 128-column block (dY read
    once).  d_out = 1320 leaves a 40-column last block; expert keys at rank 8
    and group keys at rank 16 (two experts per group, rows serving two
    slots), pair weights."""
    cfg = W.CONFIGS["olmoe_bf16"].scaled(T=300, d_model=136, d_ffn=1320, r_e=8,
                                         groups=("consecutive", 2))
    c = make_case(cfg, path, seed=14, with_w=True)
    assert max(c.ranks) <= 16 and c.d_out == 1320
    say(f"shared single-read backward {path} r={max(c.ranks)} d_out={c.d_out}")
    out = run_gpu(c, reuse_h=True)
    tol = TOL["bf16"]
    check_rel("delta", f64(out["y"]), oracle_fwd(c), tol)
    dx, dA, dB = oracle_bwd(c)
    check_all("dx", f64(out["dx"]), dx, tol)
    check_all("dA", f64(out["dA"]), dA, tol)
    check_rel("dB", f64(out["dB"]), dB, tol)
    check_dB_rows("dB", f64(out["dB"]), dB, c.ranks, c.d_out, tol)


@pytest.mark.parametrize("r_e", [4, 2])
def test_per_pair_single_read_backward(r_e):
    """Per-pair input at ranks <= 16 runs the backward whose dB pass also
    forms dH from per-column-block partials: ragged column blocks (d_out = 296
    gives blocks of 128, 128 and 40 columns), pair weights, expert keys at rank
    r_e and group keys at rank 4 r_e (8 or 16 ranks per partial)."""
    cfg = W.CONFIGS["olmoe_bf16"].scaled(T=301, d_model=296, d_ffn=104, r_e=r_e)
    for path in ("down_expertwise", "pairs_per_pair"):
        c = make_case(cfg, path, seed=10, with_w=True)
        assert max(c.ranks) <= 16
        say(f"single-read backward {path} r={max(c.ranks)} d_out={c.d_out}")
        out = run_gpu(c, reuse_h=True)
        tol = TOL["bf16"]
        check_rel("delta", f64(out["y"]), oracle_fwd(c), tol)
        dx, dA, dB = oracle_bwd(c)
        check_rel("dx", f64(out["dx"]), dx, tol)
        check_rel("dA", f64(out["dA"]), dA, tol)
        check_rel("dB", f64(out["dB"]), dB, tol)


@pytest.mark.parametrize("path", ["grouped", "pairs_shared"])
@pytest.mark.parametrize("d_ffn", [4136, 6152])
def test_wide_single_read_backward(d_ffn, path):
    """Rank-64 group keys with shared input and a wide output: the dB items
    take 512 dY columns and also form the dH partials per 512-column block
    (dY read once), which are summed per row (rows serving several slots on
    the grouped path, pair weights).  d_ffn is ragged against the 512-column
    blocks, the 128-column sub-tiles and the 64-pair stages; T gives a few
    split chunks per key."""
    cfg = W.CONFIGS["mixtral_bf16"].scaled(T=1500, d_model=136, d_ffn=d_ffn)
    c = make_case(cfg, path, seed=12, with_w=True)
    assert max(c.ranks) == 64 and c.d_out == d_ffn
    say(f"wide single-read backward {path} T={cfg.T} d_out={c.d_out}")
    out = run_gpu(c, reuse_h=True)
    tol = TOL["bf16"]
    check_rel("delta", f64(out["y"]), oracle_fwd(c), tol)
    dx, dA, dB = oracle_bwd(c)
    check_all("dx", f64(out["dx"]), dx, tol)
    check_all("dA", f64(out["dA"]), dA, tol)
    check_rel("dB", f64(out["dB"]), dB, tol)
    check_dB_rows("dB", f64(out["dB"]), dB, c.ranks, c.d_out, tol)


@pytest.mark.parametrize("with_w", [True, False])
def test_wide_single_read_mixed_ranks(with_w):
    """The wide single-read backward with group ranks 16, 32 and 64 in one
    call (uneven groups): partials past a key's rank are neither written nor
    read, and every row's dH, dA and dB still match."""
    cfg = W.CONFIGS["deepseek_bf16"].scaled(T=400, d_model=136, d_ffn=1352)
    c = make_case(cfg, "grouped", seed=17, with_w=with_w)
    assert max(c.ranks) == 64 and min(c.ranks) < 64 and c.d_out == 1352
    say(f"wide single-read backward, ranks {sorted(set(c.ranks))} d_out={c.d_out} w={with_w}")
    out = run_gpu(c, reuse_h=True)
    tol = TOL["bf16"]
    dx, dA, dB = oracle_bwd(c)
    check_all("dx", f64(out["dx"]), dx, tol)
    check_all("dA", f64(out["dA"]), dA, tol)
    check_rel("dB", f64(out["dB"]), dB, tol)
    check_dB_rows("dB", f64(out["dB"]), dB, c.ranks, c.d_out, tol)


def test_wide_single_read_long_chunks():
    """From 4096 output columns the dB items take chunks of up to 4096 pairs:
    with about 4600 pairs per group key each key splits into two chunks
    whose partials are summed by the reduce (every element checked)."""
    cfg = W.CONFIGS["mixtral_bf16"].scaled(T=4600, d_model=136, d_ffn=4136)
    c = make_case(cfg, "grouped", seed=18, with_w=True)
    assert max(c.ranks) == 64 and c.d_out >= 4096
    say(f"wide single-read backward, long chunks T={cfg.T} d_out={c.d_out}")
    out = run_gpu(c, reuse_h=True)
    tol = TOL["bf16"]
    dx, dA, dB = oracle_bwd(c)
    check_all("dx", f64(out["dx"]), dx, tol)
    check_all("dA", f64(out["dA"]), dA, tol)
    check_rel("dB", f64(out["dB"]), dB, tol)
    check_dB_rows("dB", f64(out["dB"]), dB, c.ranks, c.d_out, tol)


def test_wide_single_read_unweighted():
    """The wide single-read backward on the grouped path without pair
    weights, as the gate/up projections are timed: each row's partials (one
    run over its pairs and 512-column blocks) are summed without per-pair
    factors; rows serving two slots."""
    cfg = W.CONFIGS["mixtral_bf16"].scaled(T=1500, d_model=136, d_ffn=4136)
    c = make_case(cfg, "grouped", seed=13, with_w=False)
    assert max(c.ranks) == 64 and c.pair_w is None
    grp = c.rt.expert_to_group[c.rt.topk_ids]
    assert (grp[:, 0] == grp[:, 1]).any()   # some rows serve both slots of a token
    say(f"wide single-read backward, no pair weights T={cfg.T} d_out={c.d_out}")
    out = run_gpu(c, reuse_h=True)
    tol = TOL["bf16"]
    dx, dA, dB = oracle_bwd(c)
    check_all("dx", f64(out["dx"]), dx, tol)
    check_all("dA", f64(out["dA"]), dA, tol)
    check_rel("dB", f64(out["dB"]), dB, tol)
    check_dB_rows("dB", f64(out["dB"]), dB, c.ranks, c.d_out, tol)


def test_wide_single_read_empty_group():
    """The single-read backward at rank 64 (shared input, 1352 output
    columns) when one group has no pairs: its dA and dB are exactly zero,
    and every token's two experts share the other group, so every row
    serves two slots."""
    cfg = W.CONFIGS["mixtral_bf16"].scaled(T=300, d_model=136, d_ffn=1352)
    c = make_case(cfg, "grouped", seed=16, with_w=True)
    e2g = c.rt.expert_to_group
    keep = [e for e in range(cfg.E) if e2g[e] == 0]
    rng = np.random.default_rng(16)
    ids = np.stack([rng.permutation(keep)[:cfg.k] for _ in range(cfg.T)]).astype(np.int32)
    c.rt = W.Routing(ids, c.rt.topk_w, e2g, c.rt.group_rank, c.rt.expert_rank)
    assert max(c.ranks) == 64 and c.d_out == 1352
    say(f"wide single-read backward, empty group T={cfg.T} d_out={c.d_out}")
    out = run_gpu(c, reuse_h=True)
    off = np.concatenate([[0], np.cumsum(c.ranks)])
    lo, hi = off[1], off[2]
    assert not out["dA"][lo:hi].any() and not out["dB"][c.d_out * lo: c.d_out * hi].any()
    tol = TOL["bf16"]
    dx, dA, dB = oracle_bwd(c)
    check_all("dx", f64(out["dx"]), dx, tol)
    check_rel("dA", f64(out["dA"]), dA, tol)
    check_rel("dB", f64(out["dB"]), dB, tol)


def test_max_rank_and_many_groups():
    cfg = W.CONFIGS["olmoe_bf16"].scaled(T=150, d_model=128, d_ffn=64, r_e=64,
                                         groups=("consecutive", 4))
    c = make_case(cfg, "grouped", seed=9)
    assert max(c.ranks) == 256
    out = run_gpu(c)
    check_rel("delta", f64(out["y"]), oracle_fwd(c), TOL["bf16"])
    dx, dA, dB = oracle_bwd(c)
    check_rel("dx", f64(out["dx"]), dx, TOL["bf16"])
    check_rel("dA", f64(out["dA"]), dA, TOL["bf16"])
    check_rel("dB", f64(out["dB"]), dB, TOL["bf16"])
    cfg = W.CONFIGS["olmoe_bf16"].scaled(T=100, d_model=64, d_ffn=64, E=256, k=16, r_e=2,
                                         groups=("consecutive", 1))
    c = make_case(cfg, "grouped", seed=10)
    assert c.n_keys == 256
    out = run_gpu(c)
    check_rel("delta", f64(out["y"]), oracle_fwd(c), TOL["bf16"])
