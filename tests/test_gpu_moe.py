"""GPU parity of the adapted expert projection (ace_moe_lora_fwd): the frozen
expert GEMM with the adapter update in its epilogue, against the fp64 oracle
(oracle.ace_oracle.adapted_projection, pinned in test_oracle_pins.py).

Sizes: the small cases keep several 128-row tiles per expert and ragged tails
(d_in not a multiple of the 32-element K-block, d_out not a multiple of the
256-column tile, rows per expert not a multiple of 128); the full-size cases
run the launch configuration of the bench and check sampled tokens.
Tolerance: rel-L2 over the output, 2e-2 for bf16 and 1e-5 for fp32."""
import numpy as np
import pytest
import torch

from oracle import ace_oracle as O
from paper_2609_06072_amd import workloads as W
from gpu_harness import TOL, check_all, f64, make_case, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a HIP device")
    from paper_2609_06072_amd import ace  # noqa: F401  (fails loudly if libace.so is missing)


SMALL = {
    "tiny_fp32": W.CONFIGS["tiny_fp32"].scaled(T=300, d_model=136, d_ffn=264),
    "olmoe_bf16": W.CONFIGS["olmoe_bf16"].scaled(T=330, d_model=264, d_ffn=136),
    "qwen_bf16": W.CONFIGS["qwen_bf16"].scaled(T=301, d_model=264, d_ffn=296),
    "deepseek_bf16": W.CONFIGS["deepseek_bf16"].scaled(T=299, d_model=256, d_ffn=184),
    "mixtral_bf16": W.CONFIGS["mixtral_bf16"].scaled(T=517, d_model=264, d_ffn=520),
}

# adapter rows of each path (the base GEMM always tiles the expert-keyed rows)
MOE_PATHS = ["grouped", "expertwise", "pairs_shared", "down_expertwise", "pairs_per_pair"]


def proj_of(c):
    return "gate" if c.input_mode == W.INPUT_SHARED and "gate" in c.cfg.projections else (
        "down" if c.input_mode != W.INPUT_SHARED else c.cfg.projections[0])


def run_moe(c, Wt, base_only=False, y=None):
    from paper_2609_06072_amd import ace
    dev = c.x.device
    ids = torch.from_numpy(c.rt.topk_ids).to(dev)
    E, G = c.cfg.E, c.rt.G
    ert = ace.ace_group_permute(ids, E, None, G, W.ROWS_EXPERT)
    if y is None:
        y = torch.zeros(c.cfg.P, c.d_out, dtype=c.x.dtype, device=dev)
    if base_only:
        ace.ace_moe_lora_fwd(c.x, Wt, ert, y, input_mode=c.input_mode)
    elif c.mode == W.ROWS_EXPERT:
        ace.ace_moe_lora_fwd(c.x, Wt, ert, y, [c.cfg.r_e] * E, list(range(E)), c.cfg.alpha, c.A,
                             c.B, ert, input_mode=c.input_mode)
    else:
        e2g = torch.from_numpy(c.rt.expert_to_group).to(dev)
        art = ace.ace_group_permute(ids, E, e2g, G, c.mode)
        ace.ace_moe_lora_fwd(c.x, Wt, ert, y, c.ranks, [int(g) for g in c.rt.expert_to_group],
                             c.cfg.alpha, c.A, c.B, art, input_mode=c.input_mode)
    torch.cuda.synchronize()
    return y


def oracle_y(c, Wt, ids=None, x=None, base_only=False):
    ids = c.rt.topk_ids.astype(np.int64) if ids is None else ids
    x = f64(c.x) if x is None else x
    if base_only:
        return O.expert_projection(x, f64(Wt), ids, c.cfg.E, input_mode=c.input_mode)
    return O.adapted_projection(x, f64(Wt), f64(c.A), f64(c.B), c.ranks, c.cfg.alpha, ids,
                                c.cfg.E, c.e2g, c.n_keys, input_mode=c.input_mode)


def case_and_weights(cfg, path, seed=0):
    c = make_case(cfg, path, seed=seed)
    Wt = W.draw_expert_weights(cfg, proj_of(c), seed=seed, device="cuda")
    assert tuple(Wt.shape) == (cfg.E, c.d_out, c.d_in)
    return c, Wt


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
@pytest.mark.parametrize("path", MOE_PATHS)
def test_moe_parity_small(name, path):
    cfg = SMALL[name]
    c, Wt = case_and_weights(cfg, path)
    say(f"moe small {name} {path} T={cfg.T} d_in={c.d_in} d_out={c.d_out}")
    y = run_moe(c, Wt)
    check_all("y", f64(y), oracle_y(c, Wt), TOL[cfg.dtype])


@pytest.mark.parametrize("name", ["tiny_fp32", "olmoe_bf16", "mixtral_bf16"])
def test_moe_base_only(name):
    cfg = SMALL[name]
    for path in ("expertwise", "down_expertwise"):
        c, Wt = case_and_weights(cfg, path, seed=1)
        y = run_moe(c, Wt, base_only=True)
        check_all("W_e x", f64(y), oracle_y(c, Wt, base_only=True), TOL[cfg.dtype])


@pytest.mark.parametrize("path", ["grouped", "down_expertwise", "pairs_per_pair"])
def test_moe_zero_base_is_the_adapter_update(path):
    """W = 0 leaves the adapter update alone, checked at the bf16 bar on its
    own scale (with W_e x present the update is a few percent of y)."""
    cfg = SMALL["olmoe_bf16"]
    c, Wt = case_and_weights(cfg, path, seed=2)
    y = run_moe(c, torch.zeros_like(Wt))
    ref = O.lora_delta(f64(c.x), f64(c.A), f64(c.B), c.ranks, cfg.alpha,
                       c.rt.topk_ids.astype(np.int64), cfg.E, c.e2g, c.n_keys,
                       input_mode=c.input_mode)
    check_all("adapter update", f64(y), ref, TOL["bf16"])


def test_moe_dropped_pairs_and_untouched_rows():
    cfg = SMALL["olmoe_bf16"]
    c, Wt = case_and_weights(cfg, "grouped", seed=3)
    ids = c.rt.topk_ids.copy()
    ids[::7, 0] = cfg.E + 5            # out of range: the pair is dropped
    c.rt.topk_ids[:] = ids
    y0 = torch.full((cfg.P, c.d_out), 7.0, dtype=c.x.dtype, device="cuda")
    y = run_moe(c, Wt, y=y0)
    dropped = np.arange(0, cfg.T, 7) * cfg.k
    yd = f64(y)
    assert np.all(yd[dropped] == 7.0)
    keep = np.setdiff1d(np.arange(cfg.P), dropped)
    check_all("y", yd[keep], oracle_y(c, Wt)[keep], TOL["bf16"])


def test_moe_empty_input():
    from paper_2609_06072_amd import ace
    cfg = SMALL["olmoe_bf16"].scaled(T=0)
    c, Wt = case_and_weights(cfg, "grouped")
    y = torch.zeros(0, c.d_out, dtype=torch.bfloat16, device="cuda")
    run_moe(c, Wt, y=y)
    assert ace.ace_last_error() == ""


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("r_e", [1, 3, 6])
def test_moe_odd_ranks(dtype, r_e):
    """Ranks that are not multiples of the fragment width take the masked
    loads of B."""
    cfg = W.CONFIGS["olmoe_bf16"].scaled(T=200, d_model=136, d_ffn=96, dtype=dtype, r_e=r_e)
    for path in ("grouped", "down_expertwise"):
        c, Wt = case_and_weights(cfg, path, seed=4)
        check_all("y", f64(run_moe(c, Wt)), oracle_y(c, Wt), TOL[dtype])


def test_moe_max_rank_and_many_experts():
    cfg = W.CONFIGS["olmoe_bf16"].scaled(T=150, d_model=128, d_ffn=64, r_e=64,
                                         groups=("consecutive", 4))
    c, Wt = case_and_weights(cfg, "grouped", seed=5)
    assert max(c.ranks) == 256
    check_all("y", f64(run_moe(c, Wt)), oracle_y(c, Wt), TOL["bf16"])
    cfg = W.CONFIGS["olmoe_bf16"].scaled(T=100, d_model=64, d_ffn=64, E=256, k=16, r_e=2,
                                         groups=("consecutive", 1))
    c, Wt = case_and_weights(cfg, "grouped", seed=6)
    assert c.n_keys == 256
    check_all("y", f64(run_moe(c, Wt)), oracle_y(c, Wt), TOL["bf16"])


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_moe_many_rows_per_expert(dtype):
    """At >= 1024 routed rows per expert on average the launch switches to
    256 x 256 tiles; ragged d_in, d_out and segment tails there too."""
    cfg = W.CONFIGS["mixtral_bf16"].scaled(T=2600, k=1, E=2, d_model=264, d_ffn=136, dtype=dtype,
                                           groups=("consecutive", 1))
    assert cfg.P >= 1024 * cfg.E
    for path in ("grouped", "down_expertwise"):
        c, Wt = case_and_weights(cfg, path, seed=11)
        check_all("y", f64(run_moe(c, Wt)), oracle_y(c, Wt), TOL[dtype])


def test_moe_deterministic():
    cfg = SMALL["qwen_bf16"]
    c, Wt = case_and_weights(cfg, "grouped", seed=7)
    a = run_moe(c, Wt)
    b = run_moe(c, Wt)
    assert torch.equal(a, b)


@pytest.mark.parametrize("name", ["olmoe_bf16", "qwen_bf16", "deepseek_bf16", "mixtral_bf16"])
@pytest.mark.parametrize("path", ["grouped", "expertwise", "down_expertwise"])
def test_moe_parity_full_size_sampled(name, path):
    cfg = W.CONFIGS[name]
    c, Wt = case_and_weights(cfg, path)
    say(f"moe full-size {name} {path} T={cfg.T} d_in={c.d_in} d_out={c.d_out}")
    y = run_moe(c, Wt)
    k = cfg.k
    rng = np.random.default_rng(321)
    toks = np.sort(rng.choice(cfg.T, size=min(32, cfg.T), replace=False))
    ids = c.rt.topk_ids[toks].astype(np.int64)
    if c.input_mode == W.INPUT_SHARED:
        x = f64(c.x[torch.as_tensor(toks, device="cuda")])
    else:
        pairs = (toks[:, None] * k + np.arange(k)[None, :]).ravel()
        x = f64(c.x[torch.as_tensor(pairs, device="cuda")])
    rows = (toks[:, None] * k + np.arange(k)[None, :]).ravel()
    ref = oracle_y(c, Wt, ids=ids, x=x)
    check_all("y(sampled tokens)", f64(y[torch.as_tensor(rows, device="cuda")]), ref,
              TOL[cfg.dtype])
