"""Synthetic workload generator: seeds, shapes, budget identity, skew."""
import numpy as np
import pytest

from paper_2609_06072_amd import workloads as W


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
def test_budget_identity(name):
    """Sec. 3.3: sum_g r_g (d_in + d_out) = sum_e r_e (d_in + d_out)."""
    cfg = W.CONFIGS[name]
    rt = W.make_routing(cfg, seed=0)
    assert int(rt.group_rank.sum()) == cfg.E * cfg.r_e
    for proj in cfg.projections:
        d_in, d_out, _ = cfg.proj_dims(proj)
        assert W.budget(rt.group_rank, d_in, d_out) == W.budget([cfg.r_e] * cfg.E, d_in, d_out)


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
def test_routing_shapes_and_determinism(name):
    cfg = W.CONFIGS[name]
    a = W.make_routing(cfg, seed=0)
    b = W.make_routing(cfg, seed=0)
    c = W.make_routing(cfg, seed=1)
    assert a.topk_ids.shape == (cfg.T, cfg.k) and a.topk_ids.dtype == np.int32
    assert np.array_equal(a.topk_ids, b.topk_ids) and np.array_equal(a.expert_to_group, b.expert_to_group)
    assert not np.array_equal(a.topk_ids, c.topk_ids)
    # distinct experts per token, in range
    assert (a.topk_ids >= 0).all() and (a.topk_ids < cfg.E).all()
    s = np.sort(a.topk_ids, axis=1)
    assert (np.diff(s, axis=1) > 0).all()
    # weights are softmax probabilities, in descending order
    assert (np.diff(a.topk_w, axis=1) <= 0).all() and (a.topk_w.sum(1) <= 1 + 1e-6).all()


def test_group_structures():
    assert list(W.make_routing(W.CONFIGS["tiny_fp32"]).expert_to_group) == [0, 0, 1, 1, 2, 2, 3, 3]
    for name, G, size in (("olmoe_bf16", 16, 4), ("qwen_bf16", 15, 4), ("mixtral_bf16", 2, 4)):
        rt = W.make_routing(W.CONFIGS[name])
        assert rt.G == G and set(np.bincount(rt.expert_to_group)) == {size}
    rt = W.make_routing(W.CONFIGS["deepseek_bf16"])
    sizes = np.bincount(rt.expert_to_group)
    assert sizes.sum() == 64 and set(sizes) <= {2, 4, 8}
    assert list(rt.group_rank) == list(8 * sizes)


def test_zipf_skew():
    cfg = W.CONFIGS["olmoe_bf16"]
    st = W.describe(cfg, W.make_routing(cfg))
    assert 0.85 < st["load_entropy"] < 0.97 and st["max_over_mean_load"] > 3
    cfg = W.CONFIGS["mixtral_bf16"]
    st = W.describe(cfg, W.make_routing(cfg))
    assert st["load_entropy"] > 0.99


def test_bf16_rounding():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 3.14159], dtype=np.float32)
    r = W.round_bf16_np(x)
    assert r[0] == 1.0 and r[1] == 1.0 and r[2] == np.float32(1.0 + 2 ** -6) and r[3] == -2.5
    torch = pytest.importorskip("torch")
    t = torch.from_numpy(x).to(torch.bfloat16).float().numpy()
    assert np.array_equal(t, r)


def test_tensor_draws():
    cfg = W.CONFIGS["olmoe_bf16"].scaled(T=64, d_model=128, d_ffn=96)
    rt = W.make_routing(cfg)
    t = W.make_proj(cfg, "gate", rt.group_rank)
    import torch
    assert t.x.shape == (64, 128) and t.x.dtype == torch.bfloat16
    assert t.A.shape == (int(rt.group_rank.sum()), 128)
    assert t.B.shape == (96 * int(rt.group_rank.sum()),)
    assert t.dy.shape == (cfg.P, 96)
    t2 = W.make_proj(cfg, "gate", rt.group_rank)
    assert torch.equal(t.A, t2.A)
    d = W.make_proj(cfg, "down", [cfg.r_e] * cfg.E)
    assert d.x.shape == (cfg.P, 96) and d.d_out == 128
