"""ace_group_permute_noalloc (the permutation with the library's static
scratch instead of a caller workspace) against ace_group_permute, bit for
bit, on two calls in a row, the second smaller than the first, then an
oversized problem that must be rejected before any launch."""
import numpy as np
import pytest
import torch

from paper_2609_06072_amd import workloads as W

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _compare(a, b, T, k):
    """Every meaningful entry of two routings of the same ids: the tables,
    and the first U rows / the routed pairs."""
    torch.cuda.synchronize()
    assert torch.equal(a.counts, b.counts) and torch.equal(a.offsets, b.offsets)
    U = int(a.offsets[-1])
    P = T * k
    if P > 0:
        assert torch.equal(a.row_token[:U], b.row_token[:U])
        assert torch.equal(a.row_slots[:U], b.row_slots[:U])
        assert torch.equal(a.pair_row[:P], b.pair_row[:P])
        n = int(a.row_pair[U])
        assert torch.equal(a.row_pair[:U + 1], b.row_pair[:U + 1])
        assert torch.equal(a.pair_list[:n], b.pair_list[:n])
    assert torch.equal(a.n_dropped, b.n_dropped)
    return U


def test_noalloc_permute_matches_workspace_permute():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a HIP device")
    from paper_2609_06072_amd import ace
    cases = [
        # (config, T, mode): the larger problem first, then a smaller one,
        # so the second call runs on a scratch that holds the first's tables
        ("olmoe_bf16", None, ace.ACE_ROWS_GROUP_DEDUP),
        ("qwen_bf16", 1001, ace.ACE_ROWS_EXPERT),
    ]
    for name, T, mode in cases:
        cfg = W.CONFIGS[name] if T is None else W.CONFIGS[name].scaled(T=T)
        rt = W.make_routing(cfg, seed=3)
        ids = torch.from_numpy(rt.topk_ids).cuda()
        ids[::9, 0] = cfg.E + 3            # some dropped pairs
        e2g = torch.from_numpy(rt.expert_to_group).cuda()
        n_keys = cfg.E if mode == ace.ACE_ROWS_EXPERT else rt.G
        need = ace.ace_workspace_bytes(ace.ACE_OP_PERMUTE, cfg.T, cfg.k, 0, 0, n_keys, 0)
        assert need <= ace.ACE_PERMUTE_SCRATCH_BYTES
        _say(f"noalloc permute {name} T={cfg.T} k={cfg.k} mode={mode} scratch {need} B")
        grp = None if mode == ace.ACE_ROWS_EXPERT else e2g
        ref = ace.ace_group_permute(ids, cfg.E, grp, rt.G, mode)
        out = ace.Routing(cfg.T, cfg.k, n_keys)
        ace.ace_group_permute_noalloc(ids, cfg.E, grp, rt.G, mode, out)
        U = _compare(out, ref, cfg.T, cfg.k)
        assert (out.c.n_keys, out.c.mode) == (n_keys, mode)
        assert U > 0 and ace.ace_routing_check(out) == ace.ace_routing_check(ref) > 0
    # a problem whose tables exceed the static scratch: rejected on the host
    T, k, E = 1 << 20, 8, 256
    big = ace.ace_workspace_bytes(ace.ACE_OP_PERMUTE, T, k, 0, 0, E, 0)
    assert big > ace.ACE_PERMUTE_SCRATCH_BYTES
    ids = torch.zeros(T, k, dtype=torch.int32, device="cuda")
    out = ace.Routing(T, k, E)
    with pytest.raises(ace.AceError) as ei:
        ace.ace_group_permute_noalloc(ids, E, None, E, ace.ACE_ROWS_EXPERT, out)
    assert ei.value.status == ace.ACE_ERR_UNSUPPORTED and "scratch" in str(ei.value)
