"""C-ABI checks that need no GPU: the library loads, exports every function
include/ace.h declares, and rejects bad arguments on the host before any
launch (no HIP call is reached on these paths).

The rejection tests hand the library fake device addresses.  Each asserts
the validation status it expects, never ACE_ERR_HIP: a case that got past
validation would fail here (the launch fails without a device) instead of
passing.  They are skipped where a device is visible, where such a launch
would dereference the fake addresses."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ace.h")


@pytest.fixture(scope="module")
def ace():
    from paper_2609_06072_amd import ace as mod
    return mod


@pytest.fixture
def no_device():
    import torch
    if torch.cuda.is_available():
        pytest.skip("fake device addresses are only passed where no kernel can be launched")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ace_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("ace_group_permute", "ace_grouped_lora_fwd", "ace_grouped_lora_bwd",
              "ace_expertwise_lora_fwd", "ace_expertwise_lora_bwd"):
        assert n in names


def test_exports_every_declared_symbol(ace):
    lib = ace.raw_lib()
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert set(declared_functions()) == set(ace.EXPORTS)


def test_workspace_bytes(ace):
    f = ace.ace_workspace_bytes(ace.ACE_OP_FWD, 4096, 8, 2048, 1024, 16, 32)
    assert f >= 4096 * 8 * 32 * 2 and f % 256 == 0     # h per row, r padded
    p = ace.ace_workspace_bytes(ace.ACE_OP_PERMUTE, 4096, 8, 0, 0, 64, 0)
    assert p > 0 and p % 256 == 0
    b1 = ace.ace_workspace_bytes(ace.ACE_OP_BWD, 4096, 8, 2048, 1024, 16, 32)
    b2 = ace.ace_workspace_bytes(ace.ACE_OP_BWD, 4096, 8, 2048, 1024, 16, 64)
    assert 0 < b1 < b2 and b1 % 256 == 0
    with pytest.raises(ace.AceError):
        ace.ace_workspace_bytes(ace.ACE_OP_BWD, 10, 0, 8, 8, 1, 1)
    with pytest.raises(ace.AceError):
        ace.ace_workspace_bytes(ace.ACE_OP_BWD, 10, 2, 8, 8, 300, 1)


def _routing(ace, T=4, k=2, n_keys=2, mode=0):
    # fake (never dereferenced) device addresses: validation fails before use
    r = ace.AceRouting(0x1000, 0x2000, 0x3000, 0x4000, 0x5000, 0x6000, 0x7000, 0x8000, n_keys, mode,
                       T, k)
    return r


def test_permute_rejects_bad_arguments(ace, no_device):
    lib = ace.raw_lib()
    r = _routing(ace)
    ws = ctypes.c_void_p(0x10000)
    ids = ctypes.c_void_p(0x20000)
    e2g = ctypes.c_void_p(0x30000)
    cases = [
        dict(k=0, status=ace.ACE_ERR_UNSUPPORTED),
        dict(k=33, status=ace.ACE_ERR_UNSUPPORTED),
        dict(E=0, status=ace.ACE_ERR_UNSUPPORTED),
        dict(E=257, status=ace.ACE_ERR_UNSUPPORTED),
        dict(G=257, status=ace.ACE_ERR_UNSUPPORTED),
        dict(T=-1, status=ace.ACE_ERR_INVALID_ARG),
        dict(mode=7, status=ace.ACE_ERR_INVALID_ARG),
        dict(e2g=None, status=ace.ACE_ERR_INVALID_ARG),
        dict(ids=None, status=ace.ACE_ERR_INVALID_ARG),
        dict(ws_bytes=4, status=ace.ACE_ERR_WORKSPACE),
        dict(T=1 << 27, k=16, status=ace.ACE_ERR_UNSUPPORTED),
    ]
    for c in cases:
        a = dict(ids=ids, T=4, k=2, E=8, e2g=e2g, G=2, mode=0, ws=ws, ws_bytes=1 << 20)
        a.update(c)
        st = lib.ace_group_permute(a["ids"], a["T"], a["k"], a["E"], a["e2g"], a["G"], a["mode"],
                                   ctypes.byref(r), a["ws"], a["ws_bytes"], None)
        assert st == c["status"], (c, ace.ace_last_error())
        assert ace.ace_last_error()
    assert lib.ace_group_permute(ids, 4, 2, 8, e2g, 2, 0, None, ws, 1 << 20, None) == ace.ACE_ERR_INVALID_ARG


def test_group_expert_permute_rejects_bad_arguments(ace, no_device):
    lib = ace.raw_lib()
    rg, re_ = _routing(ace), _routing(ace)
    ws = ctypes.c_void_p(0x10000)
    ids = ctypes.c_void_p(0x20000)
    e2g = ctypes.c_void_p(0x30000)
    need = (ace.ace_workspace_bytes(ace.ACE_OP_PERMUTE, 4, 2, 0, 0, 2, 0)
            + ace.ace_workspace_bytes(ace.ACE_OP_PERMUTE, 4, 2, 0, 0, 8, 0))
    cases = [
        dict(k=0, status=ace.ACE_ERR_UNSUPPORTED),
        dict(E=257, status=ace.ACE_ERR_UNSUPPORTED),
        dict(G=0, status=ace.ACE_ERR_UNSUPPORTED),
        dict(T=-1, status=ace.ACE_ERR_INVALID_ARG),
        dict(mode=ace.ACE_ROWS_EXPERT, status=ace.ACE_ERR_INVALID_ARG),   # not a group mode
        dict(mode=7, status=ace.ACE_ERR_INVALID_ARG),
        dict(e2g=None, status=ace.ACE_ERR_INVALID_ARG),
        dict(ids=None, status=ace.ACE_ERR_INVALID_ARG),
        dict(same=True, status=ace.ACE_ERR_INVALID_ARG),
        dict(ws_bytes=need - 4, status=ace.ACE_ERR_WORKSPACE),            # one routing's worth
        dict(ws=None, status=ace.ACE_ERR_WORKSPACE),
    ]
    for c in cases:
        a = dict(ids=ids, T=4, k=2, E=8, e2g=e2g, G=2, mode=0, ws=ws, ws_bytes=need, same=False)
        a.update(c)
        st = lib.ace_group_expert_permute(a["ids"], a["T"], a["k"], a["E"], a["e2g"], a["G"],
                                          a["mode"], ctypes.byref(rg),
                                          ctypes.byref(rg if a["same"] else re_), a["ws"],
                                          a["ws_bytes"], None)
        assert st == c["status"], (c, ace.ace_last_error())
        assert ace.ace_last_error()
    assert lib.ace_group_expert_permute(ids, 4, 2, 8, e2g, 2, 0, None, ctypes.byref(re_), ws, need,
                                        None) == ace.ACE_ERR_INVALID_ARG


def test_forward_backward_reject_bad_arguments(ace, no_device):
    lib = ace.raw_lib()
    ranks = (ctypes.c_int32 * 2)(16, 16)
    p = ctypes.c_void_p(0x100000)      # 16-byte aligned fake device address
    bad = ctypes.c_void_p(0x100002)

    def fwd(**kw):
        a = dict(dtype=ace.ACE_BF16, im=0, T=4, k=2, d_in=64, d_out=32, G=2, ranks=ranks,
                 alpha=16.0, x=p, A=p, B=p, w=None, rt=_routing(ace), y=p)
        a.update(kw)
        return lib.ace_grouped_lora_fwd(a["dtype"], a["im"], a["T"], a["k"], a["d_in"], a["d_out"],
                                        a["G"], a["ranks"], a["alpha"], a["x"], a["A"], a["B"],
                                        a["w"], ctypes.byref(a["rt"]), a["y"], None, 0, None)

    assert fwd(dtype=5) == ace.ACE_ERR_INVALID_ARG
    assert fwd(im=3) == ace.ACE_ERR_INVALID_ARG
    assert fwd(d_in=60) == ace.ACE_ERR_UNSUPPORTED          # bf16 rows need multiples of 8
    assert fwd(dtype=ace.ACE_F32, d_in=60) == ace.ACE_ERR_WORKSPACE  # fp32 accepts it; no ws
    assert fwd(G=0) == ace.ACE_ERR_UNSUPPORTED
    assert fwd(ranks=(ctypes.c_int32 * 2)(16, 300)) == ace.ACE_ERR_UNSUPPORTED
    assert fwd(ranks=(ctypes.c_int32 * 2)(0, 16)) == ace.ACE_ERR_UNSUPPORTED
    assert fwd(ranks=None) == ace.ACE_ERR_INVALID_ARG
    assert fwd(alpha=float("nan")) == ace.ACE_ERR_INVALID_ARG
    assert fwd(x=bad) == ace.ACE_ERR_INVALID_ARG
    assert fwd(y=bad) == ace.ACE_ERR_INVALID_ARG
    assert fwd(rt=_routing(ace, T=5)) == ace.ACE_ERR_INVALID_ARG      # built for another T
    assert fwd(rt=_routing(ace, n_keys=3)) == ace.ACE_ERR_INVALID_ARG
    assert fwd(rt=_routing(ace, mode=ace.ACE_ROWS_EXPERT)) == ace.ACE_ERR_INVALID_ARG
    assert fwd(rt=_routing(ace, mode=ace.ACE_ROWS_GROUP_DEDUP), im=1) == ace.ACE_ERR_INVALID_ARG
    assert fwd(k=40) == ace.ACE_ERR_UNSUPPORTED
    # expert-wise calls want expert-keyed routing
    st = lib.ace_expertwise_lora_fwd(ace.ACE_BF16, 0, 4, 2, 64, 32, 2, 8, 16.0, p, p, p, None,
                                     ctypes.byref(_routing(ace, mode=0)), p, None, 0, None)
    assert st == ace.ACE_ERR_INVALID_ARG
    # backward: workspace checked before anything runs
    st = lib.ace_grouped_lora_bwd(ace.ACE_BF16, 0, 4, 2, 64, 32, 2, ranks, 16.0, p, p, p, None,
                                  ctypes.byref(_routing(ace)), None, p, p, p, p, p, 16, None)
    assert st == ace.ACE_ERR_WORKSPACE
    st = lib.ace_grouped_lora_bwd(ace.ACE_BF16, 0, 4, 2, 64, 32, 2, ranks, 16.0, p, p, p, None,
                                  ctypes.byref(_routing(ace)), None, p, p, None, p, p, 1 << 30,
                                  None)
    assert st == ace.ACE_ERR_INVALID_ARG
    # h_fwd must be a forward workspace (256-byte aligned)
    h_bad = ctypes.c_void_p(0x100010)
    st = lib.ace_grouped_lora_bwd(ace.ACE_BF16, 0, 4, 2, 64, 32, 2, ranks, 16.0, p, p, p, None,
                                  ctypes.byref(_routing(ace)), h_bad, p, p, p, p, p, 1 << 30, None)
    assert st == ace.ACE_ERR_INVALID_ARG


def test_cka_rejects_bad_arguments(ace, no_device):
    lib = ace.raw_lib()
    ws = ctypes.c_void_p(0x10000)
    X, A, B, S = (ctypes.c_void_p(a) for a in (0x1000, 0x2000, 0x3000, 0x4000))
    ok_ws = ace.ace_workspace_bytes(ace.ACE_OP_CKA, 100, 1, 64, 32, 8, 4)
    assert ok_ws > 0 and ok_ws % 256 == 0
    inv, uns, wsp = ace.ACE_ERR_INVALID_ARG, ace.ACE_ERR_UNSUPPORTED, ace.ACE_ERR_WORKSPACE
    cases = [
        (7, 100, 64, 32, 8, 4, ok_ws, inv),        # unknown dtype
        (1, 100, 64, 32, 8, 65, ok_ws, uns),       # rank above 64
        (1, 100, 64, 32, 0, 4, ok_ws, uns),        # no experts
        (1, 100, 60, 32, 8, 4, ok_ws, uns),        # d_in not a multiple of 8 (bf16)
        (1, -1, 64, 32, 8, 4, ok_ws, inv),         # negative probe size
        (1, 100, 64, 32, 8, 4, ok_ws - 256, wsp),  # workspace too small
    ]
    for dt, N, d_in, d_out, E, r, wsb, want in cases:
        st = lib.ace_pairwise_cka(dt, N, d_in, d_out, E, r, X, A, B, S, ws, wsb, None)
        assert st == want, (dt, N, d_in, d_out, E, r, wsb, st, ace.ace_last_error())
        assert ace.ace_last_error()
    with pytest.raises(ace.AceError):
        ace.ace_workspace_bytes(ace.ACE_OP_CKA, 100, 1, 64, 32, 8, 65)



def test_moe_fwd_rejects_bad_arguments(ace, no_device):
    lib = ace.raw_lib()
    T, k, E, G = 4, 2, 4, 2
    ert = _routing(ace, T, k, n_keys=E, mode=ace.ACE_ROWS_EXPERT)
    art = _routing(ace, T, k, n_keys=G, mode=ace.ACE_ROWS_GROUP_DEDUP)
    ranks = (ctypes.c_int32 * G)(8, 8)
    ekey = (ctypes.c_int32 * E)(0, 1, 0, 1)
    bad_key = (ctypes.c_int32 * E)(0, 1, 2, 1)
    x, W, A, B, y = (ctypes.c_void_p(a) for a in (0x1000, 0x2000, 0x3000, 0x4000, 0x5000))
    ws = ctypes.c_void_p(0x100000)
    need = ace.ace_workspace_bytes(ace.ACE_OP_FWD, T, k, 64, 32, G, 8)
    base = dict(dt=1, im=0, T=T, k=k, d_in=64, d_out=32, E=E, x=x, W=W, ert=ert, n_keys=G,
                ranks=ranks, ekey=ekey, A=A, B=B, art=art, y=y, ws=ws, wsb=need)
    inv, uns, wsp = ace.ACE_ERR_INVALID_ARG, ace.ACE_ERR_UNSUPPORTED, ace.ACE_ERR_WORKSPACE
    cases = [
        (dict(dt=7), inv),                         # unknown dtype
        (dict(im=ace.ACE_INPUT_COMBINED), inv),    # combined output is not a projection
        (dict(d_in=60), uns),                      # not a multiple of 8 (bf16)
        (dict(E=3), inv),                          # expert routing has 4 keys
        (dict(ert=art), inv),                      # not expert-keyed
        (dict(W=None), inv),
        (dict(ekey=bad_key), inv),                 # key outside [0, G)
        (dict(ranks=None), inv),
        (dict(wsb=256), wsp),                      # below h per pair (P * 32 * 4 bytes)
        (dict(ws=None), wsp),
        (dict(im=ace.ACE_INPUT_PER_PAIR), inv),    # dedup rows need the shared input
        (dict(n_keys=-1), inv),
    ]
    for c, want in cases:
        a = dict(base, **c)
        st = lib.ace_moe_lora_fwd(a["dt"], a["im"], a["T"], a["k"], a["d_in"], a["d_out"], a["E"],
                                  a["x"], a["W"], ctypes.byref(a["ert"]), a["n_keys"], a["ranks"],
                                  a["ekey"], 16.0, a["A"], a["B"], ctypes.byref(a["art"]), a["y"],
                                  a["ws"], a["wsb"], None)
        assert st == want, (c, st, ace.ace_last_error())
    # expert-keyed adapter rows need the identity key map
    ert2 = _routing(ace, T, k, n_keys=E, mode=ace.ACE_ROWS_EXPERT)
    r4 = (ctypes.c_int32 * E)(8, 8, 8, 8)
    st = lib.ace_moe_lora_fwd(1, 0, T, k, 64, 32, E, x, W, ctypes.byref(ert), E, r4, ekey, 16.0,
                              A, B, ctypes.byref(ert2), y, ws, need * 2, None)
    assert st == ace.ACE_ERR_INVALID_ARG


def test_row_pair_required_at_every_size(ace, no_device):
    """row_pair has P + 1 entries, so it exists at T = 0 too (the permutation
    writes its last entry, the pair count): a NULL row_pair is rejected by
    both permutation calls and by the forward even when T = 0."""
    lib = ace.raw_lib()
    ws = ctypes.c_void_p(0x10000)
    ids = ctypes.c_void_p(0x20000)
    e2g = ctypes.c_void_p(0x30000)

    def no_row_pair(mode=0, n_keys=2):
        return ace.AceRouting(0x1000, 0x2000, 0x3000, 0x4000, 0x5000, 0x6000, None, 0x8000,
                              n_keys, mode, 0, 2)

    st = lib.ace_group_permute(ids, 0, 2, 8, e2g, 2, 0, ctypes.byref(no_row_pair()), ws, 1 << 20,
                               None)
    assert st == ace.ACE_ERR_INVALID_ARG, ace.ace_last_error()
    need = (ace.ace_workspace_bytes(ace.ACE_OP_PERMUTE, 0, 2, 0, 0, 2, 0)
            + ace.ace_workspace_bytes(ace.ACE_OP_PERMUTE, 0, 2, 0, 0, 8, 0))
    st = lib.ace_group_expert_permute(ids, 0, 2, 8, e2g, 2, 0, ctypes.byref(_routing(ace, T=0)),
                                      ctypes.byref(no_row_pair(ace.ACE_ROWS_EXPERT, 8)), ws,
                                      max(need, 256), None)
    assert st == ace.ACE_ERR_INVALID_ARG, ace.ace_last_error()
    ranks = (ctypes.c_int32 * 2)(16, 16)
    p = ctypes.c_void_p(0x100000)
    st = lib.ace_grouped_lora_fwd(ace.ACE_BF16, 0, 0, 2, 64, 32, 2, ranks, 16.0, p, p, p, None,
                                  ctypes.byref(no_row_pair()), p, p, 1 << 20, None)
    assert st == ace.ACE_ERR_INVALID_ARG, ace.ace_last_error()


def test_noalloc_permute_rejects_oversized_problem(ace, no_device):
    """The no-allocation permutation refuses, before any HIP call, a problem
    whose count tables exceed its static scratch."""
    lib = ace.raw_lib()
    T, k, E = 1 << 20, 8, 256
    assert ace.ace_workspace_bytes(ace.ACE_OP_PERMUTE, T, k, 0, 0, E, 0) > ace.ACE_PERMUTE_SCRATCH_BYTES
    r = _routing(ace, T=T, k=k, n_keys=E, mode=ace.ACE_ROWS_EXPERT)
    st = lib.ace_group_permute_noalloc(ctypes.c_void_p(0x20000), T, k, E, None, E,
                                       ace.ACE_ROWS_EXPERT, ctypes.byref(r), None)
    assert st == ace.ACE_ERR_UNSUPPORTED, ace.ace_last_error()
    assert "scratch" in ace.ace_last_error()
