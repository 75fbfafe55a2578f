"""ctypes binding of libace (include/ace.h).

Argument marshalling only: torch supplies device memory and the current HIP
stream; every step of the computation runs in the library's HIP kernels.
Importing this module loads libace.so and raises if it is missing -- there is
no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libace.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"libace.so not found at {LIB_PATH}; build it with "
                      "`python -m paper_2609_06072_amd.build`")
_lib = ctypes.CDLL(LIB_PATH)

ACE_OK, ACE_ERR_INVALID_ARG, ACE_ERR_UNSUPPORTED, ACE_ERR_WORKSPACE, ACE_ERR_HIP = 0, -1, -2, -3, -4
ACE_F32, ACE_BF16 = 0, 1
ACE_ROWS_GROUP_DEDUP, ACE_ROWS_GROUP_PAIRS, ACE_ROWS_EXPERT = 0, 1, 2
ACE_INPUT_SHARED, ACE_INPUT_PER_PAIR, ACE_INPUT_COMBINED = 0, 1, 2
ACE_OP_PERMUTE, ACE_OP_FWD, ACE_OP_BWD, ACE_OP_CKA = 0, 1, 2, 3

EXPORTS = ("ace_group_permute", "ace_group_expert_permute", "ace_grouped_lora_fwd", "ace_grouped_lora_bwd",
           "ace_expertwise_lora_fwd", "ace_expertwise_lora_bwd", "ace_workspace_bytes",
           "ace_routing_check", "ace_last_error", "ace_pairwise_cka", "ace_similarity_graph",
           "ace_louvain", "ace_group_anchors", "ace_consolidate_adapters", "ace_moe_lora_fwd",
           "ace_group_permute_noalloc")
ACE_PERMUTE_SCRATCH_BYTES = 4 << 20


class AceRouting(ctypes.Structure):
    _fields_ = [("counts", ctypes.c_void_p), ("offsets", ctypes.c_void_p),
                ("row_token", ctypes.c_void_p), ("row_slots", ctypes.c_void_p),
                ("pair_row", ctypes.c_void_p), ("n_dropped", ctypes.c_void_p),
                ("row_pair", ctypes.c_void_p), ("pair_list", ctypes.c_void_p),
                ("n_keys", ctypes.c_int32), ("mode", ctypes.c_int32),
                ("T", ctypes.c_int32), ("k", ctypes.c_int32)]


_i32, _f32, _vp, _sz = ctypes.c_int32, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t
_R = ctypes.POINTER(AceRouting)
_lib.ace_group_permute.argtypes = [_vp, _i32, _i32, _i32, _vp, _i32, _i32, _R, _vp, _sz, _vp]
_lib.ace_group_permute.restype = _i32
_lib.ace_group_permute_noalloc.argtypes = [_vp, _i32, _i32, _i32, _vp, _i32, _i32, _R, _vp]
_lib.ace_group_permute_noalloc.restype = _i32
_lib.ace_group_expert_permute.argtypes = [_vp, _i32, _i32, _i32, _vp, _i32, _i32, _R, _R, _vp, _sz,
                                          _vp]
_lib.ace_group_expert_permute.restype = _i32
_FWD = [_i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _f32, _vp, _vp, _vp, _vp, _R, _vp, _vp, _sz, _vp]
_BWD = [_i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _f32, _vp, _vp, _vp, _vp, _R, _vp, _vp, _vp,
        _vp, _vp, _vp, _sz, _vp]
_lib.ace_grouped_lora_fwd.argtypes = _FWD
_lib.ace_grouped_lora_fwd.restype = _i32
_lib.ace_grouped_lora_bwd.argtypes = _BWD
_lib.ace_grouped_lora_bwd.restype = _i32
_EFWD = list(_FWD)
_EFWD[7] = _i32          # rank instead of group_rank pointer
_EBWD = list(_BWD)
_EBWD[7] = _i32
_lib.ace_expertwise_lora_fwd.argtypes = _EFWD
_lib.ace_expertwise_lora_fwd.restype = _i32
_lib.ace_expertwise_lora_bwd.argtypes = _EBWD
_lib.ace_expertwise_lora_bwd.restype = _i32
_lib.ace_workspace_bytes.argtypes = [_i32, _i32, _i32, _i32, _i32, _i32, _i32]
_lib.ace_workspace_bytes.restype = _sz
_lib.ace_routing_check.argtypes = [_R, ctypes.POINTER(ctypes.c_int32), _vp]
_lib.ace_routing_check.restype = _i32
_lib.ace_pairwise_cka.argtypes = [_i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _sz,
                                  _vp]
_lib.ace_pairwise_cka.restype = _i32
_lib.ace_similarity_graph.argtypes = [_vp, _i32, _vp]
_lib.ace_similarity_graph.restype = _i32
_lib.ace_louvain.argtypes = [_vp, _i32, ctypes.c_double, _vp, ctypes.POINTER(ctypes.c_int32)]
_lib.ace_louvain.restype = _i32
_lib.ace_group_anchors.argtypes = [_vp, _i32, _vp, _i32, _vp]
_lib.ace_group_anchors.restype = _i32
_lib.ace_consolidate_adapters.argtypes = [_i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _i32, _vp,
                                          _vp, _vp, _vp, _vp, _vp]
_lib.ace_consolidate_adapters.restype = _i32
_lib.ace_moe_lora_fwd.argtypes = [_i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _R, _i32, _vp,
                                  _vp, _f32, _vp, _vp, _R, _vp, _vp, _sz, _vp]
_lib.ace_moe_lora_fwd.restype = _i32
_lib.ace_last_error.argtypes = []
_lib.ace_last_error.restype = ctypes.c_char_p


class AceError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where} failed with status {status}: {ace_last_error()}")


def ace_last_error() -> str:
    return _lib.ace_last_error().decode()


def _check(status: int, where: str) -> None:
    if status != ACE_OK:
        raise AceError(status, where)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libace must be contiguous")
    return t.data_ptr() or None


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream or None


def _dtype(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return ACE_BF16
    if t.dtype == torch.float32:
        return ACE_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _want(name: str, t, numel: Optional[int] = None, dtype=None, device=None,
          optional: bool = False) -> None:
    """Host-side shape/type check of one argument before the call (the
    library sees only pointers): numel, dtype and device must match."""
    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")


def _check_lora_args(x, A, B, ranks: Sequence[int], routing: "Routing", d_out: int,
                     input_mode: int, pair_w, y=None, dy=None, dx=None, dA=None, dB=None) -> None:
    T, k = routing.c.T, routing.c.k
    R = int(sum(int(r) for r in ranks))
    dt, dev = A.dtype, A.device
    if A.dim() != 2 or A.shape[0] != R:
        raise ValueError(f"A must be [R={R}, d_in], got {tuple(A.shape)}")
    d_in = A.shape[1]
    rows_in = T if input_mode == ACE_INPUT_SHARED else T * k
    rows_out = T if input_mode == ACE_INPUT_COMBINED else T * k
    _want("x", x, rows_in * d_in, dt, dev)
    _want("B", B, R * d_out, dt, dev)
    _want("pair_w", pair_w, T * k, torch.float32, dev, optional=True)
    if y is not None:
        _want("y", y, rows_out * d_out, dt, dev)
    if dy is not None:
        _want("dy", dy, rows_out * d_out, dt, dev)
        _want("dx", dx, rows_in * d_in, dt, dev)
        _want("dA", dA, R * d_in, torch.float32, dev)
        _want("dB", dB, R * d_out, torch.float32, dev)
    if routing.n_keys != len(ranks):
        raise ValueError(f"routing has {routing.n_keys} keys, the call has {len(ranks)}")


def ace_workspace_bytes(op: int, T: int, k: int, d_in: int, d_out: int, n_keys: int,
                        r_max: int) -> int:
    n = _lib.ace_workspace_bytes(op, T, k, d_in, d_out, n_keys, r_max)
    if n == ctypes.c_size_t(-1).value:
        raise AceError(ACE_ERR_INVALID_ARG, "ace_workspace_bytes")
    return int(n)


class Routing:
    """Owns the device arrays of an ace_routing (sized for T*k pairs)."""

    def __init__(self, T: int, k: int, n_keys: int, device="cuda"):
        P = max(1, T * k)
        i32 = dict(dtype=torch.int32, device=device)
        self.counts = torch.zeros(n_keys, **i32)
        self.offsets = torch.zeros(n_keys + 1, **i32)
        self.row_token = torch.zeros(P, **i32)
        self.row_slots = torch.zeros(P, **i32)
        self.pair_row = torch.zeros(P, **i32)
        self.n_dropped = torch.zeros(1, **i32)
        self.row_pair = torch.zeros(P + 1, **i32)
        self.pair_list = torch.zeros(P, **i32)
        self.c = AceRouting(self.counts.data_ptr(), self.offsets.data_ptr(),
                            self.row_token.data_ptr(), self.row_slots.data_ptr(),
                            self.pair_row.data_ptr(), self.n_dropped.data_ptr(),
                            self.row_pair.data_ptr(), self.pair_list.data_ptr(), n_keys, -1, T, k)

    def check_capacity(self, T: int, k: int, n_keys: int) -> None:
        """The arrays must hold a permutation of T*k pairs over n_keys keys."""
        P = max(1, T * k)
        if self.row_token.numel() < P or self.row_pair.numel() < P + 1:
            raise ValueError(f"routing holds {self.row_token.numel()} pairs, the call needs {P}")
        if self.counts.numel() != n_keys:
            raise ValueError(f"routing has room for {self.counts.numel()} keys, the call has {n_keys}")

    @property
    def n_keys(self) -> int:
        return self.c.n_keys

    @property
    def mode(self) -> int:
        return self.c.mode


def ace_group_permute(topk_ids: torch.Tensor, E: int, expert_to_group: Optional[torch.Tensor],
                      G: int, mode: int, routing: Optional[Routing] = None,
                      ws: Optional[torch.Tensor] = None, stream=None) -> Routing:
    T, k = topk_ids.shape
    n_keys = E if mode == ACE_ROWS_EXPERT else G
    _want("topk_ids", topk_ids, dtype=torch.int32)
    _want("expert_to_group", expert_to_group, E, torch.int32, topk_ids.device, optional=True)
    if routing is None:
        routing = Routing(T, k, n_keys, device=topk_ids.device)
    routing.check_capacity(T, k, n_keys)
    need = ace_workspace_bytes(ACE_OP_PERMUTE, T, k, 0, 0, n_keys, 0)
    if ws is None:
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=topk_ids.device)
    _check(_lib.ace_group_permute(_ptr(topk_ids), T, k, E, _ptr(expert_to_group), G, mode,
                                  ctypes.byref(routing.c), _ptr(ws), ws.numel(), _stream(stream)),
           "ace_group_permute")
    return routing


def ace_group_permute_noalloc(topk_ids: torch.Tensor, E: int,
                              expert_to_group: Optional[torch.Tensor], G: int, mode: int,
                              routing: Routing, stream=None) -> Routing:
    """ace_group_permute with the library's static scratch instead of a
    workspace: allocates nothing (the caller passes the routing arrays)."""
    T, k = topk_ids.shape
    n_keys = E if mode == ACE_ROWS_EXPERT else G
    _want("topk_ids", topk_ids, dtype=torch.int32)
    _want("expert_to_group", expert_to_group, E, torch.int32, topk_ids.device, optional=True)
    routing.check_capacity(T, k, n_keys)
    _check(_lib.ace_group_permute_noalloc(_ptr(topk_ids), T, k, E, _ptr(expert_to_group), G,
                                          mode, ctypes.byref(routing.c), _stream(stream)),
           "ace_group_permute_noalloc")
    return routing


def ace_group_expert_permute(topk_ids: torch.Tensor, E: int, expert_to_group: torch.Tensor,
                             G: int, group_mode: int = ACE_ROWS_GROUP_DEDUP,
                             group_routing: Optional[Routing] = None,
                             expert_routing: Optional[Routing] = None,
                             ws: Optional[torch.Tensor] = None, stream=None):
    """Group-keyed and expert-keyed routings from one pass over topk_ids."""
    T, k = topk_ids.shape
    _want("topk_ids", topk_ids, dtype=torch.int32)
    _want("expert_to_group", expert_to_group, E, torch.int32, topk_ids.device)
    if group_routing is None:
        group_routing = Routing(T, k, G, device=topk_ids.device)
    if expert_routing is None:
        expert_routing = Routing(T, k, E, device=topk_ids.device)
    group_routing.check_capacity(T, k, G)
    expert_routing.check_capacity(T, k, E)
    need = (ace_workspace_bytes(ACE_OP_PERMUTE, T, k, 0, 0, G, 0)
            + ace_workspace_bytes(ACE_OP_PERMUTE, T, k, 0, 0, E, 0))
    if ws is None:
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=topk_ids.device)
    _check(_lib.ace_group_expert_permute(_ptr(topk_ids), T, k, E, _ptr(expert_to_group), G,
                                         group_mode, ctypes.byref(group_routing.c),
                                         ctypes.byref(expert_routing.c), _ptr(ws), ws.numel(),
                                         _stream(stream)),
           "ace_group_expert_permute")
    return group_routing, expert_routing


def ace_routing_check(routing: Routing, stream=None) -> int:
    n = ctypes.c_int32(0)
    _check(_lib.ace_routing_check(ctypes.byref(routing.c), ctypes.byref(n), _stream(stream)),
           "ace_routing_check")
    return int(n.value)


def _ranks_arg(ranks: Sequence[int]):
    arr = (ctypes.c_int32 * len(ranks))(*[int(r) for r in ranks])
    return arr


def _fwd_ws(ws, T, k, d_in, d_out, n_keys, r_max, device):
    if ws is not None:
        return ws
    need = ace_workspace_bytes(ACE_OP_FWD, T, k, d_in, d_out, n_keys, r_max)
    return torch.empty(max(need, 256), dtype=torch.uint8, device=device)


def ace_grouped_lora_fwd(x, A, B, group_rank: Sequence[int], alpha: float, routing: Routing,
                         y, pair_w=None, input_mode: int = ACE_INPUT_SHARED, ws=None,
                         stream=None) -> None:
    T, k = routing.c.T, routing.c.k
    d_in, d_out = A.shape[1], y.shape[1]
    _check_lora_args(x, A, B, group_rank, routing, d_out, input_mode, pair_w, y=y)
    ranks = _ranks_arg(group_rank)
    ws = _fwd_ws(ws, T, k, d_in, d_out, len(group_rank), max(group_rank), A.device)
    _check(_lib.ace_grouped_lora_fwd(_dtype(x), input_mode, T, k, d_in, d_out, len(group_rank),
                                     ranks, alpha, _ptr(x), _ptr(A), _ptr(B), _ptr(pair_w),
                                     ctypes.byref(routing.c), _ptr(y), _ptr(ws),
                                     0 if ws is None else ws.numel(), _stream(stream)),
           "ace_grouped_lora_fwd")


def ace_grouped_lora_bwd(x, A, B, group_rank: Sequence[int], alpha: float, routing: Routing,
                         dy, dx, dA, dB, pair_w=None, input_mode: int = ACE_INPUT_SHARED,
                         ws=None, stream=None, h_fwd=None) -> None:
    """h_fwd: None, or the workspace of the forward call with the same arguments
    (the backward then reuses the forward's h instead of recomputing it)."""
    T, k = routing.c.T, routing.c.k
    d_in, d_out = A.shape[1], dy.shape[1]
    _check_lora_args(x, A, B, group_rank, routing, d_out, input_mode, pair_w, dy=dy, dx=dx,
                     dA=dA, dB=dB)
    ranks = _ranks_arg(group_rank)
    if ws is None:
        need = ace_workspace_bytes(ACE_OP_BWD, T, k, d_in, d_out, len(group_rank), max(group_rank))
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=A.device)
    _check(_lib.ace_grouped_lora_bwd(_dtype(A), input_mode, T, k, d_in, d_out, len(group_rank),
                                     ranks, alpha, _ptr(x), _ptr(A), _ptr(B), _ptr(pair_w),
                                     ctypes.byref(routing.c), _ptr(h_fwd), _ptr(dy), _ptr(dx),
                                     _ptr(dA), _ptr(dB), _ptr(ws), ws.numel(), _stream(stream)),
           "ace_grouped_lora_bwd")


def ace_expertwise_lora_fwd(x, A, B, E: int, rank: int, alpha: float, routing: Routing, y,
                            pair_w=None, input_mode: int = ACE_INPUT_SHARED, ws=None,
                            stream=None) -> None:
    T, k = routing.c.T, routing.c.k
    d_in, d_out = A.shape[1], y.shape[1]
    _check_lora_args(x, A, B, [rank] * E, routing, d_out, input_mode, pair_w, y=y)
    ws = _fwd_ws(ws, T, k, d_in, d_out, E, rank, A.device)
    _check(_lib.ace_expertwise_lora_fwd(_dtype(x), input_mode, T, k, d_in, d_out, E, rank, alpha,
                                        _ptr(x), _ptr(A), _ptr(B), _ptr(pair_w),
                                        ctypes.byref(routing.c), _ptr(y), _ptr(ws),
                                        0 if ws is None else ws.numel(), _stream(stream)),
           "ace_expertwise_lora_fwd")


def ace_expertwise_lora_bwd(x, A, B, E: int, rank: int, alpha: float, routing: Routing, dy, dx,
                            dA, dB, pair_w=None, input_mode: int = ACE_INPUT_SHARED, ws=None,
                            stream=None, h_fwd=None) -> None:
    T, k = routing.c.T, routing.c.k
    d_in, d_out = A.shape[1], dy.shape[1]
    _check_lora_args(x, A, B, [rank] * E, routing, d_out, input_mode, pair_w, dy=dy, dx=dx,
                     dA=dA, dB=dB)
    if ws is None:
        need = ace_workspace_bytes(ACE_OP_BWD, T, k, d_in, d_out, E, rank)
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=A.device)
    _check(_lib.ace_expertwise_lora_bwd(_dtype(A), input_mode, T, k, d_in, d_out, E, rank, alpha,
                                        _ptr(x), _ptr(A), _ptr(B), _ptr(pair_w),
                                        ctypes.byref(routing.c), _ptr(h_fwd), _ptr(dy), _ptr(dx),
                                        _ptr(dA), _ptr(dB), _ptr(ws), ws.numel(),
                                        _stream(stream)),
           "ace_expertwise_lora_bwd")


def ace_pairwise_cka(X, A, B, E: int, rank: int, S=None, ws=None, stream=None) -> torch.Tensor:
    """Pairwise linear CKA [E, E] (fp32) of the expert adapters A, B (packed,
    E keys of rank `rank`) on the probe rows X [N, d_in]."""
    N, d_in = X.shape
    d_out = B.numel() // (E * rank)
    if S is None:
        S = torch.empty(E, E, dtype=torch.float32, device=A.device)
    if ws is None:
        need = ace_workspace_bytes(ACE_OP_CKA, N, 1, d_in, d_out, E, rank)
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=A.device)
    _check(_lib.ace_pairwise_cka(_dtype(A), N, d_in, d_out, E, rank, _ptr(X), _ptr(A), _ptr(B),
                                 _ptr(S), _ptr(ws), ws.numel(), _stream(stream)),
           "ace_pairwise_cka")
    return S


def _host(a, dtype):
    import numpy as np
    return np.ascontiguousarray(a, dtype=dtype)


def ace_similarity_graph(S):
    """W [E, E] (float64, numpy) from the similarity matrix S [E, E] (host)."""
    import numpy as np
    S = _host(S, np.float32)
    E = S.shape[0]
    W = np.empty((E, E), dtype=np.float64)
    _check(_lib.ace_similarity_graph(S.ctypes.data, E, W.ctypes.data), "ace_similarity_graph")
    return W


def ace_louvain(W, gamma: float = 0.8):
    """(groups int32 [E], G) from the graph W [E, E] (host, float64)."""
    import numpy as np
    W = _host(W, np.float64)
    E = W.shape[0]
    groups = np.empty(E, dtype=np.int32)
    G = ctypes.c_int32(0)
    _check(_lib.ace_louvain(W.ctypes.data, E, float(gamma), groups.ctypes.data, ctypes.byref(G)),
           "ace_louvain")
    return groups, int(G.value)


def ace_group_anchors(S, expert_to_group, G: int):
    """CKA centre of every group (int32 [G])."""
    import numpy as np
    S = _host(S, np.float32)
    e2g = _host(expert_to_group, np.int32)
    anchors = np.empty(G, dtype=np.int32)
    _check(_lib.ace_group_anchors(S.ctypes.data, S.shape[0], e2g.ctypes.data, G,
                                  anchors.ctypes.data), "ace_group_anchors")
    return anchors


def ace_consolidate_adapters(A, B, E: int, rank: int, expert_to_group, G: int, anchors, A_init,
                             A_g=None, B_g=None, stream=None):
    """Group adapters (A_g, B_g, group ranks) from the expert adapters A, B
    (device); the library returns the group ranks.  A_g, B_g hold E * rank
    ranks in total (the unchanged budget)."""
    import numpy as np
    e2g = _host(expert_to_group, np.int32)
    anc = _host(anchors, np.int32)
    d_in = A.shape[1]
    d_out = B.numel() // (E * rank)
    if A_g is None:
        A_g = torch.empty(E * rank, d_in, dtype=A.dtype, device=A.device)
    if B_g is None:
        B_g = torch.empty(E * rank * d_out, dtype=B.dtype, device=B.device)
    for t, n in ((A_g, E * rank * d_in), (B_g, E * rank * d_out)):
        if t.numel() != n or t.dtype != A.dtype or t.device != A.device:
            raise ValueError("A_g / B_g must hold E * rank ranks in A's dtype and device")
    ranks = np.zeros(G, dtype=np.int32)
    _check(_lib.ace_consolidate_adapters(_dtype(A), d_in, d_out, E, rank, _ptr(A), _ptr(B),
                                         e2g.ctypes.data, G, anc.ctypes.data, _ptr(A_init),
                                         _ptr(A_g), _ptr(B_g), ranks.ctypes.data,
                                         _stream(stream)),
           "ace_consolidate_adapters")
    return A_g, B_g, [int(r) for r in ranks]


def raw_lib() -> ctypes.CDLL:
    """The loaded library (tests check exports and host-side validation)."""
    return _lib


def ace_moe_lora_fwd(x, W, expert_routing: Routing, y, key_rank: Optional[Sequence[int]] = None,
                     expert_key: Optional[Sequence[int]] = None, alpha: float = 16.0, A=None,
                     B=None, adapter_routing: Optional[Routing] = None,
                     input_mode: int = ACE_INPUT_SHARED, ws=None, stream=None) -> None:
    """y[t*k + j] = W_e xin(t, j) + s_q B_q (A_q xin(t, j)) (include/ace.h).
    key_rank None runs the plain expert projection."""
    T, k = expert_routing.c.T, expert_routing.c.k
    E, d_out, d_in = W.shape
    n_keys = 0 if key_rank is None else len(key_rank)
    ranks = _ranks_arg(key_rank) if n_keys else None
    ekey = (ctypes.c_int32 * E)(*[int(v) for v in expert_key]) if n_keys else None
    if n_keys:
        ws = _fwd_ws(ws, T, k, d_in, d_out, n_keys, max(key_rank), x.device)
    _check(_lib.ace_moe_lora_fwd(_dtype(x), input_mode, T, k, d_in, d_out, E, _ptr(x), _ptr(W),
                                 ctypes.byref(expert_routing.c), n_keys, ranks, ekey, alpha,
                                 _ptr(A), _ptr(B),
                                 ctypes.byref(adapter_routing.c) if adapter_routing else None,
                                 _ptr(y), _ptr(ws), 0 if ws is None else ws.numel(),
                                 _stream(stream)),
           "ace_moe_lora_fwd")
