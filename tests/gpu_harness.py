"""Shared helpers of the GPU parity tests: run one projection through the HIP
library (C-ABI via the ctypes binding) and through the fp64 oracle on the
same seeded inputs."""
from __future__ import annotations

import dataclasses
import sys
from typing import Optional, Sequence

import numpy as np
import torch

from oracle import ace_oracle as O
from paper_2609_06072_amd import workloads as W

TOL = {"bf16": 2e-2, "f32": 1e-5}

PATHS = {
    # name: (row mode, input mode override (None = projection's), key kind)
    "grouped": (W.ROWS_GROUP_DEDUP, W.INPUT_SHARED, "group"),
    "expertwise": (W.ROWS_EXPERT, W.INPUT_SHARED, "expert"),
    "down_expertwise": (W.ROWS_EXPERT, W.INPUT_PER_PAIR, "expert"),
    "pairs_shared": (W.ROWS_GROUP_PAIRS, W.INPUT_SHARED, "group"),
    "pairs_per_pair": (W.ROWS_GROUP_PAIRS, W.INPUT_PER_PAIR, "group"),
    # down projection with the output combined per token (per-pair input)
    "combined": (W.ROWS_GROUP_DEDUP, W.INPUT_COMBINED, "group"),
    "combined_expertwise": (W.ROWS_EXPERT, W.INPUT_COMBINED, "expert"),
}
WEIGHTED = ("grouped", "pairs_per_pair", "combined", "combined_expertwise")


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


@dataclasses.dataclass
class Case:
    cfg: W.MoEConfig
    rt: W.Routing
    mode: int
    input_mode: int
    ranks: list
    e2g: Optional[np.ndarray]   # None for expert keys
    n_keys: int
    d_in: int
    d_out: int
    x: torch.Tensor
    A: torch.Tensor
    B: torch.Tensor
    dy: torch.Tensor
    pair_w: Optional[torch.Tensor]


def make_case(cfg: W.MoEConfig, path: str, seed: int = 0, with_w: bool = False,
              device: str = "cuda", proj: Optional[str] = None) -> Case:
    mode, im, kind = PATHS[path]
    rt = W.make_routing(cfg, seed)
    if proj is None:
        if im in (W.INPUT_PER_PAIR, W.INPUT_COMBINED):
            proj = "down"
        else:
            proj = "gate" if "gate" in cfg.projections else cfg.projections[0]
    if kind == "group":
        ranks = [int(r) for r in rt.group_rank]
        e2g = rt.expert_to_group
        n_keys = rt.G
    else:
        ranks = [cfg.r_e] * cfg.E
        e2g = None
        n_keys = cfg.E
    t = W.make_proj(cfg, proj, ranks, seed=seed, device=device)
    x, dy = t.x, t.dy
    x_mode = W.INPUT_PER_PAIR if im == W.INPUT_COMBINED else im
    if t.input_mode != x_mode:
        rows = cfg.T if im == W.INPUT_SHARED else cfg.P
        x = W.draw_tensor((rows, t.d_in), 1.0, seed, "x" if im == W.INPUT_SHARED else "h",
                          cfg.dtype, device)
    if im == W.INPUT_COMBINED:   # gradient of the combined output: one row per token
        dy = W.draw_tensor((cfg.T, t.d_out), 1.0, seed, proj + ".dy_combined", cfg.dtype, device)
    pair_w = torch.from_numpy(rt.topk_w).to(device) if with_w else None
    return Case(cfg, rt, mode, im, ranks, e2g, n_keys, t.d_in, t.d_out, x, t.A, t.B, dy, pair_w)


def run_gpu(c: Case, fwd: bool = True, bwd: bool = True, y_in=None, dx_in=None,
            reuse_h: bool = False):
    """Forward and/or backward through the library; with reuse_h the
    backward reads h from the forward's workspace (h_fwd)."""
    from paper_2609_06072_amd import ace
    dev = c.x.device
    ids = torch.from_numpy(c.rt.topk_ids).to(dev)
    e2g = torch.from_numpy(c.rt.expert_to_group).to(dev)
    routing = ace.ace_group_permute(ids, c.cfg.E, None if c.mode == W.ROWS_EXPERT else e2g,
                                    c.rt.G, c.mode)
    out = {"routing": routing}
    P = c.cfg.P
    fws = None
    if fwd:
        rows = c.cfg.T if c.input_mode == W.INPUT_COMBINED else P
        y = torch.zeros(rows, c.d_out, dtype=c.x.dtype, device=dev) if y_in is None else y_in.clone()
        need = ace.ace_workspace_bytes(ace.ACE_OP_FWD, c.cfg.T, c.cfg.k, c.d_in, c.d_out,
                                       c.n_keys, max(c.ranks))
        fws = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
        if c.mode == W.ROWS_EXPERT:
            ace.ace_expertwise_lora_fwd(c.x, c.A, c.B, c.cfg.E, c.cfg.r_e, c.cfg.alpha, routing, y,
                                        pair_w=c.pair_w, input_mode=c.input_mode, ws=fws)
        else:
            ace.ace_grouped_lora_fwd(c.x, c.A, c.B, c.ranks, c.cfg.alpha, routing, y,
                                     pair_w=c.pair_w, input_mode=c.input_mode, ws=fws)
        out["y"] = y
    h_fwd = fws if (reuse_h and fwd) else None
    if bwd:
        dx = torch.zeros_like(c.x) if dx_in is None else dx_in.clone()
        R = sum(c.ranks)
        dA = torch.full((R, c.d_in), float("nan"), dtype=torch.float32, device=dev)
        dB = torch.full((R * c.d_out,), float("nan"), dtype=torch.float32, device=dev)
        if c.mode == W.ROWS_EXPERT:
            ace.ace_expertwise_lora_bwd(c.x, c.A, c.B, c.cfg.E, c.cfg.r_e, c.cfg.alpha, routing,
                                        c.dy, dx, dA, dB, pair_w=c.pair_w, input_mode=c.input_mode,
                                        h_fwd=h_fwd)
        else:
            ace.ace_grouped_lora_bwd(c.x, c.A, c.B, c.ranks, c.cfg.alpha, routing, c.dy, dx, dA,
                                     dB, pair_w=c.pair_w, input_mode=c.input_mode, h_fwd=h_fwd)
        out.update(dx=dx, dA=dA, dB=dB)
    torch.cuda.synchronize()
    return out


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def oracle_args(c: Case, ids: Optional[np.ndarray] = None, x: Optional[np.ndarray] = None,
                w: Optional[np.ndarray] = None):
    ids = c.rt.topk_ids.astype(np.int64) if ids is None else ids
    x = f64(c.x) if x is None else x
    if w is None and c.pair_w is not None:
        w = c.rt.topk_w.astype(np.float64)
    return (x, f64(c.A), f64(c.B), c.ranks, c.cfg.alpha, ids, c.cfg.E, c.e2g, c.n_keys), w


def oracle_fwd(c: Case) -> np.ndarray:
    a, w = oracle_args(c)
    return O.lora_delta(*a, input_mode=c.input_mode, pair_w=w)


def oracle_bwd(c: Case):
    a, w = oracle_args(c)
    return O.lora_grads(*a, f64(c.dy), input_mode=c.input_mode, pair_w=w)


def check_rel(name: str, got, ref, tol: float) -> float:
    e = O.rel_l2(got, ref)
    assert np.all(np.isfinite(np.asarray(got))), f"{name}: non-finite values"
    assert e <= tol, f"{name}: rel L2 {e:.3e} > {tol:.1e}"
    return e


def check_rows(name: str, got, ref, tol: float, row_len: Optional[int] = None) -> float:
    """Per-row companion of check_rel: every row's rel-L2 must be within tol,
    and a row that is exactly zero in the reference (a dropped pair, a token
    no pair reads, an empty key) must be exactly zero.  A whole-tensor norm
    alone lets one wrong row in a few thousand pass; this catches an error
    confined to a few rows or one column chunk.  Returns the worst row's
    rel-L2."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, f"{name}: shape {got.shape} != {ref.shape}"
    if row_len is not None:
        got, ref = got.reshape(-1, row_len), ref.reshape(-1, row_len)
    elif got.ndim == 1:
        got, ref = got[None, :], ref[None, :]
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    rn = np.sqrt((ref * ref).sum(axis=1))
    en = np.sqrt(((got - ref) ** 2).sum(axis=1))
    zero = rn == 0.0
    bad_zero = np.nonzero(zero & (np.abs(got).max(axis=1, initial=0.0) != 0.0))[0]
    assert bad_zero.size == 0, f"{name}: rows {bad_zero[:8].tolist()} should be exactly zero"
    rel = np.where(zero, 0.0, en / np.where(zero, 1.0, rn))
    worst = int(np.argmax(rel)) if rel.size else 0
    e = float(rel[worst]) if rel.size else 0.0
    assert e <= tol, f"{name}: row {worst} rel L2 {e:.3e} > {tol:.1e}"
    return e


def check_dB_rows(name: str, got, ref, ranks: Sequence[int], d_out: int, tol: float) -> float:
    """check_rows on dB per rank index: key q's block is [d_out, r_q]
    row-major; each of its r_q columns (d_out values) is one row here."""
    got = np.asarray(got, dtype=np.float64).reshape(-1)
    ref = np.asarray(ref, dtype=np.float64).reshape(-1)
    g_cols, r_cols = [], []
    o = 0
    for r in ranks:
        n = d_out * int(r)
        g_cols.append(got[o:o + n].reshape(d_out, int(r)).T)
        r_cols.append(ref[o:o + n].reshape(d_out, int(r)).T)
        o += n
    return check_rows(name, np.concatenate(g_cols), np.concatenate(r_cols), tol)


def check_all(name: str, got, ref, tol: float, row_len: Optional[int] = None) -> float:
    """Whole-tensor rel-L2 (the contract) and the per-row check."""
    e = check_rel(name, got, ref, tol)
    check_rows(name, got, ref, tol, row_len)
    return e
