"""Seeded synthetic MoE workloads for grouped adapter execution.

This module only draws inputs: routing (top-k expert ids and router weights),
expert-to-group maps, per-group ranks and the dense tensors (x, A, B, dY).  It
holds none of the method's arithmetic, so both the fp64 oracle side of the
tests and the GPU side (tests, bench) can take their inputs from it.

Shapes follow the MoE backbones of the paper's model-configuration table
(OLMoE-1B-7B, Qwen1.5-MoE-A2.7B, Moonlight/DeepSeek-style 64 routed experts)
plus a Mixtral-like 8-expert layer; the paper's training data is replaced by
synthetic routing whose skew is set by a Zipf popularity law.

Recipe (every stream is an independent child of ``SeedSequence(seed)``):
  * routing   -- logits ~ N(0, sigma) ("normal") or log((i+1)^-s) + Gumbel(0,1)
                 ("zipf"; Gumbel-top-k draws k experts without replacement in
                 proportion to popularity).  top-k by descending logit, ties to
                 the lower expert id; weights = softmax over all E logits,
                 gathered at the top-k, not renormalised.
  * groups    -- "consecutive" (g = e // m), "random_equal" (a seeded
                 permutation cut into groups of m), "uneven" (sizes drawn from
                 {2,4,8}, capped by what is left, until they cover E).
  * ranks     -- r_g = |G_g| * r_e, so sum_g r_g = E * r_e (fixed budget,
                 Sec. 3.3 rank consolidation).
  * tensors   -- x ~ N(0,1), A ~ N(0, 1/d_in) (std d_in^-1/2), B ~ N(0, 0.02)
                 (std 0.02), dY ~ N(0,1); bf16 configs round with RNE.
  * frozen expert weights of a projection (the base GEMM that the adapter
    update can be fused into) -- W_e ~ N(0, 1/d_in), one [d_out, d_in] matrix
    per expert, stream "<proj>.W".
  * probe and expert adapters for the consolidation step (Sec. 3.3: N probe
    hidden states go through every expert adapter of a layer; the paper uses
    N = 10,000 training tokens after a warm-up of expert-wise LoRA) --
    probe rows ~ N(mu, 1) with a per-feature offset mu ~ N(0, 1); the experts
    fall into planted clusters (the config's group scheme), and expert e's
    adapter is its cluster's base plus independent noise:
    A_e = A_c + nu * N(0, 1/d_in), B_e = B_c + nu * N(0, 0.02^2), with
    A_c ~ N(0, 1/d_in), B_c ~ N(0, 0.02^2); nu = 0.5 by default.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# Row modes and input modes, mirroring include/ace.h.
ROWS_GROUP_DEDUP = 0
ROWS_GROUP_PAIRS = 1
ROWS_EXPERT = 2
INPUT_SHARED = 0
INPUT_PER_PAIR = 1
INPUT_COMBINED = 2

_STREAMS = ("router", "groups", "x", "h", "gate.A", "gate.B", "gate.dy",
            "up.A", "up.B", "up.dy", "down.A", "down.B", "down.dy", "y_in",
            "dx_in", "extra", "gate.dy_combined", "up.dy_combined", "down.dy_combined",
            "probe", "probe.mu", "cka.clusters", "cka.A", "cka.B", "cka.A_noise", "cka.B_noise",
            "cka.A_init", "gate.W", "up.W", "down.W")


@dataclasses.dataclass(frozen=True)
class MoEConfig:
    name: str
    dtype: str                 # "f32" or "bf16"
    T: int                     # tokens
    d_model: int
    d_ffn: int
    E: int                     # routed experts
    k: int                     # top-k
    routing: Tuple[str, float]  # ("normal", sigma) or ("zipf", s)
    groups: Tuple[str, int]    # ("consecutive", m) | ("random_equal", m) | ("uneven", 0)
    r_e: int                   # expert-wise rank
    projections: Tuple[str, ...]
    alpha: float = 16.0

    @property
    def P(self) -> int:
        return self.T * self.k

    def proj_dims(self, proj: str) -> Tuple[int, int, int]:
        """(d_in, d_out, input_mode) of a projection of the gated FFN."""
        if proj in ("gate", "up"):
            return self.d_model, self.d_ffn, INPUT_SHARED
        if proj == "down":
            return self.d_ffn, self.d_model, INPUT_PER_PAIR
        raise ValueError(proj)

    def scaled(self, **kw) -> "MoEConfig":
        return dataclasses.replace(self, **kw)


CONFIGS: Dict[str, MoEConfig] = {
    c.name: c for c in [
        MoEConfig("tiny_fp32", "f32", 256, 512, 1024, 8, 2, ("normal", 1.0),
                  ("consecutive", 2), 8, ("up",)),
        MoEConfig("olmoe_bf16", "bf16", 4096, 2048, 1024, 64, 8, ("zipf", 0.8),
                  ("random_equal", 4), 8, ("gate", "up", "down")),
        MoEConfig("qwen_bf16", "bf16", 8192, 2048, 1408, 60, 4, ("zipf", 0.8),
                  ("random_equal", 4), 16, ("gate", "up", "down")),
        MoEConfig("deepseek_bf16", "bf16", 8192, 2048, 1408, 64, 6, ("zipf", 1.0),
                  ("uneven", 0), 8, ("gate", "up", "down")),
        MoEConfig("mixtral_bf16", "bf16", 16384, 4096, 14336, 8, 2, ("normal", 0.5),
                  ("random_equal", 4), 16, ("gate", "up", "down")),
    ]
}
CONFIG_ORDER = ["tiny_fp32", "olmoe_bf16", "qwen_bf16", "deepseek_bf16", "mixtral_bf16"]


def seed_for(seed: int, stream: str) -> np.random.SeedSequence:
    return np.random.SeedSequence(entropy=seed, spawn_key=(_STREAMS.index(stream),))


def rng_for(seed: int, stream: str) -> np.random.Generator:
    return np.random.default_rng(seed_for(seed, stream))


def torch_seed_for(seed: int, stream: str) -> int:
    return int(seed_for(seed, stream).generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1))


@dataclasses.dataclass
class Routing:
    topk_ids: np.ndarray        # int32 [T, k]
    topk_w: np.ndarray          # float32 [T, k]
    expert_to_group: np.ndarray  # int32 [E]
    group_rank: np.ndarray      # int32 [G]
    expert_rank: int

    @property
    def G(self) -> int:
        return int(self.group_rank.shape[0])


def draw_topk(logits: np.ndarray, k: int) -> Tuple[np.ndarray, np.ndarray]:
    """Top-k by descending logit (ties to the lower id) and softmax weights."""
    order = np.argsort(-logits, axis=1, kind="stable")[:, :k]
    z = logits - logits.max(axis=1, keepdims=True)
    p = np.exp(z)
    p /= p.sum(axis=1, keepdims=True)
    w = np.take_along_axis(p, order, axis=1)
    return order.astype(np.int32), w.astype(np.float32)


def draw_logits(T: int, E: int, routing: Tuple[str, float], rng: np.random.Generator) -> np.ndarray:
    kind, par = routing
    if kind == "normal":
        return rng.normal(0.0, par, size=(T, E))
    if kind == "zipf":
        pop = -par * np.log(np.arange(1, E + 1, dtype=np.float64))
        return pop[None, :] + rng.gumbel(0.0, 1.0, size=(T, E))
    raise ValueError(kind)


def draw_groups(E: int, groups: Tuple[str, int], rng: np.random.Generator) -> np.ndarray:
    kind, m = groups
    e2g = np.empty(E, dtype=np.int32)
    if kind == "consecutive":
        e2g[:] = np.arange(E) // m
        return e2g
    if kind == "identity":
        e2g[:] = np.arange(E)
        return e2g
    perm = rng.permutation(E)
    if kind == "random_equal":
        if E % m:
            raise ValueError("E must be a multiple of the group size")
        e2g[perm] = np.arange(E) // m
        return e2g
    if kind == "uneven":
        sizes: List[int] = []
        left = E
        while left > 0:
            choices = [s for s in (2, 4, 8) if s <= left] or [left]
            s = int(rng.choice(choices))
            sizes.append(s)
            left -= s
        start = 0
        for g, s in enumerate(sizes):
            e2g[perm[start:start + s]] = g
            start += s
        return e2g
    raise ValueError(kind)


def make_routing(cfg: MoEConfig, seed: int = 0) -> Routing:
    logits = draw_logits(cfg.T, cfg.E, cfg.routing, rng_for(seed, "router"))
    ids, w = draw_topk(logits, cfg.k)
    e2g = draw_groups(cfg.E, cfg.groups, rng_for(seed, "groups"))
    G = int(e2g.max()) + 1
    sizes = np.bincount(e2g, minlength=G)
    return Routing(ids, w, e2g, (sizes * cfg.r_e).astype(np.int32), cfg.r_e)


# ---------------------------------------------------------------------------
# dense tensors (torch, so that large configs can be drawn straight on a device)
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def round_bf16_np(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32."""
    b = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = ((b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000))
    return r.view(np.float32)


def draw_tensor(shape: Sequence[int], std: float, seed: int, stream: str, dtype: str,
                device: str = "cpu", sub: int = 0):
    """N(0, std^2) tensor in the storage dtype ("f32"/"bf16"); torch tensor."""
    torch = _torch()
    g = torch.Generator(device=device)
    g.manual_seed(torch_seed_for(seed, stream) + 7919 * sub)
    t = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    if dtype == "bf16":
        return t.to(torch.bfloat16)
    if dtype == "f32":
        return t
    raise ValueError(dtype)


@dataclasses.dataclass
class ProjTensors:
    proj: str
    d_in: int
    d_out: int
    input_mode: int
    x: object    # torch [T, d_in] (shared) or [P, d_in] (per pair)
    A: object    # torch [R, d_in]
    B: object    # torch flat [d_out * R]: per-key blocks [d_out, r_key] back to back
    dy: object   # torch [P, d_out]


def make_proj(cfg: MoEConfig, proj: str, ranks: Sequence[int], seed: int = 0,
              device: str = "cpu") -> ProjTensors:
    """Tensors of one adapted projection for the given per-key ranks."""
    d_in, d_out, im = cfg.proj_dims(proj)
    R = int(sum(int(r) for r in ranks))
    rows = cfg.T if im == INPUT_SHARED else cfg.P
    xs = "x" if im == INPUT_SHARED else "h"
    x = draw_tensor((rows, d_in), 1.0, seed, xs, cfg.dtype, device)
    A = draw_tensor((R, d_in), 1.0 / math.sqrt(d_in), seed, proj + ".A", cfg.dtype, device)
    B = draw_tensor((d_out * R,), 0.02, seed, proj + ".B", cfg.dtype, device)
    dy = draw_tensor((cfg.P, d_out), 1.0, seed, proj + ".dy", cfg.dtype, device)
    return ProjTensors(proj, d_in, d_out, im, x, A, B, dy)


def budget(ranks: Sequence[int], d_in: int, d_out: int) -> int:
    """Trainable adapter parameters for the given ranks (Sec. 3.1.1 / 3.3)."""
    return int(sum(int(r) for r in ranks)) * (d_in + d_out)


def describe(cfg: MoEConfig, rt: Routing) -> Dict[str, object]:
    """Routing statistics used to report how skewed a draw is."""
    load = np.bincount(rt.topk_ids.ravel(), minlength=cfg.E).astype(np.float64)
    p = load / load.sum()
    nz = p[p > 0]
    ent = float(-(nz * np.log(nz)).sum() / math.log(cfg.E))
    return {"P": cfg.P, "E": cfg.E, "G": rt.G, "load_entropy": ent,
            "max_over_mean_load": float(load.max() / load.mean())}


@dataclasses.dataclass
class ProbeAdapters:
    X: object          # torch [N, d_in]
    A: object          # torch [E*r, d_in]
    B: object          # torch flat: expert e's [d_out, r] block at d_out * r * e
    clusters: np.ndarray  # int32 [E]: planted cluster of every expert
    d_in: int
    d_out: int
    E: int
    r: int


def make_probe_adapters(cfg: MoEConfig, proj: str = "gate", N: int = 10000, noise: float = 0.5,
                        seed: int = 0, device: str = "cpu") -> ProbeAdapters:
    """Probe set and expert-wise adapters of one projection for the CKA step
    (recipe in the module notes)."""
    torch = _torch()
    d_in, d_out, _ = cfg.proj_dims(proj)
    E, r = cfg.E, cfg.r_e
    clusters = draw_groups(E, cfg.groups, rng_for(seed, "cka.clusters"))
    C = int(clusters.max()) + 1
    idx = torch.from_numpy(clusters.astype(np.int64)).to(device)
    X = draw_tensor((N, d_in), 1.0, seed, "probe", "f32", device)
    X += draw_tensor((d_in,), 1.0, seed, "probe.mu", "f32", device)
    Ac = draw_tensor((C, r, d_in), 1.0 / math.sqrt(d_in), seed, "cka.A", "f32", device)
    An = draw_tensor((E, r, d_in), noise / math.sqrt(d_in), seed, "cka.A_noise", "f32", device)
    Bc = draw_tensor((C, d_out, r), 0.02, seed, "cka.B", "f32", device)
    Bn = draw_tensor((E, d_out, r), 0.02 * noise, seed, "cka.B_noise", "f32", device)
    A = (Ac[idx] + An).reshape(E * r, d_in)
    B = (Bc[idx] + Bn).reshape(-1)
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    return ProbeAdapters(X.to(dt).contiguous(), A.to(dt).contiguous(), B.to(dt).contiguous(),
                         clusters, d_in, d_out, E, r)


def draw_lora_init_A(rows: int, d_in: int, seed: int = 0, dtype: str = "bf16", device: str = "cpu"):
    """Standard LoRA initialisation of A rows (Kaiming-uniform with a = sqrt(5),
    i.e. U(-1/sqrt(d_in), 1/sqrt(d_in))): the draw that fills the extra rank
    rows of a consolidated group adapter.  torch [rows, d_in]."""
    torch = _torch()
    g = torch.Generator(device=device)
    g.manual_seed(torch_seed_for(seed, "cka.A_init"))
    t = (torch.rand(rows, d_in, generator=g, device=device, dtype=torch.float32) * 2 - 1)
    t.mul_(1.0 / math.sqrt(d_in))
    return t.to(torch.bfloat16 if dtype == "bf16" else torch.float32)



def draw_expert_weights(cfg: MoEConfig, proj: str, seed: int = 0, device: str = "cpu"):
    """Frozen expert weights of one projection: torch [E, d_out, d_in],
    N(0, 1/d_in), in the config's storage dtype."""
    d_in, d_out, _ = cfg.proj_dims(proj)
    return draw_tensor((cfg.E, d_out, d_in), 1.0 / math.sqrt(d_in), seed, proj + ".W", cfg.dtype,
                       device)
