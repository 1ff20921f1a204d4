"""Seeded synthetic inputs for the MoE-layer hot path.

This module only draws inputs: source ids, router logits (with the popularity
and source-hotspot skews that the paper's routing observations motivate,
Sec. 2.2.2 and Figs. 3-4), the local-expert placement list, activations and
expert weights.  It holds none of the layer's arithmetic, so the HIP path and
the CPU oracle can both be fed from it without sharing any computation.

Every tensor comes from its own numpy ``PCG64`` stream, keyed by
``(seed, tensor tag, expert)`` through ``SeedSequence``, so any piece can be
drawn on its own (routing without weights, one expert without the others) and
the big weight sets are filled in parallel threads.  bf16 tensors are drawn in
fp32 as N(0, 0.02) and rounded to nearest-even bf16; they are returned as raw
``uint16`` bit patterns.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import os

import numpy as np

# Tags that separate the independent streams of one seed.
_TAG = {
    "src": 1, "logits": 2, "bias": 3, "local": 4, "x": 5,
    "w_gate": 6, "w_up": 7, "w_down": 8,
    "sh_gate": 9, "sh_up": 10, "sh_down": 11,
    "place_counts": 12, "place_bias": 13, "place_x0": 14, "place_m": 15,
    "gate_bias": 16,
}

WEIGHT_STD = 0.02


@dataclasses.dataclass(frozen=True)
class MoeConfig:
    """Shape and input recipe of one MoE layer workload."""
    name: str
    T: int            # tokens in the batch
    H: int            # hidden size
    E: int            # routed experts (gating width)
    k: int            # experts per token
    I: int            # routed expert intermediate size
    S: int            # source DP engines
    E_local: int      # experts hosted on this GPU
    n_shared: int = 0
    I_shared: int = 0
    bias: str = "none"        # none | zipf | source_hot | zipf_per_source
    zipf_s: float = 1.0
    hot_per_source: int = 0
    hot_bias: float = 0.0
    src_layout: str = "uniform"   # uniform | blocks | interleaved
    local_layout: str = "all"     # all (identity) | choice (random subset)
    # router gate function (moe_dims.flags: 0 softmax over the picks, 1 full
    # softmax, 2 sigmoid) and its parameters
    gate: int = 0
    gate_bias_std: float = 0.0    # selection-only bias N(0, std) per expert (sigmoid gates)
    routed_scale: float = 1.0
    n_group: int = 0
    topk_group: int = 0

    @property
    def dims(self) -> dict:
        return dict(T=self.T, H=self.H, E=self.E, k=self.k, I=self.I, S=self.S,
                    E_local=self.E_local, n_shared=self.n_shared,
                    I_shared=self.I_shared if self.n_shared else 0)

    @property
    def gated(self) -> bool:
        """Whether the router differs from the default (softmax over the picks)."""
        return bool(self.gate or self.gate_bias_std or self.routed_scale != 1.0 or self.n_group > 1)

    def replace(self, **kw) -> "MoeConfig":
        return dataclasses.replace(self, **kw)


# The five workloads: a tiny case, a Mixtral-shaped decode step, a
# DeepSeek-V2-Lite-shaped prefill, a Qwen3-30B-A3B-shaped prefill (the model of
# the paper's evaluation, Sec. 7.1) and one GPU's share of a DeepSeek-V3-shaped
# expert-parallel layer.
CONFIGS: dict[str, MoeConfig] = {
    "tiny": MoeConfig("tiny", T=256, H=128, E=8, k=2, I=256, S=4, E_local=8),
    "decode_mixtral": MoeConfig(
        "decode_mixtral", T=64, H=4096, E=8, k=2, I=14336, S=4, E_local=8,
        bias="zipf", zipf_s=1.0),
    "prefill_dsv2_lite": MoeConfig(
        "prefill_dsv2_lite", T=4096, H=2048, E=64, k=6, I=1408, S=4, E_local=64,
        n_shared=2, I_shared=1408, bias="zipf", zipf_s=1.0),
    "prefill_qwen3_30b_a3b": MoeConfig(
        "prefill_qwen3_30b_a3b", T=8192, H=2048, E=128, k=8, I=768, S=8,
        E_local=128, bias="source_hot", hot_per_source=8, hot_bias=2.0),
    "ep_share_dsv3": MoeConfig(
        "ep_share_dsv3", T=16384, H=7168, E=256, k=8, I=2048, S=8, E_local=32,
        n_shared=1, I_shared=2048, bias="zipf_per_source", zipf_s=1.2,
        src_layout="blocks", local_layout="choice"),
}
CONFIG_ORDER = list(CONFIGS)

# The DeepSeek-V3 share again with DeepSeek-V3's own router: sigmoid scores
# with a selection-only bias, 8 groups of 32 experts of which 4 stay, routed
# scale 2.5.  Not one of the five workloads above; a second routing family on
# the same kernels.
CONFIGS["ep_share_dsv3_v3router"] = CONFIGS["ep_share_dsv3"].replace(
    name="ep_share_dsv3_v3router", gate=2, gate_bias_std=0.02, routed_scale=2.5, n_group=8, topk_group=4)


def _rng(seed: int, tag: str, *extra: int) -> np.random.Generator:
    ss = np.random.SeedSequence([int(seed), _TAG[tag], *[int(e) for e in extra]])
    return np.random.Generator(np.random.PCG64(ss))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 to the nearest bf16 (ties to even); return the uint16 bits.

    Inputs here are finite draws, so NaN payload handling is not needed."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    t = u >> np.uint32(16)
    t &= np.uint32(1)
    t += np.uint32(0x7FFF)
    t += u
    t >>= np.uint32(16)
    return t.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen raw bf16 bits to fp32 exactly."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal_bf16(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    a = rng.standard_normal(int(np.prod(shape)), dtype=np.float32)
    a *= np.float32(std)
    return f32_to_bf16_bits(a).reshape(shape)


def make_src(cfg: MoeConfig, seed: int = 0) -> np.ndarray:
    """Source DP engine of each token, int32 in [0, S)."""
    if cfg.src_layout == "uniform":
        return _rng(seed, "src").integers(0, cfg.S, size=cfg.T, dtype=np.int32)
    if cfg.src_layout == "blocks":
        # Source-major contiguous blocks, as tokens sit in an EP receive buffer.
        return np.minimum(np.arange(cfg.T, dtype=np.int64) * cfg.S // max(cfg.T, 1),
                          cfg.S - 1).astype(np.int32)
    if cfg.src_layout == "interleaved":
        return (np.arange(cfg.T, dtype=np.int32) % cfg.S).astype(np.int32)
    raise ValueError(cfg.src_layout)


def _zipf_log_bias(rng: np.random.Generator, E: int, s: float) -> np.ndarray:
    # Popularity rank 1..E in a random order; exp(bias) is proportional to
    # rank**-s, so the softmax mass of expert e follows a Zipf(s) law.
    rank = 1.0 + rng.permutation(E).astype(np.float64)
    return (-s * np.log(rank)).astype(np.float32)


def make_logits(cfg: MoeConfig, src: np.ndarray, seed: int = 0) -> np.ndarray:
    """Router logits [T, E] fp32: N(0,1) plus the workload's skew."""
    logits = _rng(seed, "logits").standard_normal((cfg.T, cfg.E), dtype=np.float32)
    brng = _rng(seed, "bias")
    if cfg.bias == "none":
        pass
    elif cfg.bias == "zipf":
        logits += _zipf_log_bias(brng, cfg.E, cfg.zipf_s)[None, :]
    elif cfg.bias == "zipf_per_source":
        per_src = np.stack([_zipf_log_bias(brng, cfg.E, cfg.zipf_s) for _ in range(cfg.S)])
        logits += per_src[src]
    elif cfg.bias == "source_hot":
        perm = brng.permutation(cfg.E)
        hot = np.zeros((cfg.S, cfg.E), dtype=np.float32)
        h = cfg.hot_per_source
        for s in range(cfg.S):
            sel = perm[(s * h) % cfg.E: (s * h) % cfg.E + h]
            hot[s, sel] = np.float32(cfg.hot_bias)
        logits += hot[src]
    else:
        raise ValueError(cfg.bias)
    return np.ascontiguousarray(logits, dtype=np.float32)


def make_local_experts(cfg: MoeConfig, seed: int = 0) -> np.ndarray | None:
    """Experts hosted on this GPU, in slot order (None = all experts, identity)."""
    if cfg.local_layout == "all":
        assert cfg.E_local == cfg.E
        return None
    if cfg.local_layout == "choice":
        return _rng(seed, "local").choice(cfg.E, cfg.E_local, replace=False).astype(np.int32)
    raise ValueError(cfg.local_layout)


def make_x(cfg: MoeConfig, seed: int = 0) -> np.ndarray:
    """Token activations [T, H], bf16 bits."""
    return _normal_bf16(_rng(seed, "x"), (cfg.T, cfg.H), WEIGHT_STD)


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _expert_stack(seed: int, tag: str, n: int, shape, std: float) -> np.ndarray:
    out = np.empty((n, *shape), dtype=np.uint16)

    def fill(e: int) -> None:
        out[e] = _normal_bf16(_rng(seed, tag, e), shape, std)

    with _cf.ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(fill, range(n)))
    return out


def make_weights(cfg: MoeConfig, seed: int = 0, experts=None) -> dict:
    """Expert weights as bf16 bits, nn.Linear layout (out-features, in-features).

    Returns ``w_gate``/``w_up`` [E_local, I, H] and ``w_down`` [E_local, H, I]
    for the hosted slots, plus ``sh_gate``/``sh_up`` [n_sh, I_sh, H] and
    ``sh_down`` [n_sh, H, I_sh] when the layer has shared experts.  Routed
    weights are keyed by the global expert id hosted in each slot, so one
    expert's weights do not depend on where it is placed.  ``experts`` may
    override the hosted global ids."""
    if experts is None:
        loc = make_local_experts(cfg, seed)
        experts = np.arange(cfg.E, dtype=np.int32) if loc is None else loc
    experts = [int(e) for e in experts]
    n = len(experts)
    out = {}
    for tag, shape in (("w_gate", (cfg.I, cfg.H)), ("w_up", (cfg.I, cfg.H)),
                       ("w_down", (cfg.H, cfg.I))):
        arr = np.empty((n, *shape), dtype=np.uint16)

        def fill(i: int, tag=tag, shape=shape, arr=arr) -> None:
            arr[i] = _normal_bf16(_rng(seed, tag, experts[i]), shape, WEIGHT_STD)

        with _cf.ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(n)))
        out[tag] = arr
    if cfg.n_shared:
        out["sh_gate"] = _expert_stack(seed, "sh_gate", cfg.n_shared, (cfg.I_shared, cfg.H), WEIGHT_STD)
        out["sh_up"] = _expert_stack(seed, "sh_up", cfg.n_shared, (cfg.I_shared, cfg.H), WEIGHT_STD)
        out["sh_down"] = _expert_stack(seed, "sh_down", cfg.n_shared, (cfg.H, cfg.I_shared), WEIGHT_STD)
    return out


def make_gate_bias(cfg: MoeConfig, seed: int = 0) -> np.ndarray | None:
    """The router's selection-only bias [E] fp32 (None when the router has none)."""
    if not cfg.gate_bias_std:
        return None
    return (_rng(seed, "gate_bias").standard_normal(cfg.E) * cfg.gate_bias_std).astype(np.float32)


def make_routing(cfg: MoeConfig, seed: int = 0) -> dict:
    """The cheap part of a workload: src, logits, the router's bias and the
    local-expert list."""
    src = make_src(cfg, seed)
    return dict(src=src, logits=make_logits(cfg, src, seed), gate_bias=make_gate_bias(cfg, seed),
                local_experts=make_local_experts(cfg, seed))


def make_workload(cfg: MoeConfig, seed: int = 0, weights: bool = True) -> dict:
    """Everything one MoE layer call needs, as numpy arrays."""
    w = make_routing(cfg, seed)
    w["x"] = make_x(cfg, seed)
    if weights:
        w.update(make_weights(cfg, seed))
    return w


# ---------------------------------------------------------------------------
# Inputs of source-aware expert placement: the statistics of one profiling
# window (Sec. 5.1) for every MoE layer of a model, the source/rank cost
# matrix, the current placement and the capacities.


@dataclasses.dataclass(frozen=True)
class PlaceConfig:
    """Shape and input recipe of one placement problem."""
    name: str
    L: int                  # MoE layers placed together
    S: int                  # source DP engines
    E: int                  # experts per layer
    G: int                  # EP ranks
    k: int                  # experts per token
    tokens_per_source: int  # tokens each source routes through a layer per window
    zipf_s: float = 1.0     # per-source Zipf popularity (its own ranking per source and layer)
    hot_per_source: int = 0  # extra affinity of each source for its own expert set
    hot_bias: float = 0.0
    m_uniform: float = 64.0  # migration cost per changed indicator, in token units
    x0_layout: str = "contiguous"  # contiguous (rank g hosts experts [g E/G, (g+1) E/G)) | random

    @property
    def cap(self) -> np.ndarray:
        return np.full(self.G, -(-self.E // self.G), dtype=np.int32)


# A small case, the Qwen3-30B-A3B deployment of the paper's evaluation (48 MoE
# layers of 128 experts, DP8 attention feeding EP8, Sec. 7.1), a
# DeepSeek-V3-shaped model on EP8 (58 MoE layers of 256 experts) and the same
# model spread over 64 ranks with 64 sources (the largest D the kernel stages).
PLACE_CONFIGS: dict[str, PlaceConfig] = {
    "place_tiny": PlaceConfig("place_tiny", L=3, S=4, E=16, G=4, k=2, tokens_per_source=256,
                              hot_per_source=2, hot_bias=1.5, x0_layout="random"),
    "place_qwen3_30b_a3b": PlaceConfig("place_qwen3_30b_a3b", L=48, S=8, E=128, G=8, k=8,
                                       tokens_per_source=4096, zipf_s=1.0, hot_per_source=8,
                                       hot_bias=2.0),
    "place_dsv3_ep8": PlaceConfig("place_dsv3_ep8", L=58, S=8, E=256, G=8, k=8,
                                  tokens_per_source=4096, zipf_s=1.2),
    "place_dsv3_ep64": PlaceConfig("place_dsv3_ep64", L=58, S=64, E=256, G=64, k=8,
                                   tokens_per_source=512, zipf_s=1.2, x0_layout="random"),
}


def make_place_inputs(cfg: PlaceConfig, seed: int = 0) -> dict:
    """A [L,S,E] int64 window counts, D [S,G] fp64, x0 [L,E] int32, cap [G].

    Source s of layer l routes tokens_per_source * k pairs, multinomially over
    experts with probabilities proportional to exp(bias), where the bias is a
    per-source Zipf(zipf_s) log-popularity over its own random ranking plus
    hot_bias on hot_per_source experts of its own.  Source s sits with rank
    s * G // S: reaching that rank costs 0, any other 1.  M is uniform
    (m_uniform), so it is not drawn."""
    L, S, E, G = cfg.L, cfg.S, cfg.E, cfg.G
    brng = _rng(seed, "place_bias")
    crng = _rng(seed, "place_counts")
    A = np.empty((L, S, E), dtype=np.int64)
    for l in range(L):
        for s in range(S):
            bias = _zipf_log_bias(brng, E, cfg.zipf_s).astype(np.float64)
            if cfg.hot_per_source:
                bias[brng.choice(E, cfg.hot_per_source, replace=False)] += cfg.hot_bias
            p = np.exp(bias - bias.max())
            A[l, s] = crng.multinomial(cfg.tokens_per_source * cfg.k, p / p.sum())
    home = np.arange(S) * G // S
    D = np.ones((S, G), dtype=np.float64)
    D[np.arange(S), home] = 0.0
    if cfg.x0_layout == "contiguous":
        x0 = np.tile((np.arange(E) * G // E).astype(np.int32), (L, 1))
    elif cfg.x0_layout == "random":
        xr = _rng(seed, "place_x0")
        x0 = np.stack([np.repeat(np.arange(G, dtype=np.int32), -(-E // G))[:E][xr.permutation(E)]
                       for _ in range(L)])
    else:
        raise ValueError(cfg.x0_layout)
    return dict(A=A, D=D, x0=np.ascontiguousarray(x0, dtype=np.int32), cap=cfg.cap,
                m_uniform=cfg.m_uniform)


def make_migration_costs(L: int, E: int, G: int, seed: int = 0, scale: float = 64.0) -> np.ndarray:
    """A non-uniform M [L,E,G] fp64 in [0, scale), for tests of the M input."""
    return _rng(seed, "place_m").uniform(0.0, scale, size=(L, E, G))
