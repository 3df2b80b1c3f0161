"""Seeded synthetic inputs for the CAP expert-parallel MoE layer.

This module is shared by the CPU oracle (tests) and the GPU path (tests, bench).
It holds none of the method's arithmetic: no top-k, gating, pruning, layout,
FFN, combine, co-activation or placement logic lives here.  It only draws
random inputs with the shapes and structure of the paper's workloads:

* Router logits follow a latent-topic model.  The paper observes structured
  expert co-activation (Sec. IV-A, Fig. "Expert co-activation matrix") and that
  hot experts get higher routing scores (Sec. VII, Fig. "Hot experts tend to get
  higher routing scores").  Each token draws a topic u uniformly; experts are
  cut into equal clusters (a seeded permutation, deliberately non-contiguous in
  expert id so sequential placement is not already co-activation optimal); the
  logit is ``2.0*[cluster(e)==u] + b_e + N(0,1)`` with ``b_e = -s*ln(rank_e)``
  the log of a Zipf(s) popularity over a second seeded permutation.
* Activations x ~ N(0,1) (bf16 configs) or N(0, 0.02^2) (the tiny fp32 config).
* Expert weights: W1, W3 ~ N(0, 1/d); W2 ~ N(0, 1/(144*inter)), which keeps the
  layer output at rms ~0.05 so the relative tolerance is meaningful.  The tiny
  fp32 config uses N(0, 0.02^2) for every weight.
* Random draws the method itself needs (the zero-score pick of the co-activation
  grouping algorithm) are drawn here and passed in as an input permutation.

Every stream comes from ``numpy.random.SeedSequence(seed).spawn`` so each part
(logits, activations, each expert's weights, ...) can be regenerated alone.
bf16 tensors are returned as ``uint16`` bit patterns (round to nearest even).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

# Stream indices into SeedSequence(seed).spawn(N_STREAMS).
_S_CLUSTER, _S_POP, _S_TOPIC, _S_NOISE, _S_ACT, _S_WEIGHT, _S_RAND, _S_TRACE, _S_AUX = range(9)
N_STREAMS = 9


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    T: int              # total tokens over all virtual ranks
    d: int              # hidden size
    E: int              # routed experts
    k: int              # top-k
    inter: int          # SwiGLU intermediate size of a routed expert
    R: int              # virtual ranks (GPUs)
    ranks_per_node: int
    n_clusters: int     # latent topics / expert clusters
    zipf_s: float       # Zipf exponent of expert popularity
    dtype: str          # "f32" or "bf16": activations and weights
    n_shared: int = 0   # always-active shared experts
    shared_inter: int = 0
    act_std: float = 1.0
    w_std: float | None = None  # fixed std for every weight (tiny config); None -> scaled init
    trace_tokens: int = 8192    # tokens in the routing trace that feeds placement

    @property
    def tokens_per_rank(self) -> int:
        return self.T // self.R

    @property
    def E_loc(self) -> int:
        return self.E // self.R

    @property
    def nodes(self) -> int:
        return self.R // self.ranks_per_node

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


# The five workload shapes.  Shapes follow Qwen3-30B-A3B, DeepSeek-V2-Lite and
# DeepSeek-V3 MoE layers; the paper evaluates the first two (Sec. VIII-A).
CONFIGS: dict[str, Config] = {
    # Tiny fp32 layer: 4 ranks x 4 experts, top-2, N(0,0.02) weights and activations.
    "c1": Config("c1", T=256, d=128, E=16, k=2, inter=256, R=4, ranks_per_node=4,
                 n_clusters=4, zipf_s=1.1, dtype="f32", act_std=0.02, w_std=0.02,
                 trace_tokens=256),
    # Same tiny shape with unit-scale activations and scaled weights, so that
    # the absolute tolerance term does not dominate.
    "c1u": Config("c1u", T=256, d=128, E=16, k=2, inter=256, R=4, ranks_per_node=4,
                  n_clusters=4, zipf_s=1.1, dtype="f32", act_std=1.0, w_std=None,
                  trace_tokens=256),
    # Qwen3-30B-A3B shape, 8 ranks x 16 experts, 4096 tokens per rank.
    "c2": Config("c2", T=32768, d=2048, E=128, k=8, inter=768, R=8, ranks_per_node=8,
                 n_clusters=8, zipf_s=1.1, dtype="bf16"),
    # Same layer on 2 nodes x 8 ranks x 8 experts.
    "c3": Config("c3", T=16384, d=2048, E=128, k=8, inter=768, R=16, ranks_per_node=8,
                 n_clusters=8, zipf_s=1.1, dtype="bf16"),
    # DeepSeek-V2-Lite shape: 64 routed + 2 shared experts (1408 each), top-6.
    "c4": Config("c4", T=8192, d=2048, E=64, k=6, inter=1408, R=8, ranks_per_node=8,
                 n_clusters=8, zipf_s=1.2, dtype="bf16", n_shared=2, shared_inter=1408),
    # DeepSeek-V3 shape: 256 routed + 1 shared expert, top-8, 4 nodes x 8 ranks.
    "c5": Config("c5", T=32768, d=7168, E=256, k=8, inter=2048, R=32, ranks_per_node=8,
                 n_clusters=32, zipf_s=1.1, dtype="bf16", n_shared=1, shared_inter=2048),
}


def _streams(seed: int):
    return np.random.SeedSequence(seed).spawn(N_STREAMS)


def _rng(ss) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(ss))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounded = (u + (((u >> 16) & 1) + 0x7FFF).astype(np.uint32)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------- router logits
def expert_clusters(cfg: Config, seed: int = 0) -> np.ndarray:
    """cluster[e]: a seeded permutation of expert ids cut into equal chunks."""
    perm = _rng(_streams(seed)[_S_CLUSTER]).permutation(cfg.E)
    size = cfg.E // cfg.n_clusters
    cluster = np.empty(cfg.E, dtype=np.int64)
    cluster[perm] = np.arange(cfg.E) // size
    return cluster


def expert_bias(cfg: Config, seed: int = 0) -> np.ndarray:
    """b_e = -s * ln(rank_e): log Zipf(s) popularity (normaliser dropped, shift-invariant)."""
    rank = _rng(_streams(seed)[_S_POP]).permutation(cfg.E) + 1
    return -cfg.zipf_s * np.log(rank.astype(np.float64))


def _latent_topic_logits(cfg: Config, seed: int, n_tokens: int, topic_ss, noise_ss) -> np.ndarray:
    cluster = expert_clusters(cfg, seed)
    bias = expert_bias(cfg, seed)
    topic = _rng(topic_ss).integers(0, cfg.n_clusters, size=n_tokens)
    noise = _rng(noise_ss).standard_normal((n_tokens, cfg.E))
    logits = 2.0 * (cluster[None, :] == topic[:, None]) + bias[None, :] + noise
    return np.ascontiguousarray(logits.astype(np.float32))


def logits(cfg: Config, seed: int = 0) -> np.ndarray:
    """fp32 router logits [T][E] of the evaluated batch."""
    s = _streams(seed)
    return _latent_topic_logits(cfg, seed, cfg.T, s[_S_TOPIC], s[_S_NOISE])


def trace_logits(cfg: Config, seed: int = 0) -> np.ndarray:
    """fp32 logits [trace_tokens][E] of an independent batch from the same model.

    This is the routing trace that feeds co-activation placement (the paper
    collects about 8,000 tokens offline before placing experts, Sec. VIII-G)."""
    a, b = _streams(seed)[_S_TRACE].spawn(2)
    return _latent_topic_logits(cfg, seed, cfg.trace_tokens, a, b)


def iid_logits(T: int, E: int, seed: int = 0) -> np.ndarray:
    """i.i.d. N(0,1) fp32 logits (uniform routing)."""
    return np.ascontiguousarray(
        _rng(_streams(seed)[_S_AUX]).standard_normal((T, E)).astype(np.float32))


# ---------------------------------------------------------------- activations
def activations_f32(cfg: Config, seed: int = 0, rows: slice | None = None) -> np.ndarray:
    """x [T][d] as fp32 values (already bf16-representable for bf16 configs)."""
    x = _rng(_streams(seed)[_S_ACT]).standard_normal((cfg.T, cfg.d), dtype=np.float32)
    x *= np.float32(cfg.act_std)
    if rows is not None:
        x = x[rows]
    if cfg.dtype == "bf16":
        return bf16_bits_to_f32(f32_to_bf16_bits(x))
    return np.ascontiguousarray(x)


def activations(cfg: Config, seed: int = 0) -> np.ndarray:
    """x [T][d] in the config's storage type: fp32 array or uint16 bf16 bits."""
    x = _rng(_streams(seed)[_S_ACT]).standard_normal((cfg.T, cfg.d), dtype=np.float32)
    x *= np.float32(cfg.act_std)
    return f32_to_bf16_bits(x) if cfg.dtype == "bf16" else np.ascontiguousarray(x)


# ---------------------------------------------------------------- expert weights
def _expert_weight_f32(cfg: Config, seed: int, slot: int, inter: int):
    ss = _streams(seed)[_S_WEIGHT].spawn(cfg.E + 1)[slot]
    g = _rng(ss)
    if cfg.w_std is not None:
        s1 = s3 = s2 = np.float32(cfg.w_std)
    else:
        s1 = s3 = np.float32(1.0 / math.sqrt(cfg.d))
        s2 = np.float32(1.0 / (12.0 * math.sqrt(inter)))
    w1 = g.standard_normal((inter, cfg.d), dtype=np.float32) * s1
    w3 = g.standard_normal((inter, cfg.d), dtype=np.float32) * s3
    w2 = g.standard_normal((cfg.d, inter), dtype=np.float32) * s2
    return w1, w3, w2


def _store(cfg: Config, a: np.ndarray) -> np.ndarray:
    return f32_to_bf16_bits(a) if cfg.dtype == "bf16" else np.ascontiguousarray(a)


def expert_weights(cfg: Config, e: int, seed: int = 0):
    """(W1 [inter][d], W3 [inter][d], W2 [d][inter]) of routed expert e, storage type."""
    return tuple(_store(cfg, w) for w in _expert_weight_f32(cfg, seed, e, cfg.inter))


def expert_weights_f32(cfg: Config, e: int, seed: int = 0):
    """Same weights as exact fp32 values (bf16 values widened for bf16 configs)."""
    ws = _expert_weight_f32(cfg, seed, e, cfg.inter)
    if cfg.dtype == "bf16":
        return tuple(bf16_bits_to_f32(f32_to_bf16_bits(w)) for w in ws)
    return ws


def shared_weights(cfg: Config, seed: int = 0):
    """The shared experts as one SwiGLU FFN with inter = n_shared*shared_inter.

    A sum of SwiGLU FFNs equals one SwiGLU FFN over the concatenated
    intermediate dimension (stack W1 and W3 rows, concatenate W2 columns)."""
    if cfg.n_shared == 0:
        return None
    inter = cfg.n_shared * cfg.shared_inter
    return tuple(_store(cfg, w) for w in _expert_weight_f32(cfg, seed, cfg.E, inter))


def shared_weights_f32(cfg: Config, seed: int = 0):
    if cfg.n_shared == 0:
        return None
    inter = cfg.n_shared * cfg.shared_inter
    ws = _expert_weight_f32(cfg, seed, cfg.E, inter)
    if cfg.dtype == "bf16":
        return tuple(bf16_bits_to_f32(f32_to_bf16_bits(w)) for w in ws)
    return ws


# ---------------------------------------------------------------- placements / random inputs
def sequential_placement(cfg: Config):
    """Default placement: experts assigned to ranks in expert-id order."""
    e = np.arange(cfg.E, dtype=np.int32)
    return (e // cfg.E_loc).astype(np.int32), (e % cfg.E_loc).astype(np.int32)


def random_order(n: int, seed: int = 0, salt: int = 0) -> np.ndarray:
    """A uniform random permutation of range(n): the random draws of the
    grouping algorithm's zero-score pick, passed to it as an input."""
    ss = _streams(seed)[_S_RAND].spawn(salt + 1)[salt]
    return _rng(ss).permutation(n).astype(np.int64)


def router_weights(cfg: Config, seed: int = 0) -> np.ndarray:
    """Router weights W_g [E][d] ~ N(0, 1/d) as bf16 bits, so x W_g^T has unit
    scale for unit-scale x (inputs of the fused router front end)."""
    return random_rows(cfg.E, cfg.d, "bf16", seed, salt=11, std=1.0 / np.sqrt(cfg.d))


def random_rows(n_rows: int, d: int, dtype: str, seed: int = 0, salt: int = 0, std: float = 0.05):
    """Seeded random rows (e.g. stand-in expert outputs for combine-only cases)."""
    ss = _streams(seed)[_S_AUX].spawn(salt + 2)[salt + 1]
    a = _rng(ss).standard_normal((n_rows, d), dtype=np.float32) * np.float32(std)
    return f32_to_bf16_bits(a) if dtype == "bf16" else np.ascontiguousarray(a)
