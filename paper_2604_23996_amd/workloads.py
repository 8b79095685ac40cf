"""Seeded synthetic inputs for the SMoES MoE layer.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic (no routing, no statistics, no MI). Both the HIP path and
the CPU oracle consume the arrays it returns, so it is the single source of
every input value. Arrays are NumPy; bf16 tensors are returned as their raw
uint16 bit patterns (round-to-nearest-even from float32).

Workload shapes follow the paper's MoE-VLM setting: LLaVA-style sequences in
which each image contributes a block of vision tokens followed by text tokens
(Supplementary A.1: 576 CLIP tokens per image), pushed through MoE layers shaped
like the backbones of the supplementary backbone table (DeepSeekMoE: 64 routed +
2 shared experts, top-6; Qwen3-MoE: 128 experts, top-8; hidden 2048), with
N_bins = 8 contiguous bins (Sec. 3.3, Sec. 3.5). The vision share of 65-86 %
matches the prefill token mixes of the supplementary transfer-ratio table.
The paper's datasets are not used; these draws stand in for them.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclass(frozen=True)
class LayerConfig:
    """Shape of one SMoES MoE layer workload."""

    name: str
    samples: Tuple[Tuple[int, int], ...]  # (vision tokens, text tokens) per sample
    d: int  # hidden size D
    E: int  # routed experts N_e
    k: int  # top-k
    inter: int  # expert FFN inner size
    n_shared: int  # always-on shared experts (merged inner size n_shared*inter)
    n_bins: int  # N_bins
    dtype: str  # activation / expert-weight storage type: "f32" or "bf16"
    seed: int
    vision_clusters: int = 1  # Gaussian components for the vision means
    interp_frac: float = 0.0  # share of tokens drawn as 50/50 vision-text blends
    logit_bias: bool = False  # per-expert N(0,1) bias added to the router logits
    update_stats: bool = False  # re-estimate the Gaussian statistics in the timed call
    tau_scale: float = 0.5  # tau = tau_scale * d (Sec. 3.5: tau = 0.5 D)
    beta: float = 0.99  # EMA decay (Sec. 3.5)

    @property
    def T(self) -> int:
        return sum(v + t for v, t in self.samples)

    @property
    def n_batch(self) -> int:
        return len(self.samples)

    @property
    def n_per_bin(self) -> int:
        return self.E // self.n_bins

    @property
    def shared_inter(self) -> int:
        return self.n_shared * self.inter

    @property
    def tau(self) -> float:
        return self.tau_scale * self.d


def _rep(n: int, v: int, t: int) -> Tuple[Tuple[int, int], ...]:
    return tuple((v, t) for _ in range(n))


# The five workloads: the small fp32 parity case, the DeepSeekMoE-like layer
# that throughput is quoted on, a fine-grained-expert layer, the
# DeepSeekMoE-like layer at training batch size, and a large skewed layer.
CONFIGS: List[LayerConfig] = [
    LayerConfig("tiny-fp32", _rep(1, 384, 128), d=256, E=8, k=2, inter=512,
                n_shared=0, n_bins=2, dtype=F32, seed=0),
    LayerConfig("deepseekmoe-vlm", _rep(4, 720, 304), d=2048, E=64, k=6,
                inter=1408, n_shared=2, n_bins=8, dtype=BF16, seed=1),
    LayerConfig("finegrained-vlm", _rep(8, 768, 256), d=2048, E=128, k=8,
                inter=768, n_shared=0, n_bins=16, dtype=BF16, seed=2,
                vision_clusters=4),
    LayerConfig("deepseekmoe-vlm-train", _rep(16, 717, 307), d=2048, E=64, k=6,
                inter=1408, n_shared=2, n_bins=8, dtype=BF16, seed=3,
                interp_frac=0.1, update_stats=True),
    LayerConfig("large-skewed-vlm", _rep(16, 768, 256), d=4096, E=160, k=6,
                inter=1536, n_shared=2, n_bins=8, dtype=BF16, seed=4,
                logit_bias=True),
]


# The benchmark's default: the largest layer that fits one GPU.
BENCH_WORKLOAD = "large-skewed-vlm"


def workload(name: str) -> LayerConfig:
    """The workload of that name (tiny-fp32, deepseekmoe-vlm, finegrained-vlm,
    deepseekmoe-vlm-train, large-skewed-vlm)."""
    for c in CONFIGS:
        if c.name == name:
            return c
    raise KeyError(f"unknown workload {name!r}; known: {[c.name for c in CONFIGS]}")


def small_config(d=64, E=8, k=2, inter=64, n_shared=1, n_bins=2, samples=((24, 8), (10, 22)),
                 dtype=F32, seed=123, **kw) -> LayerConfig:
    """A reduced layer for brute-force and multi-tile checks."""
    return LayerConfig("small", tuple(samples), d=d, E=E, k=k, inter=inter,
                       n_shared=n_shared, n_bins=n_bins, dtype=dtype, seed=seed, **kw)


# ----------------------------------------------------------------------------
# bf16 storage helpers (a storage format, not part of the method)
# ----------------------------------------------------------------------------

def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 with round-to-nearest-even; returns uint16 bits."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    # finite values never overflow 32 bits here; NaNs are fixed up below
    rounding = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    out = ((u + rounding) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bits to float32."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


# ----------------------------------------------------------------------------
# Layer inputs
# ----------------------------------------------------------------------------

@dataclass
class LayerInputs:
    cfg: LayerConfig
    x: np.ndarray  # [T, d] float32, or uint16 bf16 bits
    modality_id: np.ndarray  # [T] uint8, 0 = vision, 1 = text
    sample_offsets: np.ndarray  # [n_batch + 1] int32
    w_gate: np.ndarray  # [E, d] float32
    logit_bias: Optional[np.ndarray]  # [E] float32 or None
    expert_to_bin: np.ndarray  # [E] int32
    w13: np.ndarray  # [E, 2*inter, d]: rows [0, inter) gate, [inter, 2*inter) up
    w2: np.ndarray  # [E, d, inter]
    ws13: Optional[np.ndarray]  # [2*S*inter, d] merged shared gate/up, or None
    ws2: Optional[np.ndarray]  # [d, S*inter] merged shared down, or None
    mu_vision: np.ndarray = field(repr=False, default=None)  # generator means (float32)
    mu_text: np.ndarray = field(repr=False, default=None)

    def as_f32(self, name: str) -> np.ndarray:
        """A stored array widened exactly to float32 (bf16 bits are decoded)."""
        a = getattr(self, name)
        if a is None:
            return None
        if a.dtype == np.uint16:
            return bf16_bits_to_f32(a)
        return a


def _unit_norm_mean(rng: np.random.Generator, d: int) -> np.ndarray:
    v = rng.standard_normal(d, dtype=np.float32)
    return (v * np.float32(4.0 / np.linalg.norm(v.astype(np.float64)))).astype(np.float32)


def _store(a: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == BF16:
        return f32_to_bf16_bits(a)
    return np.ascontiguousarray(a, dtype=np.float32)


def make_layer_inputs(cfg: LayerConfig, with_weights: bool = True) -> LayerInputs:
    """Draw every input of one layer call, in a fixed order, from one seeded stream."""
    rng = np.random.default_rng(cfg.seed)
    d, T = cfg.d, cfg.T
    # 1. modality means, each N(0, I) scaled to norm 4
    mu_v = np.stack([_unit_norm_mean(rng, d) for _ in range(cfg.vision_clusters)])
    mu_t = _unit_norm_mean(rng, d)
    mu_v_bar = mu_v.mean(axis=0).astype(np.float32)
    # 2. layout: each sample is a vision block followed by a text block
    modality_id = np.empty(T, dtype=np.uint8)
    offsets = np.zeros(cfg.n_batch + 1, dtype=np.int32)
    pos = 0
    for i, (nv, nt) in enumerate(cfg.samples):
        modality_id[pos:pos + nv] = 0
        modality_id[pos + nv:pos + nv + nt] = 1
        pos += nv + nt
        offsets[i + 1] = pos
    is_v = modality_id == 0
    # 3. vision cluster per vision token
    cluster = np.zeros(T, dtype=np.int64)
    if cfg.vision_clusters > 1:
        cluster[is_v] = rng.integers(0, cfg.vision_clusters, size=int(is_v.sum()))
    # 4. x = own mean + N(0, I)
    own = np.where(is_v[:, None], mu_v[cluster], mu_t[None, :])
    x = own + rng.standard_normal((T, d), dtype=np.float32)
    # 5. cross-modal fusion: mix toward the other modality's mean by u ~ U(0, 0.5)
    u = rng.uniform(0.0, 0.5, size=T).astype(np.float32)
    other = np.where(is_v[:, None], mu_t[None, :], mu_v_bar[None, :])
    mixed = (1.0 - u)[:, None] * x + u[:, None] * other
    # 6. interpolated tokens: 0.5 a + 0.5 b, a ~ N(mu_v, I), b ~ N(mu_t, I)
    if cfg.interp_frac > 0:
        n_int = int(round(cfg.interp_frac * T))
        sel = rng.choice(T, size=n_int, replace=False)
        a = mu_v_bar[None, :] + rng.standard_normal((n_int, d), dtype=np.float32)
        b = mu_t[None, :] + rng.standard_normal((n_int, d), dtype=np.float32)
        mixed[sel] = 0.5 * a + 0.5 * b
    x = mixed.astype(np.float32)
    # 7. router weights, kept float32
    w_gate = (np.float32(0.02) * rng.standard_normal((cfg.E, d), dtype=np.float32))
    # 8. per-expert logit bias
    bias = rng.standard_normal(cfg.E, dtype=np.float32) if cfg.logit_bias else None
    # 9. expert weights: every matrix from its own child stream of the seed, so
    #    the matrices can be drawn in parallel and still be reproducible
    w13 = w2 = ws13 = ws2 = None
    if with_weights:
        wdt = np.uint16 if cfg.dtype == BF16 else np.float32
        w13 = np.empty((cfg.E, 2 * cfg.inter, d), dtype=wdt)
        w2 = np.empty((cfg.E, d, cfg.inter), dtype=wdt)
        si = cfg.shared_inter
        if cfg.n_shared > 0:
            ws13 = np.empty((2 * si, d), dtype=wdt)
            ws2 = np.empty((d, si), dtype=wdt)
        jobs = [(w13, e) for e in range(cfg.E)] + [(w2, e) for e in range(cfg.E)]
        if cfg.n_shared > 0:
            jobs += [(ws13, None), (ws2, None)]
        children = np.random.SeedSequence([cfg.seed, 0x5EED]).spawn(len(jobs))

        def draw(i):
            arr, e = jobs[i]
            dst = arr if e is None else arr[e]
            buf = np.random.default_rng(children[i]).standard_normal(dst.shape, dtype=np.float32)
            buf *= np.float32(0.02)
            dst[...] = _store(buf, cfg.dtype)

        workers = max(1, min(16, os.cpu_count() or 1))
        with cf.ThreadPoolExecutor(max_workers=workers) as ex:
            list(ex.map(draw, range(len(jobs))))
    # 10. activation storage type
    x_store = _store(x, cfg.dtype)
    # 12. fixed contiguous bins
    e2b = (np.arange(cfg.E) // cfg.n_per_bin).astype(np.int32)
    return LayerInputs(cfg, x_store, modality_id, offsets, w_gate.astype(np.float32),
                       None if bias is None else bias.astype(np.float32), e2b,
                       w13, w2, ws13, ws2, mu_vision=mu_v_bar, mu_text=mu_t)


def aligned_router(inp: LayerInputs, strength: float = 0.05) -> np.ndarray:
    """W_gate tilted so that the first half of every bin's experts leans to
    vision and the second half of the bins to text: W + s * sign (x) (mu_v - mu_t).

    Gives MI values of 1e-4..3e-2 nats, which makes MI comparisons well
    conditioned; the tilt is an input choice, not part of the method."""
    cfg = inp.cfg
    sign = np.where(inp.expert_to_bin < cfg.n_bins // 2, 1.0, -1.0).astype(np.float32)
    diff = (inp.mu_vision - inp.mu_text).astype(np.float32)
    return (inp.w_gate + np.float32(strength) * sign[:, None] * diff[None, :]).astype(np.float32)


# ----------------------------------------------------------------------------
# Inputs for the per-call checks (each entry point fed with the same arrays)
# ----------------------------------------------------------------------------

def random_offsets(rng: np.random.Generator, T: int, n_batch: int, allow_empty=False) -> np.ndarray:
    """Sorted sample boundaries 0 = o_0 <= ... <= o_n = T."""
    if n_batch == 1:
        return np.array([0, T], dtype=np.int32)
    lo = 0 if allow_empty else 1
    if not allow_empty and T < n_batch:
        raise ValueError("T < n_batch with non-empty samples")
    if allow_empty:
        cuts = np.sort(rng.integers(0, T + 1, size=n_batch - 1))
    else:
        cuts = np.sort(rng.choice(np.arange(lo, T), size=n_batch - 1, replace=False))
    return np.concatenate([[0], cuts, [T]]).astype(np.int32)


def random_probs(rng: np.random.Generator, T: int, E: int, concentration: float = 1.0) -> np.ndarray:
    """Rows on the probability simplex (Dirichlet draws), float32."""
    p = rng.dirichlet(np.full(E, concentration), size=T)
    p = np.maximum(p, 1e-30)
    return (p / p.sum(axis=1, keepdims=True)).astype(np.float32)


def random_soft_scores(rng: np.random.Generator, T: int) -> np.ndarray:
    """Soft modality scores [T, 2] (column 0 vision, column 1 text), float32."""
    a = rng.uniform(0.0, 1.0, size=T).astype(np.float32)
    return np.stack([a, np.float32(1.0) - a], axis=1).astype(np.float32)


def random_bin_map(rng: np.random.Generator, E: int, n_bins: int, contiguous=True) -> np.ndarray:
    """expert_to_bin with exactly E / n_bins experts per bin."""
    base = np.arange(E) // (E // n_bins)
    if contiguous:
        return base.astype(np.int32)
    return rng.permutation(base).astype(np.int32)


def random_topk(rng: np.random.Generator, T: int, E: int, k: int, skew: float = 0.0) -> np.ndarray:
    """k distinct experts per token. skew > 0 concentrates tokens on few experts."""
    keys = rng.random((T, E))
    if skew > 0:
        keys = keys * np.exp(-skew * np.arange(E) / E)[None, :]
    return np.argsort(-keys, axis=1, kind="stable")[:, :k].astype(np.int32)


def random_gauss_state(rng: np.random.Generator, d: int, count: float = 1000.0) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """A plausible caller-owned Gaussian-statistics state (N, S_mu, S_sigma2), float32."""
    n = np.array([count, 0.5 * count], dtype=np.float32)
    mu = rng.standard_normal((2, d)).astype(np.float32) * np.float32(0.3)
    var = rng.uniform(0.5, 2.0, size=(2, d)).astype(np.float32)
    return n, (n[:, None] * mu).astype(np.float32), (n[:, None] * var).astype(np.float32)


# ----------------------------------------------------------------------------
# Inputs of the attention-accumulated score (Sec. 3.2.1)
# ----------------------------------------------------------------------------

@dataclass
class AttnInputs:
    """One attention layer's tensors for the attention-accumulated score."""

    samples: Tuple[Tuple[int, int], ...]
    q: np.ndarray  # [T, H, d_head] bf16 bits
    k: np.ndarray  # [T, H_kv, d_head] bf16 bits
    v: np.ndarray  # [T, H_kv, d_head] bf16 bits
    x: np.ndarray  # [T, D] residual input of the attention sublayer, bf16 bits
    x_attn: np.ndarray  # [T, D] attention sublayer output, bf16 bits
    m_in: np.ndarray  # [T, 2] float32 input scores (vision, text)
    modality_id: np.ndarray  # [T] uint8, 0 vision / 1 text
    sample_offsets: np.ndarray  # [n_batch + 1] int32

    @property
    def T(self) -> int:
        return int(self.sample_offsets[-1])


def make_attention_inputs(samples, d: int, n_heads: int, n_kv_heads: int, head_dim: int, seed: int,
                          logit_std: float = 2.0) -> AttnInputs:
    """Seeded draws: q, k, v ~ N(0, s^2) with s^2 = logit_std, so that the logits
    q.k / sqrt(d_head) have standard deviation logit_std; x ~ N(0, 1) and
    x_attn ~ N(0, 0.5^2) per element; m_in soft scores with vision share
    U(0, 1). Samples are laid out vision block then text block, as in the
    layer workloads."""
    rng = np.random.default_rng(seed)
    T = sum(v + t for v, t in samples)
    s = np.float32(np.sqrt(logit_std))
    def draw(shape, scale):
        return f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32) * np.float32(scale))
    q = draw((T, n_heads, head_dim), s)
    k = draw((T, n_kv_heads, head_dim), s)
    v = draw((T, n_kv_heads, head_dim), 1.0)
    x = draw((T, d), 1.0)
    x_attn = draw((T, d), 0.5)
    m_in = random_soft_scores(rng, T)
    mid = np.concatenate([np.concatenate([np.zeros(a, np.uint8), np.ones(b, np.uint8)]) for a, b in samples]) \
        if samples else np.zeros(0, np.uint8)
    offsets = np.concatenate([[0], np.cumsum([a + b for a, b in samples])]).astype(np.int32)
    return AttnInputs(tuple(samples), q, k, v, x, x_attn, m_in, mid, offsets)


def random_gmm_state(rng: np.random.Generator, d: int, K: int, count: float = 1000.0,
                     spread: float = 0.5) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """EMA state of a K-component mixture per modality, components seeded
    apart: counts count * U(0.5, 1.5), means N(0, spread^2) per column,
    variances U(0.5, 2); returns float32 (N[2, K], S_mu[2, K, d], S_sigma2[2, K, d])."""
    n = (count * rng.uniform(0.5, 1.5, (2, K))).astype(np.float32)
    mu = (rng.standard_normal((2, K, d)) * spread).astype(np.float32)
    var = rng.uniform(0.5, 2.0, (2, K, d)).astype(np.float32)
    return n, (n[:, :, None] * mu).astype(np.float32), (n[:, :, None] * var).astype(np.float32)
