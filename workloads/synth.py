"""Seeded synthetic decode workloads with the shapes of the paper's evaluation.

The paper measures on real models (GLM-4-9B, Llama-3-8B, ...) over long-context
benchmarks (Section 5.1).  Neither weights nor datasets are used here: these
generators stand in for them with inputs of the same shapes (query/KV head counts,
head dimension, context length, page or block size, token budget) and with a
controllable temporal locality of the selected pages:

* keys and values are i.i.d. N(0, 1), drawn in float32 and rounded (nearest-even)
  to the storage dtype; the rounded values are *the* inputs of every consumer;
* a small set of "hot" pages per KV head gets +2.0 along one random unit direction
  added to all of its keys before rounding, so that some pages are persistently
  relevant;
* queries follow an AR(1) process per element, q_t = rho * q_{t-1} + sigma * eps_t,
  which gives consecutive decode steps overlapping selections (Section 2.2 reports
  about 68% overlap on real models);
* the Llama-shaped workload re-draws its hot set every 16 steps (a drifting context).

Every random stream is a PCG64 generator seeded by
``SeedSequence([2606, config_id, layer, stream, ...])`` with stream ids
K=0, V=1, hot set=2, queries=3, drift=4; per-KV-head streams append the head index,
so any head's pages can be regenerated on their own.

Nothing in this module computes any part of the decode method.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np

SEED_ROOT = 2606
STREAM_K, STREAM_V, STREAM_HOT, STREAM_Q, STREAM_DRIFT, STREAM_PREFILL = 0, 1, 2, 3, 4, 5
HOT_SHIFT = 2.0


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    cfg_id: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    dtype: str  # "f16" | "bf16"
    context: int  # tokens in the KV cache
    page_size: int
    k_select: int  # top-K budget in pages
    forced: str  # "none" | "first_last" | "initial_local2"
    forced_in_budget: bool  # True: |A| = k_select (forced included); False: |A| = k_select + n_forced
    meta_kind: str  # "minmax" (Quest) | "mean" (block-mean keys)
    steps: int  # timed decode steps after the step-0 prefill stand-in
    layers: int
    hot_count: int  # hot pages per KV head
    rho: float
    sigma: float
    drift_every: int = 0  # re-draw the hot set every this many steps (0 = never)
    alpha: float = 0.5
    beta: float = 0.5
    gamma: float = 0.0

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def num_pages(self) -> int:
        return (self.context + self.page_size - 1) // self.page_size

    def forced_pages(self, num_pages: Optional[int] = None) -> List[int]:
        n = self.num_pages if num_pages is None else num_pages
        if self.forced == "none":
            return []
        if self.forced == "first_last":
            return sorted({0, n - 1})
        if self.forced == "initial_local2":
            return sorted({0, n - 2, n - 1})
        raise ValueError(self.forced)

    @property
    def selected_count(self) -> int:
        nf = len(self.forced_pages())
        k = self.k_select if self.forced_in_budget else self.k_select + nf
        return min(k, self.num_pages)


def _ar_sigma(rho: float) -> float:
    # unit stationary variance of the AR(1) query process
    return math.sqrt(1.0 - rho * rho)


CONFIGS: Dict[str, Config] = {
    c.name: c
    for c in [
        Config("tiny", 0, 4, 1, 128, "f16", 2048, 16, 16, "none", True, "minmax",
               16, 1, 8, 0.9, 0.44),
        Config("glm32k", 1, 32, 2, 128, "bf16", 32768, 16, 128, "first_last", True, "minmax",
               64, 1, 64, 0.9, _ar_sigma(0.9)),
        Config("glm128k", 2, 32, 2, 128, "bf16", 131072, 16, 256, "none", True, "minmax",
               128, 40, 82, 0.95, _ar_sigma(0.95)),
        Config("llama64k", 3, 32, 8, 128, "f16", 65536, 16, 128, "none", True, "minmax",
               128, 32, 82, 0.85, _ar_sigma(0.85), drift_every=16),
        Config("infllm128k", 4, 32, 2, 128, "bf16", 131072, 64, 64, "initial_local2", False, "mean",
               128, 40, 20, 0.9, _ar_sigma(0.9)),
    ]
}


# ----------------------------------------------------------------------------- dtype helpers

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns the uint16 bit patterns."""
    u = np.array(x, dtype=np.float32, copy=True).view(np.uint32)
    bias = u >> np.uint32(16)
    bias &= np.uint32(1)
    bias += np.uint32(0x7FFF)
    u += bias
    u >>= np.uint32(16)
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def f32_to_dtype_bits(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    if dtype == "f16":
        return np.asarray(x, dtype=np.float32).astype(np.float16).view(np.uint16)
    raise ValueError(dtype)


def bits_to_f64(b: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 value of each stored 16-bit element."""
    if dtype == "bf16":
        return bf16_bits_to_f32(b).astype(np.float64)
    if dtype == "f16":
        return np.asarray(b, dtype=np.uint16).view(np.float16).astype(np.float64)
    raise ValueError(dtype)


# ----------------------------------------------------------------------------- generators

def _rng(*words: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, *words])))


def _hot_direction_and_pages(cfg: Config, layer: int, head: int, num_pages: int):
    rng = _rng(cfg.cfg_id, layer, STREAM_HOT, head)
    n_hot = min(cfg.hot_count, num_pages)
    pages = np.sort(rng.choice(num_pages, size=n_hot, replace=False)).astype(np.int64)
    u = rng.standard_normal(cfg.head_dim)
    u = (u / np.linalg.norm(u)).astype(np.float32)
    return u, pages


def hot_pages(cfg: Config, layer: int, head: int, epoch: int = 0,
              num_pages: Optional[int] = None) -> np.ndarray:
    """Hot pages of one KV head at drift epoch ``epoch`` (epoch = step // drift_every)."""
    n = cfg.num_pages if num_pages is None else num_pages
    _, pages = _hot_direction_and_pages(cfg, layer, head, n)
    for e in range(1, epoch + 1):
        rng = _rng(cfg.cfg_id, layer, STREAM_DRIFT, head, e)
        others = np.setdiff1d(np.arange(n), pages)
        k = min(len(pages), len(others))
        pages = np.sort(rng.choice(others, size=k, replace=False)).astype(np.int64)
    return pages


@dataclasses.dataclass
class LayerInputs:
    cfg: Config
    layer: int
    epoch: int
    k_bits: np.ndarray  # [Hkv][N][page][d] uint16, logical page order
    v_bits: np.ndarray  # [Hkv][N][page][d] uint16
    hot: np.ndarray  # [Hkv][H] int64

    def k64(self) -> np.ndarray:
        return bits_to_f64(self.k_bits, self.cfg.dtype)

    def v64(self) -> np.ndarray:
        return bits_to_f64(self.v_bits, self.cfg.dtype)


def layer_inputs(cfg: Config, layer: int = 0, epoch: int = 0,
                 num_pages: Optional[int] = None, heads: Optional[List[int]] = None) -> LayerInputs:
    """Keys and values of one layer, rounded to the config dtype.

    ``num_pages`` shrinks the context (tests); ``heads`` restricts to some KV heads.
    """
    n = cfg.num_pages if num_pages is None else num_pages
    hs = list(range(cfg.num_kv_heads)) if heads is None else list(heads)
    shape = (n, cfg.page_size, cfg.head_dim)
    k_bits = np.empty((len(hs),) + shape, dtype=np.uint16)
    v_bits = np.empty((len(hs),) + shape, dtype=np.uint16)
    hot_all = []
    for i, h in enumerate(hs):
        u, _ = _hot_direction_and_pages(cfg, layer, h, n)
        hot = hot_pages(cfg, layer, h, epoch, n)
        kb = _rng(cfg.cfg_id, layer, STREAM_K, h).standard_normal(shape, dtype=np.float32)
        kb[hot] += np.float32(HOT_SHIFT) * u
        k_bits[i] = f32_to_dtype_bits(kb, cfg.dtype)
        del kb
        vb = _rng(cfg.cfg_id, layer, STREAM_V, h).standard_normal(shape, dtype=np.float32)
        v_bits[i] = f32_to_dtype_bits(vb, cfg.dtype)
        del vb
        hot_all.append(hot)
    return LayerInputs(cfg, layer, epoch, k_bits, v_bits, np.stack(hot_all))


def query_trajectory(cfg: Config, layer: int = 0, steps: Optional[int] = None):
    """AR(1) queries for steps 0..steps (step 0 stands in for the last prefill token).

    Returns (latent float32 [T+1][Hq][d], stored bits uint16 [T+1][Hq][d]).
    """
    t_total = (cfg.steps if steps is None else steps) + 1
    rng = _rng(cfg.cfg_id, layer, STREAM_Q)
    shape = (cfg.num_q_heads, cfg.head_dim)
    lat = np.empty((t_total,) + shape, dtype=np.float32)
    lat[0] = rng.standard_normal(shape, dtype=np.float32)
    rho, sig = np.float32(cfg.rho), np.float32(cfg.sigma)
    for t in range(1, t_total):
        lat[t] = rho * lat[t - 1] + sig * rng.standard_normal(shape, dtype=np.float32)
    return lat, f32_to_dtype_bits(lat, cfg.dtype)


def prefill_trajectory(cfg: Config, layer: int = 0, rows: int = 16, stride: int = 1):
    """The queries of `rows` prefill tokens `stride` tokens apart, ending with the step-0
    query: the AR(1) process run backwards from q_0 (it is time-reversible), drawn from its
    own stream; `stride` steps of it at once are one step with coefficient rho^stride and
    noise sigma * sqrt((1 - rho^(2 stride)) / (1 - rho^2)).  Returns stored bits uint16
    [rows][Hq][d] in time order."""
    lat0, _ = query_trajectory(cfg, layer, steps=0)
    rng = _rng(cfg.cfg_id, layer, STREAM_PREFILL) if stride == 1 else _rng(cfg.cfg_id, layer, STREAM_PREFILL, stride)
    shape = (cfg.num_q_heads, cfg.head_dim)
    lat = np.empty((rows,) + shape, dtype=np.float32)
    lat[rows - 1] = lat0[0]
    rho_s = cfg.rho ** stride
    sig_s = cfg.sigma * math.sqrt((1.0 - rho_s * rho_s) / (1.0 - cfg.rho * cfg.rho)) if stride > 1 else cfg.sigma
    rho, sig = np.float32(rho_s), np.float32(sig_s)
    for r in range(rows - 2, -1, -1):
        lat[r] = rho * lat[r + 1] + sig * rng.standard_normal(shape, dtype=np.float32)
    return f32_to_dtype_bits(lat, cfg.dtype)


def page_table_permutation(num_logical: int, num_physical: int, seed: int) -> np.ndarray:
    """A random injective logical->physical page map (tests of the paged layout)."""
    rng = _rng(9999, seed)
    return rng.permutation(num_physical)[:num_logical].astype(np.int32)


def to_physical(bits: np.ndarray, page_table: np.ndarray, num_physical: int) -> np.ndarray:
    """Scatter logically ordered pages [Hkv][N][...] into physical slots [Hkv][num_physical][...]."""
    out = np.zeros((bits.shape[0], num_physical) + bits.shape[2:], dtype=bits.dtype)
    out[:, page_table] = bits
    return out
