"""Seeded synthetic decode workloads for the retrospective sparse-attention step.

This module only *draws inputs*: prefill keys/values, the keys/values appended at
each decode step, and the query of each step.  It holds none of the method's
arithmetic (no scoring, selection, masking, attention or merging), so that both
the CPU oracle and the GPU path can consume the very same bits without sharing
any code that computes a result.

Shapes follow the paper's evaluation models (Llama-3.1-8B attention layout:
8 KV heads, 32 query heads, head_dim 128; Section "Experimental Setup").  The
paper's benchmarks (LongGenBench, PG-19, reasoning sets) need trained weights and
datasets; these seeded Gaussian streams stand in for them, with a planted
locality in the queries (each query is noise plus half of a random earlier key)
so that page selection moves from step to step.

bf16 workloads are rounded to bf16 on the host (round-to-nearest-even) and handed
out as float32 arrays whose values are exactly representable in bf16, so that a
float32 consumer and a bf16 consumer see identical numbers.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

__all__ = ["Spec", "Generator", "QueryWindow", "DecoderInputs", "CONFIGS", "config",
           "round_bf16", "config4_combos"]


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); return float32.

    Only finite inputs are expected (the generator draws Gaussians).
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).reshape(x.shape)


@dataclass(frozen=True)
class Spec:
    """One synthetic decode workload (a single attention layer)."""

    name: str
    batch: int
    num_kv_heads: int
    group: int              # query heads per KV head (GQA); h_q = num_kv_heads * group
    head_dim: int
    page_size: int
    budget: int             # token budget B (the minimum one with budget_permille)
    window: int             # W = number of past queries revisited each step
    steps: int
    dtype: str              # "f32" or "bf16"
    prefill: Tuple[int, ...]  # prefill length of each sequence
    tokens_per_step: int = 1  # tokens appended per step; the step's query sits on the last
    key_model: str = "normal"  # "normal" | "outlier" | "drift"
    outlier_channels: int = 0
    outlier_scale: float = 1.0
    drift_step: float = 0.0
    seed: int = 0
    budget_permille: int = 0  # relative budget: max(B, len * permille / 1000) tokens per step
    reuse_interval: int = 0   # top-k reuse: selection refreshed on steps t % f == 0 (0, 1: every step)

    @property
    def num_q_heads(self) -> int:
        return self.num_kv_heads * self.group

    @property
    def max_tokens(self) -> int:
        return max(self.prefill) + self.steps * self.tokens_per_step

    @property
    def max_pages(self) -> int:
        return -(-self.max_tokens // self.page_size)

    @property
    def k_max(self) -> int:
        return min(self.budget // self.page_size, self.max_pages)

    @property
    def rows(self) -> int:
        return (self.window + 1) * self.group

    def replace(self, **kw) -> "Spec":
        d = dict(self.__dict__)
        d.update(kw)
        return Spec(**d)


def _config2_prefill(seed: int, batch: int) -> Tuple[int, ...]:
    rng = np.random.default_rng(np.random.SeedSequence([seed, 7]))
    return tuple(int(x) for x in rng.integers(8192, 32768, size=batch, endpoint=True))


def _make_configs() -> List[Spec]:
    c0 = Spec("tiny-fp32", batch=1, num_kv_heads=2, group=4, head_dim=64, page_size=16,
              budget=256, window=4, steps=32, dtype="f32", prefill=(2048,), seed=0)
    c1 = Spec("llama3-8b-layer-32k", batch=1, num_kv_heads=8, group=4, head_dim=128,
              page_size=16, budget=2048, window=16, steps=256, dtype="bf16",
              prefill=(32768,), key_model="outlier", outlier_channels=4,
              outlier_scale=8.0, seed=1)
    c2 = Spec("batched-serving-b16", batch=16, num_kv_heads=8, group=4, head_dim=128,
              page_size=16, budget=1024, window=8, steps=128, dtype="bf16",
              prefill=_config2_prefill(2, 16), seed=2)
    c3 = Spec("long-generation-stress", batch=4, num_kv_heads=8, group=8, head_dim=128,
              page_size=16, budget=4096, window=32, steps=4096, dtype="bf16",
              prefill=(16384,) * 4, tokens_per_step=8, key_model="drift",
              drift_step=0.01, seed=3)
    c4 = Spec("extreme-context-131k", batch=1, num_kv_heads=8, group=4, head_dim=128,
              page_size=32, budget=8192, window=64, steps=64, dtype="bf16",
              prefill=(131072,), seed=4)
    return [c0, c1, c2, c3, c4]


CONFIGS: List[Spec] = _make_configs()


def config(i: int) -> Spec:
    return CONFIGS[i]


def config4_combos() -> List[Tuple[int, int]]:
    """(budget, window) pairs of the extreme-context sweep."""
    return [(b, w) for b in (1024, 2048, 4096, 8192) for w in (0, 4, 16, 64)]


class Generator:
    """Deterministic stream of inputs for one Spec.

    * ``prefill()`` returns, per sequence, keys and values ``[n][h_k][d]``.
    * ``step(t)`` returns the tokens appended at decode step ``t``
      (``k_new, v_new``: ``[tokens_per_step][batch][h_k][d]``) and the step's query
      ``q`` (``[batch][h_q][d]``); the query is ``N(0, I) + 0.5 * K[r]`` for an
      earlier position ``r`` drawn uniformly below the query's own position.

    Keys are kept (per sequence) so later queries can plant them.
    """

    def __init__(self, spec: Spec, seed: Optional[int] = None):
        self.spec = spec
        self.seed = spec.seed if seed is None else seed
        s = spec
        self._bf16 = s.dtype == "bf16"
        self.keys = [np.zeros((s.max_tokens, s.num_kv_heads, s.head_dim), np.float32)
                     for _ in range(s.batch)]
        self.lens = [0] * s.batch
        self._mu = np.zeros((s.batch, s.num_kv_heads, s.head_dim), np.float32)
        self._outlier = None
        if s.key_model == "outlier":
            rng = np.random.default_rng(np.random.SeedSequence([self.seed, 0]))
            self._outlier = np.stack([rng.choice(s.head_dim, s.outlier_channels, replace=False)
                                      for _ in range(s.num_kv_heads)])
        self._prefilled = False

    # -- helpers -------------------------------------------------------------
    def _q(self, x: np.ndarray) -> np.ndarray:
        return round_bf16(x) if self._bf16 else np.ascontiguousarray(x, np.float32)

    def _draw_keys(self, rng: np.random.Generator, b: int, n: int) -> np.ndarray:
        s = self.spec
        k = rng.standard_normal((n, s.num_kv_heads, s.head_dim), dtype=np.float32)
        if s.key_model == "outlier":
            for h in range(s.num_kv_heads):
                k[:, h, self._outlier[h]] *= np.float32(s.outlier_scale)
        elif s.key_model == "drift":
            inc = rng.standard_normal((n, s.num_kv_heads, s.head_dim), dtype=np.float32)
            inc *= np.float32(s.drift_step)
            mu = self._mu[b][None] + np.cumsum(inc, axis=0, dtype=np.float32)
            self._mu[b] = mu[-1]
            k += mu
        return self._q(k)

    # -- public ----------------------------------------------------------------
    def prefill(self) -> List[Tuple[np.ndarray, np.ndarray]]:
        s = self.spec
        out = []
        for b in range(s.batch):
            n = s.prefill[b]
            rng = np.random.default_rng(np.random.SeedSequence([self.seed, 1, b]))
            k = self._draw_keys(rng, b, n)
            v = self._q(rng.standard_normal((n, s.num_kv_heads, s.head_dim), dtype=np.float32))
            self.keys[b][:n] = k
            self.lens[b] = n
            out.append((k, v))
        self._prefilled = True
        return out

    def step(self, t: int):
        assert self._prefilled, "prefill() first"
        s = self.spec
        T = s.tokens_per_step
        rng = np.random.default_rng(np.random.SeedSequence([self.seed, 2, t]))
        k_new = np.zeros((T, s.batch, s.num_kv_heads, s.head_dim), np.float32)
        v_new = np.zeros_like(k_new)
        for b in range(s.batch):
            k = self._draw_keys(rng, b, T)
            v = self._q(rng.standard_normal((T, s.num_kv_heads, s.head_dim), dtype=np.float32))
            n = self.lens[b]
            self.keys[b][n:n + T] = k
            self.lens[b] = n + T
            k_new[:, b] = k
            v_new[:, b] = v
        q = np.zeros((s.batch, s.num_q_heads, s.head_dim), np.float32)
        for b in range(s.batch):
            pos = self.lens[b] - 1          # the query sits on the step's last token
            r = rng.integers(0, pos, size=s.num_q_heads)
            noise = rng.standard_normal((s.num_q_heads, s.head_dim), dtype=np.float32)
            heads = np.arange(s.num_q_heads) // s.group
            q[b] = noise + np.float32(0.5) * self.keys[b][r, heads]
        return k_new, v_new, self._q(q)


class QueryWindow:
    """The queries of the last W+1 steps, ``[batch][W+1][h_q][d]``.

    Row ``W`` is the current step's query, row ``r`` the query of step ``t-W+r``;
    rows of steps before the first decode step stay zero.
    """

    def __init__(self, spec: Spec):
        s = spec
        self.q = np.zeros((s.batch, s.window + 1, s.num_q_heads, s.head_dim), np.float32)

    def push(self, q: np.ndarray) -> np.ndarray:
        if self.q.shape[1] > 1:
            self.q[:, :-1] = self.q[:, 1:]
        self.q[:, -1] = q
        return self.q


class DecoderInputs:
    """Seeded inputs of a multi-layer synthetic decode with re-embedding.

    ``num_layers`` attention layers of the Spec's shape with model width
    ``d_model = h_q * d`` (the Llama layout: 32 query heads of 128 = 4096):

    * ``weights()``: per layer the query, key, value and output projections
      ``wq [d_model][h_q*d]``, ``wk``, ``wv [d_model][h_k*d]``, ``wo [h_q*d][d_model]``,
      Gaussian with variance 1/fan_in (the output projection further scaled by
      1/sqrt(num_layers), which keeps the residual stream's size bounded over depth);
    * ``prefill(layer)``: that layer's prompt keys and values, as ``Generator.prefill``
      (an independent stream per layer);
    * ``embedding(t)``: the embedding ``[batch][d_model]`` of the token decoded at step
      ``t`` (unit Gaussian).

    Trained weights do not exist here; these random ones stand in for them.  Values
    are rounded to bf16 for bf16 Specs, like every other input of this module.
    """

    def __init__(self, spec: Spec, num_layers: int, seed: Optional[int] = None):
        self.spec = spec
        self.num_layers = num_layers
        self.seed = spec.seed if seed is None else seed
        self.d_model = spec.num_q_heads * spec.head_dim
        self._bf16 = spec.dtype == "bf16"

    def _q(self, x: np.ndarray) -> np.ndarray:
        return round_bf16(x) if self._bf16 else np.ascontiguousarray(x, np.float32)

    def weights(self) -> List[dict]:
        s, dm = self.spec, self.d_model
        hq_d, hk_d = s.num_q_heads * s.head_dim, s.num_kv_heads * s.head_dim
        out = []
        for layer in range(self.num_layers):
            rng = np.random.default_rng(np.random.SeedSequence([self.seed, 10, layer]))

            def draw(rows, cols, scale):
                w = rng.standard_normal((rows, cols), dtype=np.float32)
                return self._q(w * np.float32(scale))

            out.append(dict(wq=draw(dm, hq_d, dm ** -0.5), wk=draw(dm, hk_d, dm ** -0.5),
                            wv=draw(dm, hk_d, dm ** -0.5),
                            wo=draw(hq_d, dm, (hq_d * self.num_layers) ** -0.5)))
        return out

    def prefill(self, layer: int) -> List[Tuple[np.ndarray, np.ndarray]]:
        return Generator(self.spec, seed=self.seed * 1000 + 11 + layer).prefill()

    def embedding(self, t: int) -> np.ndarray:
        rng = np.random.default_rng(np.random.SeedSequence([self.seed, 12, t]))
        return self._q(rng.standard_normal((self.spec.batch, self.d_model), dtype=np.float32))
