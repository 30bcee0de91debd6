"""Seeded synthetic decode workloads for SANTA++ attention.

This module only draws inputs; it holds none of the method's arithmetic.
Both the CPU oracle (through the tests) and the GPU path (through the tests,
``bench.py`` and ``smoke()``) read the same bytes produced here.

Recipe (one KV head of one sequence):

* ``C`` cluster centres ``mu_c = r * z / |z|`` with ``z ~ N(0, I_d)``.
* Cluster labels i.i.d. uniform over the ``C`` clusters, or Zipf-weighted
  (``w_c ~ (c+1)^-s``) for the skewed long-context workload.
* Keys ``k_i = mu_{c(i)} + sigma * N(0, I_d)``; values ``v_i ~ N(0, I_d)``.
* ``n_outliers`` key channels, drawn once per KV head, are multiplied by
  ``outlier_scale`` after the mixture draw (keys only), mimicking the large
  per-channel magnitudes of post-RoPE keys.
* One focus cluster ``f`` per KV head; each of the ``G`` query heads sharing
  the KV head gets ``q_h = mu_f + q_sigma * N(0, I_d)`` (unscaled; the softmax
  scale ``1/sqrt(d)`` is applied once by the attention itself).
* The generated suffix rows come from the same mixture as the prompt.
* Keys and values are drawn in fp32 and rounded once to bf16
  (round-to-nearest-even) for the bf16 workloads; both sides read those
  exact bf16 values.  Queries stay fp32.

The workloads stand in for the captured Qwen2.5-7B-Instruct layer cache used
by the paper's kernel benchmark (Appendix "Kernel evaluation protocol"),
which is not available: same head counts, head dimension, context lengths and
budgets, synthetic contents.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np

BF16 = "bf16"
FP32 = "fp32"


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    d: int
    N: int
    dtype: str
    n_clusters: int
    center_norm: float
    P: int
    R: int
    K: int
    T: int
    data_seeds: Sequence[int]
    sigma: float = 1.0
    q_sigma: float = 0.5
    n_outliers: int = 0
    outlier_scale: float = 10.0
    zipf: Optional[float] = None
    seed: int = 0  # sampling seed (Philox key)

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # Tiny CPU-seconds case: one head, d = 64, fp32, 16 clusters of norm 4.
    "tiny": Workload("tiny", B=1, Hq=1, Hkv=1, d=64, N=1024, dtype=FP32,
                     n_clusters=16, center_norm=4.0, P=256, R=8, K=8, T=16,
                     data_seeds=(0,)),
    # Qwen2.5-7B-shaped layer (28 Q / 4 KV heads, d = 128, bf16) at 8K.
    "qwen8k": Workload("qwen8k", B=1, Hq=28, Hkv=4, d=128, N=8192, dtype=BF16,
                       n_clusters=256, center_norm=8.0, P=1024, R=16, K=32,
                       T=64, data_seeds=(1,), n_outliers=4),
    # Headline: the same layer shape at a 32768-token prompt.
    "qwen32k": Workload("qwen32k", B=1, Hq=28, Hkv=4, d=128, N=32768,
                        dtype=BF16, n_clusters=256, center_norm=8.0, P=1024,
                        R=16, K=32, T=128, data_seeds=(2,), n_outliers=4),
    # Batched decode: 8 independent sequences, 512 generated suffix rows.
    "batched": Workload("batched", B=8, Hq=28, Hkv=4, d=128, N=32768,
                        dtype=BF16, n_clusters=256, center_norm=8.0, P=1024,
                        R=16, K=32, T=512, data_seeds=tuple(range(3, 11)),
                        n_outliers=4),
    # Long, skewed context: Zipf(1.2) cluster populations at 131072 tokens.
    "long": Workload("long", B=4, Hq=28, Hkv=4, d=128, N=131072, dtype=BF16,
                     n_clusters=256, center_norm=8.0, P=1024, R=16, K=64,
                     T=256, data_seeds=(11, 12, 13, 14), n_outliers=4,
                     zipf=1.2),
    # Limiting case: every key is its own team (P = R = 1) at 8K.
    "limit": Workload("limit", B=1, Hq=28, Hkv=4, d=128, N=8192, dtype=BF16,
                      n_clusters=256, center_norm=8.0, P=1, R=1, K=64, T=64,
                      data_seeds=(1,), n_outliers=4),
}


def round_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    return ((b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclasses.dataclass
class Batch:
    """One decode step's inputs.  K/V arrays are ``[B, Hkv, rows, d]``.

    For bf16 workloads ``K, V, sK, sV`` hold uint16 bf16 bit patterns; for
    fp32 workloads they hold float32.  ``q`` is float32 ``[B, Hq, d]``.
    """
    wl: Workload
    q: np.ndarray
    K: np.ndarray
    V: np.ndarray
    sK: np.ndarray
    sV: np.ndarray
    focus: np.ndarray  # [B, Hkv] focus cluster of the queries
    labels: Optional[np.ndarray] = None  # [B, Hkv, N] cluster of each key

    def f32(self, a: np.ndarray) -> np.ndarray:
        """The exact values as float32 (bf16 widened, or the fp32 array)."""
        return bf16_bits_to_f32(a) if self.wl.dtype == BF16 else a

    def f64(self, a: np.ndarray) -> np.ndarray:
        return self.f32(a).astype(np.float64)


def _unit_rows(rng: np.random.Generator, n: int, d: int) -> np.ndarray:
    z = rng.standard_normal((n, d))
    return z / np.linalg.norm(z, axis=1, keepdims=True)


def generate(wl: Workload, keep_labels: bool = False) -> Batch:
    """Draw one batch for ``wl``; deterministic in ``wl.data_seeds``."""
    B, Hkv, G, d, N, T = wl.B, wl.Hkv, wl.G, wl.d, wl.N, wl.T
    if len(wl.data_seeds) != B:
        raise ValueError("one data seed per sequence is required")
    store = np.uint16 if wl.dtype == BF16 else np.float32
    q = np.empty((B, wl.Hq, d), np.float32)
    K = np.empty((B, Hkv, N, d), store)
    V = np.empty((B, Hkv, N, d), store)
    sK = np.empty((B, Hkv, T, d), store)
    sV = np.empty((B, Hkv, T, d), store)
    focus = np.empty((B, Hkv), np.int64)
    labels_all = np.empty((B, Hkv, N), np.int32) if keep_labels else None
    C = wl.n_clusters
    if wl.zipf is not None:
        w = (np.arange(C, dtype=np.float64) + 1.0) ** (-wl.zipf)
        w /= w.sum()
    else:
        w = None

    def draw_labels(rng, n):
        if w is None:
            return rng.integers(0, C, size=n)
        return rng.choice(C, size=n, p=w)

    def fin(x):
        return round_bf16_bits(x) if wl.dtype == BF16 else x.astype(np.float32)

    for b in range(B):
        rng = np.random.default_rng(wl.data_seeds[b])
        for kv in range(Hkv):
            centers = (wl.center_norm * _unit_rows(rng, C, d)).astype(np.float32)
            lab = draw_labels(rng, N)
            keys = centers[lab] + np.float32(wl.sigma) * rng.standard_normal((N, d), dtype=np.float32)
            vals = rng.standard_normal((N, d), dtype=np.float32)
            outl = rng.choice(d, size=wl.n_outliers, replace=False) if wl.n_outliers else np.empty(0, np.int64)
            keys[:, outl] *= np.float32(wl.outlier_scale)
            f = int(rng.integers(0, C))
            qh = centers[f][None, :] + np.float32(wl.q_sigma) * rng.standard_normal((G, d), dtype=np.float32)
            slab = draw_labels(rng, T)
            skeys = centers[slab] + np.float32(wl.sigma) * rng.standard_normal((T, d), dtype=np.float32)
            skeys[:, outl] *= np.float32(wl.outlier_scale)
            svals = rng.standard_normal((T, d), dtype=np.float32)
            q[b, kv * G:(kv + 1) * G] = qh
            K[b, kv] = fin(keys)
            V[b, kv] = fin(vals)
            sK[b, kv] = fin(skeys)
            sV[b, kv] = fin(svals)
            focus[b, kv] = f
            if keep_labels:
                labels_all[b, kv] = lab
    return Batch(wl, q, K, V, sK, sV, focus, labels_all)


def decode_trace(wl: Workload, layers: int, steps: int):
    """Inputs of a synthetic multi-layer decode loop of ``steps`` steps.

    Layer l is a batch drawn like ``wl`` from its own data seeds, with
    ``T = steps`` suffix rows: row t of each (b, kv) is the key/value the
    loop generates at step t (drawn like the prompt's keys and values, from
    the layer's clusters).  Step t's queries are the batch's queries plus
    N(0, 0.25^2) drift per coordinate, from a generator seeded by the layer.
    Returns a list of (batch, queries [steps, B, Hq, d] fp32), one per layer.
    """
    out = []
    for layer in range(layers):
        wl_l = wl.with_(name=f"{wl.name}-layer{layer}", T=steps,
                        data_seeds=tuple(s + 7919 * (layer + 1) for s in wl.data_seeds))
        b = generate(wl_l)
        rng = np.random.default_rng([layer, 104729])
        qs = (b.q[None].astype(np.float64) + 0.25 * rng.standard_normal((steps,) + b.q.shape)).astype(np.float32)
        out.append((b, qs))
    return out


def get(name: str, **overrides) -> Batch:
    wl = WORKLOADS[name]
    if overrides:
        wl = wl.with_(**overrides)
    return generate(wl)


def small_case(seed: int, N: int, d: int, T: int = 0, logit_scale: float = 1.0,
               Hq: int = 1, Hkv: int = 1, B: int = 1):
    """Tiny unstructured inputs for statistical and invariance tests.

    Returns float64 arrays ``q [B,Hq,d]``, ``K, V [B,Hkv,N,d]`` and
    ``sK, sV [B,Hkv,T,d]`` whose values are exactly representable in fp32.
    """
    rng = np.random.default_rng(seed)
    q = (logit_scale * rng.standard_normal((B, Hq, d))).astype(np.float32).astype(np.float64)
    K = rng.standard_normal((B, Hkv, N, d)).astype(np.float32).astype(np.float64)
    V = rng.standard_normal((B, Hkv, N, d)).astype(np.float32).astype(np.float64)
    sK = rng.standard_normal((B, Hkv, T, d)).astype(np.float32).astype(np.float64)
    sV = rng.standard_normal((B, Hkv, T, d)).astype(np.float32).astype(np.float64)
    return q, K, V, sK, sV
