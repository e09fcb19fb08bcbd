"""Seeded synthetic workloads for the vector-index output head.

This module only draws random numbers and casts them to the storage dtype; it
holds none of the head's arithmetic (no scores, no top-k, no graph). Both the
HIP path and the CPU oracle receive the arrays it returns, so neither side ever
generates its own inputs.

The paper measures on real hidden states and real model matrices (Section 4,
"Output Embedding Benchmarks" and "Index Accuracy"); none are available here,
so these arrays stand in for them with the paper's shapes:

* ``W_out`` rows: ``w_i = r_i * g_i`` with ``g_i ~ N(0, I/d)`` and per-row norm
  scale ``r_i ~ LogNormal(0, 0.25)``; for the Gemma-shaped head 10 % of the rows
  (chosen without replacement) get ``r_i *= 3`` ("hub" tokens).
* queries: ``h = w_a + w_b + w_c + n`` for three distinct uniformly chosen rows
  of the *stored* matrix and ``n ~ N(0, 0.1/d)`` per coordinate.
* storage: fp32, or bf16 rounded to nearest-even from fp32 (returned as the raw
  uint16 bit patterns, so both sides read exactly the same values).

Random streams (numpy PCG64): norms and rows from ``seed_w``, hub choice from
``seed_hub``, queries from ``seed_q``. Rows are drawn in blocks so the largest
matrix (788 MB of bf16) never needs a float64 copy of itself.
"""
from __future__ import annotations

import dataclasses
import numpy as np

F32 = 0
BF16 = 1
DTYPE_NAMES = {F32: "f32", BF16: "bf16"}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to fp32 exactly."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def stored_values_f32(W: np.ndarray, dtype: int) -> np.ndarray:
    """Exact fp32 view of a stored matrix (fp32 array, or bf16 bits)."""
    return W if dtype == F32 else bf16_bits_to_f32(W)


def _cast(x64: np.ndarray, dtype: int) -> np.ndarray:
    x32 = x64.astype(np.float32)
    return x32 if dtype == F32 else f32_to_bf16_bits(x32)


def make_w(V: int, d: int, dtype: int, seed_w: int, hub_frac: float = 0.0,
           hub_scale: float = 3.0, seed_hub: int | None = None,
           block_rows: int = 8192) -> np.ndarray:
    """Synthetic output-embedding matrix [V, d] in the storage dtype."""
    rng = np.random.Generator(np.random.PCG64(seed_w))
    r = rng.lognormal(mean=0.0, sigma=0.25, size=V)
    if hub_frac > 0.0:
        hub_rng = np.random.Generator(np.random.PCG64(seed_hub if seed_hub is not None else seed_w + 2000))
        n_hub = int(round(hub_frac * V))
        r[hub_rng.choice(V, size=n_hub, replace=False)] *= hub_scale
    out = np.empty((V, d), dtype=np.float32 if dtype == F32 else np.uint16)
    inv = 1.0 / np.sqrt(d)
    for r0 in range(0, V, block_rows):
        r1 = min(V, r0 + block_rows)
        g = rng.standard_normal((r1 - r0, d)) * inv
        out[r0:r1] = _cast(g * r[r0:r1, None], dtype)
    return out


def make_queries(W: np.ndarray, dtype: int, Q: int, seed_q: int,
                 noise_var: float = 0.1, n_rows: int = 3) -> tuple[np.ndarray, np.ndarray]:
    """Queries [Q, d] in the storage dtype, and the planted row ids [Q, n_rows]."""
    V, d = W.shape
    rng = np.random.Generator(np.random.PCG64(seed_q))
    planted = np.empty((Q, n_rows), dtype=np.int64)
    H = np.empty((Q, d), dtype=np.float64)
    sd = np.sqrt(noise_var / d)
    for q in range(Q):
        idx = rng.choice(V, size=n_rows, replace=False)
        planted[q] = idx
        rows = stored_values_f32(W[idx], dtype).astype(np.float64)
        H[q] = rows.sum(axis=0) + rng.normal(0.0, sd, size=d)
    return _cast(H, dtype), planted


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic head shaped like a model from the paper's Section 4."""
    cid: int
    name: str
    V: int
    d: int
    dtype: int
    Q: int
    k: tuple
    ef: tuple
    M: int
    efC: int
    B: tuple = (1,)
    hub_frac: float = 0.0

    @property
    def M0(self) -> int:
        return 2 * self.M

    @property
    def seed_w(self) -> int:
        return 1000 + self.cid

    @property
    def seed_q(self) -> int:
        return 2000 + self.cid

    @property
    def seed_hub(self) -> int:
        return 3000 + self.cid

    @property
    def seed_levels(self) -> int:
        return 4000 + self.cid

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == F32 else 2

    def make_w(self) -> np.ndarray:
        return make_w(self.V, self.d, self.dtype, self.seed_w, self.hub_frac,
                      seed_hub=self.seed_hub)

    def make_queries(self, W: np.ndarray, Q: int | None = None):
        return make_queries(W, self.dtype, self.Q if Q is None else Q, self.seed_q)


WORKLOADS = {
    "tiny": Workload(1, "tiny-32k-d256-f32", 32768, 256, F32, 256, (50,), (64,), 16, 100),
    "qwen3-0.6b": Workload(2, "qwen3-0.6b-head-151936x1024-bf16", 151936, 1024, BF16, 1024,
                           (50,), (64, 128, 256), 32, 200),
    "llama3.2-1b": Workload(3, "llama3.2-1b-head-128256x2048-bf16", 128256, 2048, BF16, 1024,
                            (50,), (128,), 32, 200),
    "gemma3-270m": Workload(4, "gemma3-270m-head-262144x640-bf16", 262144, 640, BF16, 2048,
                            (20, 50, 100), (128,), 32, 200, hub_frac=0.10),
    "llama3.2-3b": Workload(5, "llama3.2-3b-head-128256x3072-bf16", 128256, 3072, BF16, 1024,
                            (50,), (128,), 32, 200, B=(1, 4, 16, 64)),
}
