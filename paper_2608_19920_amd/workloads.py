"""Seeded synthetic inputs for the H2O chunk step.

This module only draws random numbers and stores them in the layouts the
library and the float64 oracle both consume. It holds none of the method's
arithmetic (no attention, no score update, no selection).

Layouts (all C-contiguous, matching the paper's buffer statement in
Sec. "Sparse Attention. Key-Value Caching": keys/values are (B, H_k, N_C, d_h),
token positions are (B, H_k, N_C)):

    q        [B, Hq,  T, d]
    k_cache  [B, Hkv, M, d]      v_cache  [B, Hkv, M, d]
    k_new    [B, Hkv, T, d]      v_new    [B, Hkv, T, d]
    scores   [B, Hkv, M]  float32 (prior H2O scores)
    token_pos[B, Hkv, M]  int32

For bf16 workloads every tensor is drawn in float32 and rounded to bf16 with
round-to-nearest-even; the array handed to the oracle is the exact float32
upcast of those bf16 values, so both sides see identical numbers.

Draw order from ``numpy.random.Generator(PCG64(seed))``: q, k_cache, v_cache,
k_new, v_new, heavy-hitter slot sets, prior scores, ages; decode workloads then
draw (q, k_new, v_new) per step.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    d: int
    M: int
    T: int
    dtype: str            # "f32" or "bf16"
    heavy_frac: float     # fraction of cache slots whose key is scaled by heavy_mult
    heavy_mult: float = 4.0
    age_decay: Optional[float] = None   # prior *= exp(-age/age_decay), ages ~ U{0..age_max-1}
    age_max: int = 65536
    steps: int = 1        # decode trajectories run `steps` chunk steps of length T

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def k(self) -> int:
        return self.T

    def describe(self) -> str:
        return (f"{self.name}: B{self.B} Hq{self.Hq} Hkv{self.Hkv} d{self.d} "
                f"M{self.M} T{self.T} {self.dtype}"
                + (f" x{self.steps} steps" if self.steps > 1 else ""))


# The five synthetic GQA shapes the path is checked and measured on.
WORKLOADS: Dict[str, Workload] = {
    "tiny_f32": Workload("tiny_f32", B=1, Hq=4, Hkv=2, d=64, M=256, T=64,
                         dtype="f32", heavy_frac=0.0),
    "decode_bf16": Workload("decode_bf16", B=8, Hq=32, Hkv=8, d=64, M=4096, T=1,
                            dtype="bf16", heavy_frac=0.02, steps=16),
    "prefill_bf16": Workload("prefill_bf16", B=1, Hq=32, Hkv=8, d=128, M=8192,
                             T=1024, dtype="bf16", heavy_frac=0.02),
    "longcache_bf16": Workload("longcache_bf16", B=4, Hq=32, Hkv=8, d=128,
                               M=32768, T=512, dtype="bf16", heavy_frac=0.01,
                               age_decay=8192.0),
    "gqa7_bf16": Workload("gqa7_bf16", B=2, Hq=28, Hkv=4, d=128, M=16384,
                          T=2048, dtype="bf16", heavy_frac=0.02),
}


def custom(name="custom", *, B, Hq, Hkv, d, M, T, dtype="bf16", heavy_frac=0.0,
           age_decay=None, steps=1) -> Workload:
    return Workload(name, B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=T, dtype=dtype,
                    heavy_frac=heavy_frac, age_decay=age_decay, steps=steps)


# ---------------------------------------------------------------- bf16 storage
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


def _normal(rng, shape, dtype):
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if dtype == "bf16":
        return bf16_bits_to_f32(f32_to_bf16_bits(x))
    return x


def _apply_heavy(rng, k_cache, frac, mult):
    """Scale the keys of exactly round(frac*M) distinct slots per (b, kv-head)."""
    B, H, M, _ = k_cache.shape
    n = int(round(frac * M))
    if n == 0:
        return np.zeros((B, H, 0), np.int64)
    sets = np.empty((B, H, n), np.int64)
    for b in range(B):
        for h in range(H):
            idx = rng.choice(M, size=n, replace=False)
            sets[b, h] = idx
            k_cache[b, h, idx] *= np.float32(mult)   # power of two: exact in bf16
    return sets


def make_inputs(w: Workload, seed: int = 0) -> Dict[str, np.ndarray]:
    """Draw one chunk step's inputs (plus per-step decode draws when steps > 1).

    Returns float32 arrays holding exactly representable values for ``w.dtype``
    (for bf16 they are upcasts of bf16 values), the prior scores, token
    positions, ``pos0`` (position of the chunk's first token) and ``scale``.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    B, Hq, Hkv, d, M, T = w.B, w.Hq, w.Hkv, w.d, w.M, w.T
    out: Dict[str, np.ndarray] = {}
    out["q"] = _normal(rng, (B, Hq, T, d), w.dtype)
    kc = rng.standard_normal(size=(B, Hkv, M, d), dtype=np.float32)
    out["v_cache"] = _normal(rng, (B, Hkv, M, d), w.dtype)
    out["k_new"] = _normal(rng, (B, Hkv, T, d), w.dtype)
    out["v_new"] = _normal(rng, (B, Hkv, T, d), w.dtype)
    out["heavy"] = _apply_heavy(rng, kc, w.heavy_frac, w.heavy_mult)
    if w.dtype == "bf16":
        kc = bf16_bits_to_f32(f32_to_bf16_bits(kc))
    out["k_cache"] = kc
    prior = rng.standard_exponential(size=(B, Hkv, M), dtype=np.float32)
    if w.age_decay is not None:
        ages = rng.integers(0, w.age_max, size=(B, Hkv, M))
        prior = (prior.astype(np.float64) * np.exp(-ages / w.age_decay)).astype(np.float32)
        pos0 = w.age_max
        token_pos = (pos0 - 1 - ages).astype(np.int32)
    else:
        pos0 = M
        token_pos = np.broadcast_to(np.arange(M, dtype=np.int32), (B, Hkv, M)).copy()
    out["scores"] = prior
    out["token_pos"] = token_pos
    out["pos0"] = np.int32(pos0)
    out["scale"] = np.float32(1.0 / math.sqrt(d))
    if w.steps > 1:
        # step 0 uses the first draw above; steps 1.. draw fresh (q, k_new, v_new)
        qs, kn, vn = [out["q"]], [out["k_new"]], [out["v_new"]]
        for _ in range(w.steps - 1):
            qs.append(_normal(rng, (B, Hq, T, d), w.dtype))
            kn.append(_normal(rng, (B, Hkv, T, d), w.dtype))
            vn.append(_normal(rng, (B, Hkv, T, d), w.dtype))
        out["q_steps"] = np.stack(qs)
        out["k_new_steps"] = np.stack(kn)
        out["v_new_steps"] = np.stack(vn)
    return out
