"""Helpers for GPU parity tests: move seeded inputs to the device, run the
library through its binding, bring results back as float64 numpy."""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import elem_err, rel_err
from paper_2608_19920_amd import h2o as H

DEV = "cuda"
TDT = {"f32": torch.float32, "bf16": torch.bfloat16}
# The stated tolerances: out and lse normwise per slice, the summed weights
# and the scores element by element (see check()).
TOL = {"f32": 1e-5, "bf16": 2e-2}
# Bound on the relative error of an accumulated float32 score on the bf16
# path, the premise of the eviction band (oracle.eviction_agreement): the
# products of bf16 values are exact in float32, so a logit's error is that of
# summing d exact products, at most d * 2^-24 * scale * sum_d |q k| (about
# 2e-4 for d = 128 with keys scaled x4); a weight exp(s - lambda) carries the
# error of s and of lambda, and a sum of such non-negative weights (and the
# addition to a non-negative prior score) is no worse than its worst term.
SEL_TOL = 1e-3


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(a: np.ndarray, dtype) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV).to(dtype).contiguous()


def to_np(t: torch.Tensor) -> np.ndarray:
    if t.dtype in (torch.bfloat16, torch.float16):
        t = t.float()
    return t.detach().cpu().numpy().astype(np.float64) if t.is_floating_point() else \
        t.detach().cpu().numpy()


def device_state(x, dtype):
    tdt = TDT[dtype]
    return dict(k_cache=to_dev(x["k_cache"], tdt), v_cache=to_dev(x["v_cache"], tdt),
                scores=to_dev(x["scores"], torch.float32),
                token_pos=to_dev(x["token_pos"], torch.int32))


def run_sdpa(q, kc, vc, kn, vn, scale, dtype):
    """Runs h2o_sdpa_chunk on numpy inputs; returns (out, lse, wsum) float64."""
    tdt = TDT[dtype]
    B, Hq, T, d = q.shape
    Hkv, M = kc.shape[1], kc.shape[2]
    bufs = H.alloc_step(B, Hq, Hkv, T, M, d, tdt)
    H.h2o_sdpa_chunk(to_dev(q, tdt), to_dev(kc, tdt), to_dev(vc, tdt), to_dev(kn, tdt),
                     to_dev(vn, tdt), bufs["out"], bufs["lse"], bufs["wsum"], bufs["workspace"],
                     float(scale))
    torch.cuda.synchronize()
    return to_np(bufs["out"]), to_np(bufs["lse"]), to_np(bufs["wsum"])


def gpu_bottomk(scores_f32: np.ndarray, k: int) -> np.ndarray:
    s = to_dev(scores_f32.astype(np.float32), torch.float32)
    idx = torch.empty(*scores_f32.shape[:-1], k, dtype=torch.int32, device=DEV)
    H.h2o_bottomk(s, k, idx)
    torch.cuda.synchronize()
    return idx.cpu().numpy()


def check(dtype, out=None, lse=None, wsum=None, scores=None, extra=""):
    """The parity gates, each argument a (gpu, oracle) pair.

    out and lse: normwise relative error per slice (per (b, query head)),
    because an output element can cancel to nearly zero, where an elementwise
    relative error means nothing; rows that see no key (lse -inf) must agree
    on that. wsum and scores: element by element (oracle.elem_err), because
    the summed weight and the score are defined per key and every term of
    them is non-negative: a wrong tile of columns cannot hide behind the
    heavy hitters that dominate a row's norm. Returns the errors."""
    tol = TOL[dtype]
    errs = {}
    if out is not None:
        g, r = out
        assert np.isfinite(g).all(), "out not finite"
        errs["out"] = rel_err(g, r, (-2, -1))
    if lse is not None:
        g, r = lse
        seen = np.isfinite(r)
        assert np.array_equal(np.isfinite(g), seen), "rows that see no key differ"
        errs["lse"] = rel_err(np.where(seen, g, 0.0), np.where(seen, r, 0.0), (-1,))
    for name, pair in (("wsum", wsum), ("scores", scores)):
        if pair is not None:
            g, r = pair
            assert np.isfinite(g).all(), f"{name} not finite"
            errs[name] = elem_err(g, r, (-1,))
            errs[name + " (normwise)"] = rel_err(g, r, (-1,))
    say(f"  {extra} " + " ".join(f"{k} {v:.2e}" for k, v in errs.items()) + f" (tol {tol})")
    for k, v in errs.items():
        assert v <= tol, f"{k} error {v:.3e} above {tol}"
    return errs
