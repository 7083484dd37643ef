"""Helpers for GPU parity tests: move seeded inputs to the device, run the
library through its binding, bring results back as float64 numpy."""
from __future__ import annotations

import sys

import numpy as np
import torch

from paper_2608_19920_amd import h2o as H

DEV = "cuda"
TDT = {"f32": torch.float32, "bf16": torch.bfloat16}
TOL = {"f32": 1e-5, "bf16": 2e-2}


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
