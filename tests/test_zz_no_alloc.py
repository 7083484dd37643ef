"""h2o_chunk_step_noalloc - the chunk step with the library's own scratch
array in place of a caller's workspace - against h2o_chunk_step on the same
inputs, through the C ABI: two calls in a row, the second on a smaller
shape, every output and the whole cache state bit for bit (the two entry
points run the same kernels)."""
import numpy as np
import pytest
import torch

from paper_2608_19920_amd import h2o as H
from paper_2608_19920_amd import workloads as W
import _gpu as U
from _gpu import say

pytestmark = pytest.mark.gpu

CASES = [  # (first call, second call on a smaller shape): B, Hq, Hkv, d, M, T, dtype
    [(8, 32, 8, 64, 4096, 1, "bf16"), (2, 8, 2, 64, 700, 1, "bf16")],
    [(1, 8, 2, 128, 300, 70, "bf16"), (1, 4, 2, 64, 256, 64, "f32")],
]


def _run(shape, noalloc, seed):
    B, Hq, Hkv, d, M, T, dt = shape
    wl = W.custom("noalloc", B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=T, dtype=dt, heavy_frac=0.02)
    x = W.make_inputs(wl, seed=seed)
    tdt = U.TDT[dt]
    q, kn, vn = (U.to_dev(x[n], tdt) for n in ("q", "k_new", "v_new"))
    st = U.device_state(x, dt)
    b = H.alloc_step(B, Hq, Hkv, T, M, d, tdt)
    pos0, scale = int(x["pos0"]), float(x["scale"])
    args = (q, st["k_cache"], st["v_cache"], st["scores"], st["token_pos"], kn, vn, b["out"],
            b["lse"], b["wsum"], b["evict_idx"])
    if noalloc:
        H.h2o_chunk_step_noalloc(*args, pos0, scale)
    else:
        H.h2o_chunk_step(*args, b["workspace"], pos0, scale)
    torch.cuda.synchronize()
    return {**{n: U.to_np(b[n]) for n in ("out", "lse", "wsum", "evict_idx")},
            **{n: U.to_np(st[n]) for n in ("k_cache", "v_cache", "scores", "token_pos")}}


@pytest.mark.parametrize("case", CASES, ids=["decode", "prefill"])
def test_noalloc_equals_chunk_step(case):
    assert H.h2o_noalloc_scratch_bytes() == 32 << 20
    for i, shape in enumerate(case):
        say(f"noalloc call {i}: {shape}")
        got = _run(shape, True, seed=40 + i)
        ref = _run(shape, False, seed=40 + i)
        for n in ref:
            np.testing.assert_array_equal(got[n], ref[n], err_msg=f"call {i}: {n}")
