"""GPU parity over seeded random shapes: h2o_sdpa_chunk (chunk mode) and
h2o_sdpa_cache (cache mode, token-position mask) against the float64 oracle,
on every kernel path a shape can take (automatic, generic VALU, MFMA, and the
T = 1 decode kernels), GQA group sizes 1 to 8, cache lengths from 0 to a few
thousand slots with ragged tails, chunk lengths from 1 to 160, bf16 and
float32. Tolerances as in test_gpu_parity (2e-2 bf16, 1e-5 float32): out
and lse normwise per (b, head) slice, wsum element by element.
The whole chunk step on random shapes: the fused call bit-equal to the three
separate calls (attention, accumulate, evict and insert); the insert-first
step with each score policy, eviction and insert exact against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_19920_amd import h2o as H
from paper_2608_19920_amd import workloads as W
import _gpu as U
from _gpu import say
from test_gpu_insert_first import _positions

pytestmark = pytest.mark.gpu

N_CASES = 48


def _case(i):
    rng = np.random.default_rng(9000 + i)
    G = int(rng.choice([1, 2, 3, 4, 7, 8]))
    Hkv = int(rng.integers(1, 4))
    B = int(rng.integers(1, 3))
    d = int(rng.choice([64, 128]))
    M = int(rng.choice([0, 1, 31, 33, int(rng.integers(2, 2500))]))
    T = int(rng.choice([1, 1, int(rng.integers(2, 40)), int(rng.integers(40, 160))]))
    dt = str(rng.choice(["bf16", "bf16", "f32"]))
    paths = [-1, 0] + ([1] if dt == "bf16" else []) + ([2] if T == 1 and dt == "bf16" else [])
    path = int(rng.choice(paths))
    mode = str(rng.choice(["chunk", "cache"]))
    if mode == "cache" and T > M:
        mode = "chunk"
    kind = str(rng.choice(["state", "wild"]))
    return dict(B=B, G=G, Hkv=Hkv, d=d, M=M, T=T, dt=dt, path=path, mode=mode, kind=kind)


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_shape(i):
    c = _case(i)
    B, G, Hkv, d, M, T, dt = (c[k] for k in ("B", "G", "Hkv", "d", "M", "T", "dt"))
    say(f"sweep case {i}: {c}")
    H.h2o_debug_force_path(c["path"])
    try:
        wl = W.custom("sweep", B=B, Hq=G * Hkv, Hkv=Hkv, d=d, M=M, T=T, dtype=dt,
                      heavy_frac=0.02)
        x = W.make_inputs(wl, seed=1000 + i)
        if c["mode"] == "chunk":
            res = U.run_sdpa(x["q"], x["k_cache"], x["v_cache"], x["k_new"], x["v_new"],
                             x["scale"], dt)
            ref = oracle.sdpa_chunk(x["q"], x["k_cache"], x["v_cache"], x["k_new"],
                                    x["v_new"], x["scale"])
        else:
            tp, pos0 = _positions(B, Hkv, M, T, np.random.default_rng(i), c["kind"])
            tdt = U.TDT[dt]
            q, kc, vc = (U.to_dev(x[k], tdt) for k in ("q", "k_cache", "v_cache"))
            bufs = H.alloc_step(B, G * Hkv, Hkv, T, M, d, tdt, insert_first=True)
            H.h2o_sdpa_cache(q, kc, vc, U.to_dev(tp, torch.int32), bufs["out"], bufs["lse"],
                             bufs["wsum"], bufs["workspace"], pos0, float(x["scale"]))
            torch.cuda.synchronize()
            res = tuple(U.to_np(bufs[k]) for k in ("out", "lse", "wsum"))
            ref = oracle.sdpa_cache(x["q"], x["k_cache"], x["v_cache"], tp, pos0, x["scale"])
    finally:
        H.h2o_debug_force_path(-1)
    o, l, w = ref
    go, gl, gw = res
    # rows that see no key have lse -inf on both sides (checked in U.check)
    U.check(dt, out=(go, o), lse=(gl, l), wsum=(gw, w))


N_STEP_CASES = 24


def _step_case(i):
    rng = np.random.default_rng(7000 + i)
    G = int(rng.choice([1, 2, 4, 7, 8]))
    Hkv = int(rng.integers(1, 4))
    B = int(rng.integers(1, 3))
    d = int(rng.choice([64, 128]))
    T = int(rng.choice([1, 1, 1, int(rng.integers(2, 100))]))
    M = int(rng.integers(T, T + 3000))
    dt = str(rng.choice(["bf16", "bf16", "f32"]))
    return dict(B=B, G=G, Hkv=Hkv, d=d, M=M, T=T, dt=dt)


@pytest.mark.parametrize("i", range(N_STEP_CASES))
def test_random_step_fused_equals_calls(i):
    """h2o_chunk_step gives the same bits as h2o_sdpa_chunk + h2o_accumulate_scores
    + h2o_evict_insert on a random shape, and its attention matches the oracle."""
    c = _step_case(i)
    B, G, Hkv, d, M, T, dt = (c[k] for k in ("B", "G", "Hkv", "d", "M", "T", "dt"))
    say(f"step sweep case {i}: {c}")
    wl = W.custom("stepsweep", B=B, Hq=G * Hkv, Hkv=Hkv, d=d, M=M, T=T, dtype=dt,
                  heavy_frac=0.02)
    x = W.make_inputs(wl, seed=2000 + i)
    tdt = U.TDT[dt]
    q, kn, vn = (U.to_dev(x[n], tdt) for n in ("q", "k_new", "v_new"))
    res = []
    for fused in (False, True):
        st = U.device_state(x, dt)
        bufs = H.alloc_step(B, G * Hkv, Hkv, T, M, d, tdt)
        H.step(st, q, kn, vn, bufs, int(x["pos0"]), float(x["scale"]), fused=fused)
        torch.cuda.synchronize()
        res.append({**{n: U.to_np(bufs[n]) for n in ("out", "lse", "wsum", "evict_idx")},
                    **{n: U.to_np(st[n]) for n in ("k_cache", "v_cache", "scores", "token_pos")}})
    for n in res[0]:
        np.testing.assert_array_equal(res[1][n], res[0][n], err_msg=n)
    o, l, w = oracle.sdpa_chunk(x["q"], x["k_cache"], x["v_cache"], x["k_new"], x["v_new"],
                                x["scale"])
    U.check(dt, out=(res[1]["out"], o), lse=(res[1]["lse"], l), wsum=(res[1]["wsum"], w),
            scores=(oracle.accumulate_scores(x["scores"], res[1]["wsum"]),
                    oracle.accumulate_scores(x["scores"], w)))


N_INS_CASES = 18


@pytest.mark.parametrize("i", range(N_INS_CASES))
def test_random_step_insert_first(i):
    """h2o_chunk_step_insert_first on a random shape with a random policy:
    eviction and insert exact against the oracle, attention within tolerance,
    scores one float32 addition of the GPU's own summed weights."""
    c = _step_case(100 + i)
    B, G, Hkv, d, M, T, dt = (c[k] for k in ("B", "G", "Hkv", "d", "M", "T", "dt"))
    policy = ("h2o", "h2o_norm", "h2o_orig")[i % 3]
    say(f"insert-first sweep case {i}: {c} {policy}")
    wl = W.custom("inssweep", B=B, Hq=G * Hkv, Hkv=Hkv, d=d, M=M, T=T, dtype=dt,
                  heavy_frac=0.02, age_decay=8192.0)
    x = W.make_inputs(wl, seed=3000 + i)
    tdt = U.TDT[dt]
    st = U.device_state(x, dt)
    q, kn, vn = (U.to_dev(x[n], tdt) for n in ("q", "k_new", "v_new"))
    bufs = H.alloc_step(B, G * Hkv, Hkv, T, M, d, tdt, policy=policy, insert_first=True)
    pos0 = int(x["pos0"])
    H.h2o_chunk_step_insert_first(q, st["k_cache"], st["v_cache"], st["scores"], st["token_pos"],
                                  kn, vn, bufs["out"], bufs["lse"], bufs["wsum"],
                                  bufs["evict_idx"], bufs["workspace"], pos0, float(x["scale"]),
                                  policy)
    torch.cuda.synchronize()
    r = oracle.h2o_step_insert_first(x["k_cache"], x["v_cache"], x["scores"], x["token_pos"],
                                     x["q"], x["k_new"], x["v_new"], pos0, x["scale"], policy)
    np.testing.assert_array_equal(bufs["evict_idx"].cpu().numpy(), r["evict_idx"])
    for n in ("k_cache", "v_cache", "token_pos"):
        np.testing.assert_array_equal(U.to_np(st[n]), np.asarray(r[n], U.to_np(st[n]).dtype),
                                      err_msg=n)
    g = tuple(U.to_np(bufs[n]) for n in ("out", "lse", "wsum"))
    U.check(dt, out=(g[0], r["out"]), lse=(g[1], r["lse"]), wsum=(g[2], r["wsum"]),
            scores=(U.to_np(st["scores"]), r["scores"]))
    np.testing.assert_array_equal(st["scores"].cpu().numpy(),
                                  oracle.accumulate_scores(r["scores_inserted"], g[2]))
