"""GPU parity of the paper's step order, insert then attend (Sec. "Discussion:
SDPA Kernels for Sparse Attention"): h2o_sdpa_cache (attention over the cache
slots with the token-position mask) and h2o_chunk_step_insert_first, through
the C ABI, against the float64 oracle.

Tolerances as for the attend-then-evict path: normwise relative error per
slice <= 1e-5 (float32) and <= 2e-2 (bf16). The eviction runs on the input
scores before the chunk, so it is bit-exact; the insert is bitwise; the
accumulated scores are bit-equal to the oracle's float32 addition applied to
the GPU's own summed weights.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_19920_amd import h2o as H
from paper_2608_19920_amd import workloads as W
import _gpu as U
from _gpu import say

pytestmark = pytest.mark.gpu

SHAPES = [  # B, Hq, Hkv, d, M, T, dtype, forced path (-1 automatic)
    (1, 4, 2, 64, 256, 64, "f32", -1),
    (2, 8, 2, 128, 700, 64, "bf16", -1),       # MFMA prefill kernels
    (1, 8, 2, 128, 300, 70, "bf16", -1),
    (1, 28, 4, 128, 257, 40, "bf16", -1),
    (2, 8, 2, 64, 333, 17, "bf16", 0),         # generic kernels, bf16
    (8, 32, 8, 64, 4096, 1, "bf16", -1),       # decode kernels
    (2, 8, 4, 128, 1025, 1, "bf16", -1),
    (1, 4, 1, 64, 37, 1, "bf16", -1),
    (2, 4, 2, 64, 500, 1, "f32", -1),
    (1, 8, 2, 128, 129, 1, "bf16", 1),         # MFMA kernels with one query
    (2, 8, 2, 128, 2048, 96, "bf16", -1),      # few chunk tokens among the slots: the lse
    (1, 8, 2, 64, 1500, 64, "bf16", -1),       #   pass skips the mask on tiles a wave sees
    (1, 8, 1, 128, 4096, 2048, "bf16", -1),    # grids of whole rounds: 8-wave blocks
]


@pytest.fixture
def force(request):
    yield
    H.h2o_debug_force_path(-1)


def _positions(B, Hkv, M, T, rng, kind):
    """Token positions and pos0. 'state': slots older than the chunk, the
    chunk at pos0+i in T scattered slots; 'wild': arbitrary positions around
    the chunk (some later than every query, some rows of (0, 0) see none)."""
    pos0 = 70000
    if kind == "state":
        tp = rng.integers(0, pos0, size=(B, Hkv, M)).astype(np.int32)
        for b in range(B):
            for h in range(Hkv):
                e = np.sort(rng.choice(M, T, replace=False))
                tp[b, h, e] = pos0 + np.arange(T)
    else:
        tp = rng.integers(pos0 - 40, pos0 + T + 5, size=(B, Hkv, M)).astype(np.int32)
        tp[0, 0] = np.maximum(tp[0, 0], pos0 + T // 2)   # early queries of head (0,0) see nothing
    return tp, pos0


def _check(dt, got, ref, extra=""):
    go, gl, gw = got
    o, l, w = ref
    dead = np.isneginf(l)
    np.testing.assert_array_equal(np.isneginf(gl), dead, err_msg="rows that see no slot")
    assert not np.any(go[dead]), "a row that sees no slot must output 0"
    U.check(dt, out=(go, o), lse=(gl, l), wsum=(gw, w), extra=extra)


@pytest.mark.parametrize("kind", ["state", "wild"])
@pytest.mark.parametrize("shape", SHAPES)
def test_sdpa_cache(shape, kind, force):
    B, Hq, Hkv, d, M, T, dt, path = shape
    H.h2o_debug_force_path(path)
    wl = W.custom("cache", B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=T, dtype=dt, heavy_frac=0.02)
    say(f"sdpa_cache {wl.describe()} {kind} path {path}")
    x = W.make_inputs(wl, seed=M + T)
    tp, pos0 = _positions(B, Hkv, M, T, np.random.default_rng(M * T), kind)
    tdt = U.TDT[dt]
    q, kc, vc = (U.to_dev(x[n], tdt) for n in ("q", "k_cache", "v_cache"))
    bufs = H.alloc_step(B, Hq, Hkv, T, M, d, tdt, insert_first=True)
    H.h2o_sdpa_cache(q, kc, vc, U.to_dev(tp, torch.int32), bufs["out"], bufs["lse"],
                     bufs["wsum"], bufs["workspace"], pos0, float(x["scale"]))
    torch.cuda.synchronize()
    ref = oracle.sdpa_cache(x["q"], x["k_cache"], x["v_cache"], tp, pos0, x["scale"])
    _check(dt, tuple(U.to_np(bufs[n]) for n in ("out", "lse", "wsum")), ref)


STEP_SHAPES = [  # B, Hq, Hkv, d, M, T, dtype
    (8, 32, 8, 64, 4096, 1, "bf16"),
    (2, 8, 2, 64, 5000, 1, "bf16"),     # T = 1, more slots than the fused kernel prefetches
    (1, 8, 2, 128, 4133, 1, "bf16"),    # T = 1, d = 128, ragged last step
    (2, 8, 2, 128, 700, 64, "bf16"),
    (1, 8, 2, 128, 2048, 96, "bf16"),   # T * 16 <= M: tiles without a mask in the lse pass
    (1, 4, 2, 64, 256, 64, "f32"),
    (2, 4, 2, 64, 300, 1, "f32"),
]


@pytest.mark.parametrize("policy", ["h2o", "h2o_norm", "h2o_orig"])
@pytest.mark.parametrize("shape", STEP_SHAPES)
def test_step_insert_first(shape, policy):
    B, Hq, Hkv, d, M, T, dt = shape
    wl = W.custom("insfirst", B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=T, dtype=dt, heavy_frac=0.02,
                  age_decay=8192.0)
    say(f"insert-first step {policy} {wl.describe()}")
    x = W.make_inputs(wl, seed=23)
    tdt = U.TDT[dt]
    st = U.device_state(x, dt)
    q, kn, vn = (U.to_dev(x[n], tdt) for n in ("q", "k_new", "v_new"))
    bufs = H.alloc_step(B, Hq, Hkv, T, M, d, tdt, policy=policy, insert_first=True)
    pos0 = int(x["pos0"])
    H.h2o_chunk_step_insert_first(q, st["k_cache"], st["v_cache"], st["scores"], st["token_pos"],
                                  kn, vn, bufs["out"], bufs["lse"], bufs["wsum"],
                                  bufs["evict_idx"], bufs["workspace"], pos0, float(x["scale"]),
                                  policy)
    torch.cuda.synchronize()
    r = oracle.h2o_step_insert_first(x["k_cache"], x["v_cache"], x["scores"], x["token_pos"],
                                     x["q"], x["k_new"], x["v_new"], pos0, x["scale"], policy)
    # eviction on the scores before the chunk, and the insert: exact
    np.testing.assert_array_equal(bufs["evict_idx"].cpu().numpy(), r["evict_idx"])
    for n in ("k_cache", "v_cache", "token_pos"):
        np.testing.assert_array_equal(U.to_np(st[n]), np.asarray(r[n], U.to_np(st[n]).dtype),
                                      err_msg=n)
    g = tuple(U.to_np(bufs[n]) for n in ("out", "lse", "wsum"))
    _check(dt, g, (r["out"], r["lse"], r["wsum"]), extra=policy)
    # scores: one float32 addition of the GPU's own summed weights
    np.testing.assert_array_equal(st["scores"].cpu().numpy(),
                                  oracle.accumulate_scores(r["scores_inserted"], g[2]))
    U.check(dt, scores=(U.to_np(st["scores"]), r["scores"]), extra="scores")
    # every query sees its own key: the weights of a head sum to T*G
    np.testing.assert_allclose(g[2].sum(-1), T * (Hq // Hkv), rtol=2e-3)


@pytest.mark.parametrize("name,nheads", [("prefill_bf16", 2), ("longcache_bf16", 1),
                                         ("gqa7_bf16", 1), ("decode_bf16", 3)])
def test_full_size_insert_first_sampled_heads(name, nheads):
    """The insert-first step at a full workload size; the oracle recomputes a
    sample of (b, kv-head) pairs."""
    wl = W.WORKLOADS[name]
    say(f"full-size insert-first {wl.describe()}")
    x = W.make_inputs(wl, seed=1)
    st = U.device_state(x, "bf16")
    tdt = torch.bfloat16
    q0 = x["q_steps"][0] if "q_steps" in x else x["q"]
    kn0 = x["k_new_steps"][0] if "k_new_steps" in x else x["k_new"]
    vn0 = x["v_new_steps"][0] if "v_new_steps" in x else x["v_new"]
    q, kn, vn = (U.to_dev(a, tdt) for a in (q0, kn0, vn0))
    bufs = H.alloc_step(wl.B, wl.Hq, wl.Hkv, wl.T, wl.M, wl.d, tdt, insert_first=True)
    pos0 = int(x["pos0"])
    H.h2o_chunk_step_insert_first(q, st["k_cache"], st["v_cache"], st["scores"], st["token_pos"],
                                  kn, vn, bufs["out"], bufs["lse"], bufs["wsum"],
                                  bufs["evict_idx"], bufs["workspace"], pos0, float(x["scale"]))
    torch.cuda.synchronize()
    idx = bufs["evict_idx"].cpu().numpy()
    np.testing.assert_array_equal(idx, oracle.bottomk(x["scores"], wl.T))
    rng = np.random.default_rng(0)
    pairs = [(b, h) for b in range(wl.B) for h in range(wl.Hkv)]
    heads = [pairs[i] for i in rng.choice(len(pairs), size=nheads, replace=False)]
    kc, vc = U.to_np(st["k_cache"]), U.to_np(st["v_cache"])
    tp = st["token_pos"].cpu().numpy()
    for b, h in heads:
        np.testing.assert_array_equal(kc[b, h, idx[b, h]], kn0[b, h])
        np.testing.assert_array_equal(tp[b, h, idx[b, h]], pos0 + np.arange(wl.T))
    o, l, w = oracle.sdpa_cache(q0, kc, vc, tp, pos0, x["scale"], heads=heads)
    G = wl.G
    hq = [(b, h * G + g) for b, h in heads for g in range(G)]
    sel = lambda a, hs: np.stack([a[b, h] for b, h in hs])
    go, gl, gw = (U.to_np(bufs[n]) for n in ("out", "lse", "wsum"))
    _check("bf16", (sel(go, hq), sel(gl, hq), sel(gw, heads)),
           (sel(o, hq), sel(l, hq), sel(w, heads)), extra=f"heads {heads}")


@pytest.mark.parametrize("shape", [(8, 32, 8, 64, 4096, 1, "bf16"), (2, 8, 2, 128, 700, 64, "bf16")])
def test_insert_first_graph_replays_match_eager(shape):
    """The insert-first step captured in a HIP graph and replayed three times
    (the state advancing each time, eager steps and synchronisation between
    the replays) gives the same bits as the same steps run eagerly."""
    B, Hq, Hkv, d, M, T, dt = shape
    wl = W.custom("ifgraph", B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=T, dtype=dt, heavy_frac=0.02)
    say(f"insert-first graph replay {wl.describe()}")
    x = W.make_inputs(wl, seed=9)
    tdt = U.TDT[dt]
    q, kn, vn = (U.to_dev(x[n], tdt) for n in ("q", "k_new", "v_new"))
    pos0, scale = int(x["pos0"]), float(x["scale"])
    sg, se = U.device_state(x, dt), U.device_state(x, dt)
    bg = H.alloc_step(B, Hq, Hkv, T, M, d, tdt, insert_first=True)
    be = H.alloc_step(B, Hq, Hkv, T, M, d, tdt, insert_first=True)

    def run(st, b):
        H.h2o_chunk_step_insert_first(q, st["k_cache"], st["v_cache"], st["scores"],
                                      st["token_pos"], kn, vn, b["out"], b["lse"], b["wsum"],
                                      b["evict_idx"], b["workspace"], pos0, scale)

    stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        run(sg, bg)
    torch.cuda.synchronize()          # capture does not run the step
    for r in range(3):
        graph.replay()
        run(se, be)
        torch.cuda.synchronize()
        for n in ("out", "lse", "wsum", "evict_idx"):
            np.testing.assert_array_equal(U.to_np(bg[n]), U.to_np(be[n]), err_msg=f"replay {r} {n}")
        for n in ("k_cache", "v_cache", "scores", "token_pos"):
            np.testing.assert_array_equal(U.to_np(sg[n]), U.to_np(se[n]), err_msg=f"replay {r} {n}")
