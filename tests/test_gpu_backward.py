"""GPU parity of the fine-tuning kernels: the backward of the chunk attention
(h2o_sdpa_chunk_backward, chunk and cache mode) and the delta encoding of the
KV recurrence (h2o_kv_gather / h2o_kv_scatter), through the C ABI, against
the float64 oracle.

Gradients: normwise relative error per (b, head) slice <= 1e-5 (float32) and
<= 2e-2 (bf16, gradients stored in bf16). The forward's lse comes from the
library's own forward, as in training. bf16 runs on the MFMA kernels, and
again on the VALU kernels (path 0). Gather and scatter are bitwise.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import rel_err
from paper_2608_19920_amd import h2o as H
from paper_2608_19920_amd import workloads as W
import _gpu as U
from _gpu import say

pytestmark = pytest.mark.gpu

SHAPES = [  # B, Hq, Hkv, d, M, T, dtype
    (1, 4, 2, 64, 256, 64, "f32"),
    (2, 4, 2, 64, 100, 1, "f32"),
    (1, 8, 2, 128, 300, 70, "bf16"),        # ragged row and key blocks
    (2, 8, 2, 64, 333, 17, "bf16"),
    (1, 28, 4, 128, 257, 40, "bf16"),       # GQA 7
    (1, 4, 1, 128, 0, 20, "bf16"),          # empty cache
    (8, 32, 8, 64, 512, 1, "bf16"),         # one query, heavy hitters
    (1, 8, 2, 128, 1000, 128, "bf16"),
    (2, 32, 8, 128, 700, 64, "bf16"),       # 16 heads: XCD-grouped block order
    (1, 32, 8, 128, 2048, 256, "bf16"),     # rows passes in 8-wave blocks (whole rounds)
]
# bf16 shapes run on the MFMA kernels (-1) and on the VALU kernels (0);
# float32 has only the VALU kernels
CASES = [(sh, p) for sh in SHAPES for p in ((-1, 0) if sh[-1] == "bf16" else (-1,))]


@pytest.fixture
def force(request):
    yield
    H.h2o_debug_force_path(-1)


def _grads_check(dt, got, ref, names):
    tol = U.TOL[dt]
    for g, r, n in zip(got, ref, names):
        if r is None or r.size == 0:
            continue
        e = rel_err(g, r, axes=(-2, -1))
        say(f"  {n}: err {e:.2e} (tol {tol})")
        assert np.isfinite(g).all(), n
        assert e <= tol, n


@pytest.mark.parametrize("shape,path", CASES)
def test_backward_chunk_mode(shape, path, force):
    B, Hq, Hkv, d, M, T, dt = shape
    H.h2o_debug_force_path(path)
    wl = W.custom("bwd", B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=T, dtype=dt, heavy_frac=0.02)
    say(f"backward {wl.describe()} path {path}")
    x = W.make_inputs(wl, seed=M + 3 * T)
    tdt = U.TDT[dt]
    q, kc, vc, kn, vn = (U.to_dev(x[n], tdt) for n in ("q", "k_cache", "v_cache", "k_new",
                                                        "v_new"))
    do_np = np.random.default_rng(7).standard_normal(x["q"].shape).astype(np.float32)
    if dt == "bf16":
        do_np = W.bf16_bits_to_f32(W.f32_to_bf16_bits(do_np))
    dout = U.to_dev(do_np, tdt)
    b = H.alloc_step(B, Hq, Hkv, T, M, d, tdt)
    scale = float(x["scale"])
    H.h2o_sdpa_chunk(q, kc, vc, kn, vn, b["out"], b["lse"], b["wsum"], b["workspace"], scale)
    grads = [torch.empty_like(t) for t in (q, kc, vc, kn, vn)]
    ws = torch.empty(max(H.h2o_backward_workspace_bytes(B, Hq, Hkv, T, M, d, tdt), 16),
                     dtype=torch.uint8, device=U.DEV)
    H.h2o_sdpa_chunk_backward(q, kc, vc, kn, vn, b["lse"], dout, *grads, ws, scale)
    torch.cuda.synchronize()
    ref = oracle.sdpa_chunk_backward(x["q"], x["k_cache"], x["v_cache"], x["k_new"], x["v_new"],
                                     do_np, scale)
    _grads_check(dt, [U.to_np(g) for g in grads], ref,
                 ("dq", "dk_cache", "dv_cache", "dk_new", "dv_new"))


CACHE_SHAPES = [(1, 4, 2, 64, 256, 64, "f32"), (2, 8, 2, 128, 300, 33, "bf16"),
                (4, 8, 4, 64, 200, 1, "bf16"), (1, 32, 8, 128, 500, 40, "bf16"),
                (1, 32, 8, 128, 2048, 256, "bf16")]   # rows passes in 8-wave blocks


@pytest.mark.parametrize("shape,path", [(sh, p) for sh in CACHE_SHAPES
                                        for p in ((-1, 0) if sh[-1] == "bf16" else (-1,))])
def test_backward_cache_mode(shape, path, force):
    """Backward of h2o_sdpa_cache: the chunk sits in scattered slots, the mask
    comes from the token positions (some rows of head (0, 0) see nothing)."""
    B, Hq, Hkv, d, M, T, dt = shape
    H.h2o_debug_force_path(path)
    wl = W.custom("bwdc", B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=T, dtype=dt)
    say(f"backward, cache mode {wl.describe()} path {path}")
    x = W.make_inputs(wl, seed=5)
    rng = np.random.default_rng(5)
    pos0 = 1000
    tp = rng.integers(pos0 - 50, pos0 + T + 3, size=(B, Hkv, M)).astype(np.int32)
    tp[0, 0] = np.maximum(tp[0, 0], pos0 + T // 2)
    tdt = U.TDT[dt]
    q, kc, vc = (U.to_dev(x[n], tdt) for n in ("q", "k_cache", "v_cache"))
    tpd = U.to_dev(tp, torch.int32)
    do_np = np.random.default_rng(9).standard_normal(x["q"].shape).astype(np.float32)
    if dt == "bf16":
        do_np = W.bf16_bits_to_f32(W.f32_to_bf16_bits(do_np))
    dout = U.to_dev(do_np, tdt)
    b = H.alloc_step(B, Hq, Hkv, T, M, d, tdt, insert_first=True)
    scale = float(x["scale"])
    H.h2o_sdpa_cache(q, kc, vc, tpd, b["out"], b["lse"], b["wsum"], b["workspace"], pos0, scale)
    dq, dkc, dvc = (torch.empty_like(t) for t in (q, kc, vc))
    ws = torch.empty(max(H.h2o_backward_workspace_bytes(B, Hq, Hkv, T, M, d, tdt), 16),
                     dtype=torch.uint8, device=U.DEV)
    H.h2o_sdpa_chunk_backward(q, kc, vc, None, None, b["lse"], dout, dq, dkc, dvc, None, None,
                              ws, scale, token_pos=tpd, pos0=pos0)
    torch.cuda.synchronize()
    ref = oracle.sdpa_chunk_backward(x["q"], x["k_cache"], x["v_cache"], None, None, do_np, scale,
                                     token_pos=tp, pos0=pos0)
    _grads_check(dt, [U.to_np(g) for g in (dq, dkc, dvc)], ref[:3], ("dq", "dk", "dv"))


def _random_shapes(n, seed):
    """Seeded random small shapes: GQA groups 1-8, both head sizes, ragged M
    and T (M = 0 included), chunk or cache mode."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        G = int(rng.choice([1, 2, 4, 7, 8]))
        Hkv = int(rng.integers(1, 4))
        d = int(rng.choice([64, 128]))
        T = int(rng.integers(1, 90))
        cache = bool(rng.integers(0, 2))
        M = int(rng.integers(1 if cache else 0, 400))
        out.append((int(rng.integers(1, 3)), G * Hkv, Hkv, d, M, T, cache))
    return out


@pytest.mark.parametrize("shape", _random_shapes(10, 2024) + [(1, 8, 2, 64, 0, 37, False),
                                                              (3, 8, 4, 128, 260, 1, True)])
def test_backward_random_shapes(shape):
    """The MFMA backward (bf16) on seeded random shapes, chunk or cache mode,
    against the oracle."""
    B, Hq, Hkv, d, M, T, cache = shape
    wl = W.custom("bwdr", B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=T, dtype="bf16", heavy_frac=0.02)
    say(f"backward random {wl.describe()} cache={cache}")
    x = W.make_inputs(wl, seed=M + T + d)
    tdt = torch.bfloat16
    rng = np.random.default_rng(M * 7 + T)
    do_np = W.bf16_bits_to_f32(W.f32_to_bf16_bits(
        rng.standard_normal(x["q"].shape).astype(np.float32)))
    q, kc, vc = (U.to_dev(x[n], tdt) for n in ("q", "k_cache", "v_cache"))
    dout = U.to_dev(do_np, tdt)
    scale = float(x["scale"])
    ws = torch.empty(max(H.h2o_backward_workspace_bytes(B, Hq, Hkv, T, M, d, tdt), 16),
                     dtype=torch.uint8, device=U.DEV)
    if cache:
        pos0 = 500
        tp = rng.integers(pos0 - 30, pos0 + T + 2, size=(B, Hkv, M)).astype(np.int32)
        tpd = U.to_dev(tp, torch.int32)
        b = H.alloc_step(B, Hq, Hkv, T, M, d, tdt, insert_first=True)
        H.h2o_sdpa_cache(q, kc, vc, tpd, b["out"], b["lse"], b["wsum"], b["workspace"], pos0,
                         scale)
        grads = [torch.empty_like(t) for t in (q, kc, vc)]
        H.h2o_sdpa_chunk_backward(q, kc, vc, None, None, b["lse"], dout, *grads, None, None, ws,
                                  scale, token_pos=tpd, pos0=pos0)
        torch.cuda.synchronize()
        ref = oracle.sdpa_chunk_backward(x["q"], x["k_cache"], x["v_cache"], None, None, do_np,
                                         scale, token_pos=tp, pos0=pos0)[:3]
        names = ("dq", "dk", "dv")
    else:
        kn, vn = U.to_dev(x["k_new"], tdt), U.to_dev(x["v_new"], tdt)
        b = H.alloc_step(B, Hq, Hkv, T, M, d, tdt)
        H.h2o_sdpa_chunk(q, kc, vc, kn, vn, b["out"], b["lse"], b["wsum"], b["workspace"], scale)
        grads = [torch.empty_like(t) for t in (q, kc, vc, kn, vn)]
        H.h2o_sdpa_chunk_backward(q, kc, vc, kn, vn, b["lse"], dout, *grads, ws, scale)
        torch.cuda.synchronize()
        ref = oracle.sdpa_chunk_backward(x["q"], x["k_cache"], x["v_cache"], x["k_new"],
                                         x["v_new"], do_np, scale)
        names = ("dq", "dk_cache", "dv_cache", "dk_new", "dv_new")
    _grads_check("bf16", [U.to_np(g) for g in grads], ref, names)


@pytest.mark.parametrize("name,b,h", [("prefill_bf16", 0, 5), ("longcache_bf16", 2, 3)])
def test_backward_full_size_sampled_head(name, b, h):
    """The backward at a full prefill size (the 1024-token shape the benchmark
    times, and the long cache) in the launch configuration of that size; the
    oracle recomputes the gradients of one KV head of one batch entry (its
    group's query heads and its keys) from that slice of the inputs."""
    wl = W.WORKLOADS[name]
    say(f"backward, full size {wl.describe()}")
    x = W.make_inputs(wl, seed=1)
    tdt = torch.bfloat16
    q, kc, vc, kn, vn = (U.to_dev(x[n], tdt) for n in ("q", "k_cache", "v_cache", "k_new",
                                                        "v_new"))
    do_np = W.bf16_bits_to_f32(W.f32_to_bf16_bits(
        np.random.default_rng(11).standard_normal(x["q"].shape).astype(np.float32)))
    dout = U.to_dev(do_np, tdt)
    bufs = H.alloc_step(wl.B, wl.Hq, wl.Hkv, wl.T, wl.M, wl.d, tdt)
    scale = float(x["scale"])
    H.h2o_sdpa_chunk(q, kc, vc, kn, vn, bufs["out"], bufs["lse"], bufs["wsum"], bufs["workspace"],
                     scale)
    grads = [torch.empty_like(t) for t in (q, kc, vc, kn, vn)]
    ws = torch.empty(H.h2o_backward_workspace_bytes(wl.B, wl.Hq, wl.Hkv, wl.T, wl.M, wl.d, tdt),
                     dtype=torch.uint8, device=U.DEV)
    H.h2o_sdpa_chunk_backward(q, kc, vc, kn, vn, bufs["lse"], dout, *grads, ws, scale)
    torch.cuda.synchronize()
    got = [U.to_np(g) for g in grads]
    for g in got:
        assert np.isfinite(g).all()
    G = wl.G
    qs, bs, hs = slice(h * G, (h + 1) * G), slice(b, b + 1), slice(h, h + 1)
    ref = oracle.sdpa_chunk_backward(x["q"][bs, qs], x["k_cache"][bs, hs], x["v_cache"][bs, hs],
                                     x["k_new"][bs, hs], x["v_new"][bs, hs], do_np[bs, qs], scale)
    sel = [got[0][bs, qs]] + [g[bs, hs] for g in got[1:]]
    _grads_check("bf16", sel, ref, ("dq", "dk_cache", "dv_cache", "dk_new", "dv_new"))


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("B,Hkv,M,k,d", [(2, 3, 40, 7, 64), (8, 8, 4096, 1, 64),
                                         (1, 8, 8192, 1024, 128)])
def test_kv_delta_round_trip(B, Hkv, M, k, d, dt):
    """Gather of the slots about to be overwritten, the insert, and the
    scatter of the gathered rows back: bit-exact against the oracle and the
    cache restored bit for bit."""
    say(f"kv delta B{B} Hkv{Hkv} M{M} k{k} d{d} {dt}")
    rng = np.random.default_rng(M + k)
    tdt = U.TDT[dt]
    cache_np = rng.standard_normal((B, Hkv, M, d)).astype(np.float32)
    new_np = rng.standard_normal((B, Hkv, k, d)).astype(np.float32)
    if dt == "bf16":
        cache_np = W.bf16_bits_to_f32(W.f32_to_bf16_bits(cache_np))
        new_np = W.bf16_bits_to_f32(W.f32_to_bf16_bits(new_np))
    idx_np = np.stack([np.stack([np.sort(rng.choice(M, k, replace=False)) for _ in range(Hkv)])
                       for _ in range(B)]).astype(np.int32)
    cache, new, idx = U.to_dev(cache_np, tdt), U.to_dev(new_np, tdt), U.to_dev(idx_np, torch.int32)
    delta = torch.empty(B, Hkv, k, d, dtype=tdt, device=U.DEV)
    H.h2o_kv_gather(cache, idx, delta)
    H.h2o_kv_scatter(cache, idx, new)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(U.to_np(delta), oracle.kv_gather(cache_np, idx_np))
    np.testing.assert_array_equal(U.to_np(cache), oracle.kv_scatter(cache_np, idx_np, new_np))
    H.h2o_kv_scatter(cache, idx, delta)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(U.to_np(cache), cache_np)


def test_backward_graph_replays_match_eager():
    """The bf16 backward (split rows passes and their reduce included)
    captured in a HIP graph and replayed three times, with eager calls and
    synchronisation between the replays: every replay gives the eager bits."""
    B, Hq, Hkv, d, M, T = 1, 8, 2, 128, 1000, 128
    wl = W.custom("bwdg", B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=T, dtype="bf16", heavy_frac=0.02)
    say(f"backward graph replay {wl.describe()}")
    x = W.make_inputs(wl, seed=4)
    tdt = torch.bfloat16
    q, kc, vc, kn, vn = (U.to_dev(x[n], tdt) for n in ("q", "k_cache", "v_cache", "k_new",
                                                        "v_new"))
    dout = U.to_dev(np.random.default_rng(3).standard_normal(x["q"].shape).astype(np.float32), tdt)
    scale = float(x["scale"])
    b = H.alloc_step(B, Hq, Hkv, T, M, d, tdt)
    H.h2o_sdpa_chunk(q, kc, vc, kn, vn, b["out"], b["lse"], b["wsum"], b["workspace"], scale)
    nbytes = H.h2o_backward_workspace_bytes(B, Hq, Hkv, T, M, d, tdt)
    wg = torch.empty(nbytes, dtype=torch.uint8, device=U.DEV)
    we = torch.empty(nbytes, dtype=torch.uint8, device=U.DEV)
    gg = [torch.empty_like(t) for t in (q, kc, vc, kn, vn)]
    ge = [torch.empty_like(t) for t in (q, kc, vc, kn, vn)]
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        H.h2o_sdpa_chunk_backward(q, kc, vc, kn, vn, b["lse"], dout, *gg, wg, scale)
    torch.cuda.synchronize()
    for r in range(3):
        for g in gg:
            g.fill_(7)            # stale outputs must be overwritten by the replay
        graph.replay()
        H.h2o_sdpa_chunk_backward(q, kc, vc, kn, vn, b["lse"], dout, *ge, we, scale)
        torch.cuda.synchronize()
        for a_, e_, n in zip(gg, ge, ("dq", "dk_cache", "dv_cache", "dk_new", "dv_new")):
            np.testing.assert_array_equal(U.to_np(a_), U.to_np(e_), err_msg=f"replay {r} {n}")
