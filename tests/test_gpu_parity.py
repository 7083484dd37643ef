"""GPU parity: the HIP path through the C ABI against the float64 oracle.

Tolerances (1e-5 for float32, 2e-2 for bf16): out and lse normwise per
(b, head) slice; wsum and the accumulated scores element by element
(``_gpu.check``). Selection is bit-exact when run on the oracle's float32
score vector; the insert is bitwise. End to end, the GPU's eviction (from
its own scores) is compared with the oracle's: every slot that differs must
lie inside a band around the oracle's k-th score whose width follows from
the float32 score error bound (``_gpu.SEL_TOL``), which the scores are
checked against first.
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

BF16_PATHS = [-1, 0, 1]       # automatic, generic VALU, MFMA


@pytest.fixture
def path(request):
    p = request.param
    H.h2o_debug_force_path(p)
    yield p
    H.h2o_debug_force_path(-1)


def _check_attention(x, dtype, res, heads=None, extra=""):
    q, kc, vc, kn, vn = x["q"], x["k_cache"], x["v_cache"], x["k_new"], x["v_new"]
    o_full = oracle.sdpa_chunk(q, kc, vc, kn, vn, x["scale"], heads=heads)
    o, l, w = o_full
    go, gl, gw = res
    if heads is not None:
        G = q.shape[1] // kc.shape[1]
        hq = [(b, h * G + g) for b, h in heads for g in range(G)]
        sel = lambda a, hs: np.stack([a[b, h] for b, h in hs])
        o, go, l, gl = sel(o, hq), sel(go, hq), sel(l, hq), sel(gl, hq)
        w, gw = sel(w, heads), sel(gw, heads)
    assert np.isfinite(gl).all()
    U.check(dtype, out=(go, o), lse=(gl, l), wsum=(gw, w), extra=extra)
    return o_full


SHAPES = [  # B, Hq, Hkv, d, M, T
    (1, 4, 2, 64, 256, 64),
    (1, 1, 1, 64, 17, 5),
    (2, 8, 2, 128, 100, 33),
    (1, 7, 1, 128, 300, 70),
    (1, 8, 1, 64, 64, 16),
    (2, 4, 4, 128, 129, 1),
    (1, 28, 4, 128, 257, 40),
    (1, 4, 1, 128, 0, 20),
    (2, 16, 4, 64, 1000, 3),
    (1, 32, 8, 64, 513, 1),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "B%dHq%dHkv%dd%dM%dT%d" % s)
def test_sdpa_f32(shape):
    say(f"sdpa f32 {shape}")
    w = W.custom(**dict(zip("B Hq Hkv d M T".split(), shape)), dtype="f32", heavy_frac=0.02)
    x = W.make_inputs(w, seed=1)
    res = U.run_sdpa(x["q"], x["k_cache"], x["v_cache"], x["k_new"], x["v_new"], x["scale"], "f32")
    _check_attention(x, "f32", res)


@pytest.mark.parametrize("path", BF16_PATHS, indirect=True)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "B%dHq%dHkv%dd%dM%dT%d" % s)
def test_sdpa_bf16(shape, path):
    say(f"sdpa bf16 {shape} path {path}")
    w = W.custom(**dict(zip("B Hq Hkv d M T".split(), shape)), dtype="bf16", heavy_frac=0.02)
    x = W.make_inputs(w, seed=2)
    res = U.run_sdpa(x["q"], x["k_cache"], x["v_cache"], x["k_new"], x["v_new"], x["scale"],
                     "bf16")
    _check_attention(x, "bf16", res, extra=f"path {path}")


@pytest.mark.parametrize("shape", [(1, 8, 1, 128, 2048, 2048), (1, 8, 1, 128, 1024, 1024)],
                         ids=lambda s: "B%dHq%dHkv%dd%dM%dT%d" % s)
def test_sdpa_bf16_whole_round_grids(shape):
    """Shapes whose grids fill whole rounds of the CUs, so the plan takes
    256-row blocks of 8 waves: both passes at the first shape, the main pass
    at the second; all heads against the oracle, and the chunk step against
    the three calls."""
    say(f"sdpa bf16 whole-round grids {shape}")
    w = W.custom(**dict(zip("B Hq Hkv d M T".split(), shape)), dtype="bf16", heavy_frac=0.02)
    x = W.make_inputs(w, seed=5)
    res = U.run_sdpa(x["q"], x["k_cache"], x["v_cache"], x["k_new"], x["v_new"], x["scale"],
                     "bf16")
    _check_attention(x, "bf16", res, extra="whole-round grids")
    B, Hq, Hkv, d, M, T = shape
    q, kn, vn = (U.to_dev(x[n], torch.bfloat16) for n in ("q", "k_new", "v_new"))
    out = []
    for fused in (False, True):
        st = U.device_state(x, "bf16")
        bufs = H.alloc_step(B, Hq, Hkv, T, M, d, torch.bfloat16)
        H.step(st, q, kn, vn, bufs, int(x["pos0"]), float(x["scale"]), fused=fused)
        torch.cuda.synchronize()
        out.append([U.to_np(bufs[n]) for n in ("out", "wsum", "evict_idx")] +
                   [U.to_np(st[n]) for n in ("k_cache", "scores")])
    for a, b in zip(*out):
        np.testing.assert_array_equal(a, b)


def test_tiny_f32_full_step():
    """The 1x4x2, d64, M256, T64 float32 step: attention, accumulate, evict, insert."""
    wl = W.WORKLOADS["tiny_f32"]
    say(f"full step {wl.describe()}")
    x = W.make_inputs(wl, seed=0)
    st = U.device_state(x, "f32")
    tdt = torch.float32
    q, kn, vn = (U.to_dev(x[n], tdt) for n in ("q", "k_new", "v_new"))
    bufs = H.alloc_step(wl.B, wl.Hq, wl.Hkv, wl.T, wl.M, wl.d, tdt)
    H.h2o_sdpa_chunk(q, st["k_cache"], st["v_cache"], kn, vn, bufs["out"], bufs["lse"],
                     bufs["wsum"], bufs["workspace"], float(x["scale"]))
    torch.cuda.synchronize()
    res = tuple(U.to_np(bufs[n]) for n in ("out", "lse", "wsum"))
    o, l, w = _check_attention(x, "f32", res)
    H.h2o_accumulate_scores(st["scores"], bufs["wsum"])
    torch.cuda.synchronize()
    g_acc = st["scores"].cpu().numpy()
    # bitwise: the kernel adds exactly the float32 values it was given
    np.testing.assert_array_equal(g_acc, oracle.accumulate_scores(x["scores"], res[2]))
    o_acc = oracle.accumulate_scores(x["scores"], w)
    U.check("f32", scores=(g_acc, o_acc), extra="accumulated scores")
    # selection on the oracle's own float32 scores is bit-exact
    np.testing.assert_array_equal(U.gpu_bottomk(o_acc, wl.T), oracle.bottomk(o_acc, wl.T))
    # end-to-end eviction from the GPU's own scores + bitwise insert
    H.h2o_evict_insert(st["k_cache"], st["v_cache"], st["scores"], st["token_pos"], kn, vn,
                       bufs["wsum"], bufs["evict_idx"], int(x["pos0"]))
    torch.cuda.synchronize()
    g_idx = bufs["evict_idx"].cpu().numpy()
    np.testing.assert_array_equal(g_idx, oracle.bottomk(g_acc, wl.T))
    kc2, vc2, sc2, tp2, _ = oracle.evict_insert(x["k_cache"], x["v_cache"], g_acc, x["token_pos"],
                                                x["k_new"], x["v_new"], res[2], wl.T,
                                                int(x["pos0"]))
    np.testing.assert_array_equal(st["k_cache"].cpu().numpy(), kc2)
    np.testing.assert_array_equal(st["v_cache"].cpu().numpy(), vc2)
    np.testing.assert_array_equal(st["scores"].cpu().numpy(), sc2)
    np.testing.assert_array_equal(st["token_pos"].cpu().numpy(), tp2)


@pytest.mark.parametrize("rows,M,k,quant", [
    (1, 1, 1, None), (3, 10, 10, None), (4, 300, 64, None), (4, 300, 64, 2),
    (8, 8192, 1024, None), (8, 8192, 1024, 3), (2, 16384, 2048, 0), (64, 4096, 1, None),
    (64, 4096, 1, 0), (5, 33, 32, 1), (2, 32768, 512, None), (3, 4097, 4096, 5),
    (32, 32768, 512, 8), (2, 40000, 300, None), (1, 65537, 5000, 2), (1, 50000, 50000, 0)])
def test_bottomk_exact(rows, M, k, quant):
    """Rows past 32768 slots take the kernel that reads the keys from global
    memory in every pass; quantised scores force ties at the k-th key."""
    say(f"bottomk rows {rows} M {M} k {k} quant {quant}")
    rng = np.random.default_rng(rows * M + k)
    s = rng.standard_exponential((rows, M)).astype(np.float32)
    if quant is not None:
        s = (np.floor(s * 2 ** quant) / 2 ** quant).astype(np.float32)
    if M > 3:
        s[0, :3] = -0.0
    np.testing.assert_array_equal(U.gpu_bottomk(s, k), oracle.bottomk(s, k))


@pytest.mark.parametrize("M,k,nties", [(8192, 1024, 40), (8192, 1024, 1), (20000, 2048, 90),
                                        (40000, 512, 7), (1000, 999, 3), (300, 1, 5)])
def test_bottomk_few_keys_in_the_bin(M, k, nties):
    """Rows whose first 12-bit digit leaves few keys in the chosen bin (the
    keys are then ranked against each other), with nties copies of the k-th
    value spread over the row so that some but not all equal keys are taken."""
    say(f"bottomk few keys M {M} k {k} ties {nties}")
    rng = np.random.default_rng(M + k + nties)
    s = rng.standard_exponential((3, M)).astype(np.float32)
    for r in range(3):
        tau = np.sort(s[r])[k - 1]
        s[r, rng.choice(M, nties, replace=False)] = tau
    np.testing.assert_array_equal(U.gpu_bottomk(s, k), oracle.bottomk(s, k))


@pytest.mark.parametrize("M,nbin", [(8192, 256), (8192, 257), (20000, 256), (20000, 2049),
                                    (40000, 200), (40000, 300)])
def test_bottomk_bin_size_limits(M, nbin):
    """The k-th key's first-digit bin holds exactly nbin keys: at most 256
    are ranked against each other, more take the remaining digits (over the
    gathered keys up to 2,048 of them in rows of 16,384 slots or more, over
    the row beyond)."""
    say(f"bottomk bin size M {M} bin {nbin}")
    rng = np.random.default_rng(M + nbin)
    below = 900
    s = np.empty((2, M), np.float32)
    for r in range(2):
        low = rng.uniform(1e-3, 2e-3, below)                 # below the bin
        inbin = 1.0 + rng.integers(0, 200, nbin) / 2048.0    # [1, 1.1): one first-digit bin, ties
        high = rng.uniform(100.0, 200.0, M - below - nbin)   # above it
        row = np.concatenate([low, inbin, high]).astype(np.float32)
        s[r] = row[rng.permutation(M)]
    for k in (below + 1, below + nbin // 2, below + nbin):
        np.testing.assert_array_equal(U.gpu_bottomk(s, k), oracle.bottomk(s, k))


def test_bottomk_negative_and_huge_values():
    s = np.array([[3.0, -1.0, np.inf, -np.inf, 0.0, -0.0, 1e-45, -1e-45, 3.4e38, 2.0]],
                 np.float32)
    for k in range(0, 11):
        if k == 0:
            continue
        np.testing.assert_array_equal(U.gpu_bottomk(s, k), oracle.bottomk(s, k))


def test_selection_with_every_key_at_the_top():
    """Scores whose order key is the largest one (NaN with a full payload, a
    value no arithmetic produces): the (key, slot) minimum is then the lowest
    slots, so the selection and the decode step's argmin still choose slots
    inside the cache."""
    top = np.array([0x7FFFFFFF], np.uint32).view(np.float32)[0]
    for M, k in ((1, 1), (4096, 1), (300, 4), (9000, 7)):
        say(f"all-top keys M {M} k {k}")
        s = np.full((3, M), top, np.float32)
        np.testing.assert_array_equal(U.gpu_bottomk(s, k),
                                      np.tile(np.arange(k, dtype=np.int32), (3, 1)))
    B, Hq, Hkv, d, M = 2, 8, 2, 64, 512
    wl = W.custom("top", B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=1, dtype="bf16", heavy_frac=0.02)
    x = W.make_inputs(wl, seed=17)
    x["scores"] = np.full_like(x["scores"], top)
    q, kn, vn = (U.to_dev(x[n], torch.bfloat16) for n in ("q", "k_new", "v_new"))
    st = U.device_state(x, "bf16")
    bufs = H.alloc_step(B, Hq, Hkv, 1, M, d, torch.bfloat16)
    H.step(st, q, kn, vn, bufs, int(x["pos0"]), float(x["scale"]))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(U.to_np(bufs["evict_idx"]).reshape(-1), np.zeros(B * Hkv))


DECODE_SHAPES = [(2, 4, 4, 128, 129, 1), (1, 32, 8, 64, 513, 1), (8, 32, 8, 64, 4096, 1),
                 (3, 16, 2, 64, 1000, 1), (1, 2, 1, 64, 256, 1), (2, 8, 2, 128, 300, 1),
                 (1, 8, 8, 64, 1, 1), (1, 4, 2, 64, 0, 1)]


@pytest.mark.parametrize("shape", DECODE_SHAPES, ids=lambda s: "B%dHq%dHkv%dd%dM%dT%d" % s)
def test_sdpa_decode_path(shape):
    H.h2o_debug_force_path(2)
    try:
        say(f"decode path {shape}")
        w = W.custom(**dict(zip("B Hq Hkv d M T".split(), shape)), dtype="bf16",
                     heavy_frac=0.02)
        x = W.make_inputs(w, seed=3)
        res = U.run_sdpa(x["q"], x["k_cache"], x["v_cache"], x["k_new"], x["v_new"],
                         x["scale"], "bf16")
        _check_attention(x, "bf16", res, extra="decode path")
    finally:
        H.h2o_debug_force_path(-1)


@pytest.mark.parametrize("path_id,M,T", [(2, 1000, 1), (2, 4096, 1), (1, 1000, 33),
                                         (0, 1000, 33), (1, 4096, 64)])
def test_sdpa_very_negative_logits(path_id, M, T):
    # Every logit near -128 (about -185 in log2 units): exp2 of any logit
    # relative to a maximum of 0 underflows float32. The zero rows read past
    # the keys' end (a ragged last step or tile) must not count as logits of
    # 0 in a running maximum. Paths: 2 decode, 1 MFMA, 0 generic.
    H.h2o_debug_force_path(path_id)
    try:
        shape = dict(B=1, Hq=4, Hkv=1, d=64, M=M, T=T)
        say(f"path {path_id}, very negative logits {shape}")
        w = W.custom(**shape, dtype="bf16")
        x = W.make_inputs(w, seed=11)
        rng = np.random.Generator(np.random.PCG64(12))
        def fill(a, sign):
            v = (sign * (4.0 + 0.1 * rng.standard_normal(a.shape))).astype(np.float32)
            return W.bf16_bits_to_f32(W.f32_to_bf16_bits(v))
        x["q"] = fill(x["q"], 1.0)
        for k in ("k_cache", "k_new"):
            x[k] = fill(x[k], -1.0)
        res = U.run_sdpa(x["q"], x["k_cache"], x["v_cache"], x["k_new"], x["v_new"],
                         x["scale"], "bf16")
        _check_attention(x, "bf16", res, extra=f"path {path_id}, logits ~ -128")
    finally:
        H.h2o_debug_force_path(-1)


@pytest.mark.parametrize("path", BF16_PATHS + [2], indirect=True)
def test_bitwise_repeatable(path):
    say(f"repeatability path {path}")
    w = W.custom(B=1, Hq=8, Hkv=2, d=128, M=777, T=1 if path == 2 else 100, dtype="bf16",
                 heavy_frac=0.02)
    x = W.make_inputs(w, seed=5)
    a = U.run_sdpa(x["q"], x["k_cache"], x["v_cache"], x["k_new"], x["v_new"], x["scale"], "bf16")
    b = U.run_sdpa(x["q"], x["k_cache"], x["v_cache"], x["k_new"], x["v_new"], x["scale"], "bf16")
    for u, v in zip(a, b):
        np.testing.assert_array_equal(u, v)


def _state_to_np(st):
    return {k: (v.float() if v.dtype == torch.bfloat16 else v).cpu().numpy()
            for k, v in st.items()}


@pytest.mark.parametrize("name,nheads", [("prefill_bf16", 2), ("longcache_bf16", 2),
                                         ("gqa7_bf16", 1)])
def test_full_size_step_sampled_heads(name, nheads):
    """Full-size chunk step; the oracle recomputes a sample of (b, kv-head)
    pairs (all their query heads, all keys) and the eviction is checked on
    the sampled heads' oracle scores (bit-exact) and for validity on all."""
    wl = W.WORKLOADS[name]
    say(f"full-size {wl.describe()}")
    x = W.make_inputs(wl, seed=0)
    st = U.device_state(x, "bf16")
    tdt = torch.bfloat16
    q, kn, vn = (U.to_dev(x[n], tdt) for n in ("q", "k_new", "v_new"))
    bufs = H.alloc_step(wl.B, wl.Hq, wl.Hkv, wl.T, wl.M, wl.d, tdt)
    H.h2o_sdpa_chunk(q, st["k_cache"], st["v_cache"], kn, vn, bufs["out"], bufs["lse"],
                     bufs["wsum"], bufs["workspace"], float(x["scale"]))
    H.h2o_accumulate_scores(st["scores"], bufs["wsum"])
    torch.cuda.synchronize()
    res = tuple(U.to_np(bufs[n]) for n in ("out", "lse", "wsum"))
    g_acc = st["scores"].cpu().numpy()
    rng = np.random.default_rng(0)
    pairs = [(b, h) for b in range(wl.B) for h in range(wl.Hkv)]
    heads = [pairs[i] for i in rng.choice(len(pairs), size=nheads, replace=False)]
    o, l, w = _check_attention(x, "bf16", res, heads=heads, extra=f"heads {heads}")
    # every query row's weights sum to one: per KV head, sum_j wsum = T*G
    np.testing.assert_allclose(res[2].sum(-1), wl.T * wl.G, rtol=2e-3)
    M, k = wl.M, wl.T
    o_accs = {}
    for (b, h) in heads:
        o_acc = oracle.accumulate_scores(x["scores"][b, h], w[b, h])
        o_accs[(b, h)] = o_acc
        # the accumulated scores, element by element, at the stated tolerance
        # and at the score error bound the eviction band below rests on
        e_s = U.check("bf16", scores=(g_acc[b, h], o_acc), extra=f"scores {(b, h)}")["scores"]
        assert e_s <= U.SEL_TOL, f"score error {e_s:.2e} above the bound {U.SEL_TOL}"
        np.testing.assert_array_equal(U.gpu_bottomk(o_acc[None], k)[0],
                                      oracle.bottomk(o_acc[None], k)[0])
    H.h2o_evict_insert(st["k_cache"], st["v_cache"], st["scores"], st["token_pos"], kn, vn,
                       bufs["wsum"], bufs["evict_idx"], int(x["pos0"]))
    torch.cuda.synchronize()
    g_idx = bufs["evict_idx"].cpu().numpy()
    np.testing.assert_array_equal(g_idx, oracle.bottomk(g_acc, k))     # on the GPU's scores
    for (b, h) in heads:       # against the oracle's eviction: only near-ties may differ
        n_diff, n_band, ok = oracle.eviction_agreement(g_idx[b, h], o_accs[(b, h)], k,
                                                       U.SEL_TOL)
        say(f"  head {(b, h)}: {n_diff} of {k} evicted slots differ from the oracle's; "
            f"{n_band} oracle slots lie within the band of {U.SEL_TOL} around the k-th score")
        assert ok and n_diff <= n_band
    kc = st["k_cache"].float().cpu().numpy()
    for (b, h) in heads:
        np.testing.assert_array_equal(kc[b, h][g_idx[b, h]], x["k_new"][b, h])
        untouched = np.setdiff1d(np.arange(M), g_idx[b, h])
        np.testing.assert_array_equal(kc[b, h][untouched], x["k_cache"][b, h][untouched])
    assert (st["token_pos"].cpu().numpy()[0, 0][g_idx[0, 0]] ==
            int(x["pos0"]) + np.arange(k)).all()


def test_decode_trajectory_teacher_forced():
    """16 decode steps (T=1, k=1); before each step the oracle takes the GPU's
    state, so every step is checked on its own."""
    wl = W.WORKLOADS["decode_bf16"]
    say(f"decode {wl.describe()}")
    x = W.make_inputs(wl, seed=0)
    st = U.device_state(x, "bf16")
    tdt = torch.bfloat16
    bufs = H.alloc_step(wl.B, wl.Hq, wl.Hkv, 1, wl.M, wl.d, tdt)
    n_mismatch = 0
    for s in range(wl.steps):
        pre = _state_to_np(st)
        q, kn, vn = (U.to_dev(x[n][s], tdt) for n in ("q_steps", "k_new_steps", "v_new_steps"))
        pos = int(x["pos0"]) + s
        H.step(st, q, kn, vn, bufs, pos, float(x["scale"]))
        torch.cuda.synchronize()
        pre_k = pre["k_cache"].astype(np.float32)
        pre_v = pre["v_cache"].astype(np.float32)
        ref = oracle.h2o_step(pre_k, pre_v, pre["scores"], pre["token_pos"], x["q_steps"][s],
                              x["k_new_steps"][s], x["v_new_steps"][s], pos, x["scale"])
        go, gw = U.to_np(bufs["out"]), U.to_np(bufs["wsum"])
        U.check("bf16", out=(go, ref["out"]), wsum=(gw, ref["wsum"]), extra=f"step {s}")
        g_idx = bufs["evict_idx"].cpu().numpy()
        # the GPU's choice is the argmin of the GPU's own accumulated scores
        g_acc = oracle.accumulate_scores(pre["scores"], gw)
        np.testing.assert_array_equal(g_idx, oracle.bottomk(g_acc, 1))
        assert oracle.elem_err(g_acc, ref["scores_acc"], (-1,)) <= U.SEL_TOL
        # and agrees with the oracle's, up to near-ties of the band
        for b in range(wl.B):
            for h in range(wl.Hkv):
                n_diff, _, ok = oracle.eviction_agreement(g_idx[b, h], ref["scores_acc"][b, h],
                                                          1, U.SEL_TOL)
                assert ok, f"step {s} head {(b, h)}: eviction outside the band"
                n_mismatch += n_diff
        # and the inserted key is where the GPU says
        kc = st["k_cache"].float().cpu().numpy()
        for b in range(wl.B):
            for h in range(wl.Hkv):
                np.testing.assert_array_equal(kc[b, h, g_idx[b, h, 0]], x["k_new_steps"][s, b, h, 0])
    say(f"  eviction choices differing from the oracle over 16 steps: {n_mismatch} / "
        f"{16 * wl.B * wl.Hkv} (each inside the band)")


STEP_SHAPES = [  # B, Hq, Hkv, d, M, T, dtype
    (8, 32, 8, 64, 4096, 1, "bf16"),
    (2, 8, 2, 64, 700, 1, "bf16"),
    (1, 8, 1, 64, 37, 1, "bf16"),
    (2, 8, 4, 128, 1025, 1, "bf16"),
    (1, 2, 2, 128, 3, 1, "bf16"),
    (1, 4, 2, 64, 256, 64, "f32"),
    (1, 8, 2, 128, 300, 70, "bf16"),
    (2, 4, 2, 64, 500, 1, "f32"),
    (1, 4, 1, 64, 40000, 300, "bf16"),   # rows longer than the selection stages in LDS
    (40, 4, 4, 64, 96, 33, "bf16"),      # 160 rows: one block per row in the fused selection
    (1, 4, 1, 64, 4500, 4200, "bf16"),   # k above the fused selection's limit: separate kernels
    (1, 4, 2, 64, 64, 64, "bf16"),       # k = M: every slot is evicted
    (2, 4, 1, 64, 1000, 2, "bf16"),      # the smallest k of the fused selection
]


@pytest.mark.parametrize("shape", STEP_SHAPES)
def test_chunk_step_equals_three_calls(shape):
    """h2o_chunk_step gives the same bits as h2o_sdpa_chunk + h2o_accumulate_scores
    + h2o_evict_insert, and its attention matches the oracle."""
    B, Hq, Hkv, d, M, T, dt = shape
    wl = W.custom("step", B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=T, dtype=dt, heavy_frac=0.02)
    say(f"chunk step {wl.describe()}")
    x = W.make_inputs(wl, seed=11)
    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    q, kn, vn = (U.to_dev(x[n], tdt) for n in ("q", "k_new", "v_new"))
    res = []
    for fused in (False, True):
        st = U.device_state(x, dt)
        bufs = H.alloc_step(B, Hq, Hkv, T, M, d, tdt)
        H.step(st, q, kn, vn, bufs, int(x["pos0"]), float(x["scale"]), fused=fused)
        torch.cuda.synchronize()
        res.append({**{n: U.to_np(bufs[n]) for n in ("out", "lse", "wsum", "evict_idx")},
                    **{n: U.to_np(st[n]) for n in ("k_cache", "v_cache", "scores", "token_pos")}})
    for n in res[0]:
        np.testing.assert_array_equal(res[1][n], res[0][n], err_msg=n)
    _check_attention(x, dt, (res[1]["out"], res[1]["lse"], res[1]["wsum"]), extra="fused")
    # the accumulated scores of the kept slots against the oracle's
    ref = oracle.h2o_step(x["k_cache"], x["v_cache"], x["scores"], x["token_pos"], x["q"],
                          x["k_new"], x["v_new"], int(x["pos0"]), x["scale"])
    g_acc = oracle.accumulate_scores(x["scores"], res[1]["wsum"])
    U.check(dt, scores=(g_acc, ref["scores_acc"]), extra="accumulated scores")


@pytest.mark.parametrize("shape", STEP_SHAPES)
def test_attend_then_evict_equals_step(shape):
    """h2o_chunk_step_attend then h2o_chunk_step_evict, the second on another
    stream after an event, give the bits of h2o_chunk_step."""
    B, Hq, Hkv, d, M, T, dt = shape
    wl = W.custom("halves", B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=T, dtype=dt, heavy_frac=0.02)
    say(f"attend + evict {wl.describe()}")
    x = W.make_inputs(wl, seed=13)
    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    q, kn, vn = (U.to_dev(x[n], tdt) for n in ("q", "k_new", "v_new"))
    pos0, scale = int(x["pos0"]), float(x["scale"])
    res = []
    for halves in (False, True):
        st = U.device_state(x, dt)
        b = H.alloc_step(B, Hq, Hkv, T, M, d, tdt)
        args = (q, st["k_cache"], st["v_cache"], st["scores"], st["token_pos"], kn, vn, b["out"],
                b["lse"], b["wsum"], b["evict_idx"], b["workspace"], pos0, scale)
        torch.cuda.synchronize()
        if halves:
            side = torch.cuda.Stream()
            H.h2o_chunk_step(*args, part="attend")
            ev = torch.cuda.Event()
            ev.record()
            side.wait_event(ev)
            with torch.cuda.stream(side):
                H.h2o_chunk_step(*args, part="evict")
        else:
            H.h2o_chunk_step(*args)
        torch.cuda.synchronize()
        res.append({**{n: U.to_np(b[n]) for n in ("out", "lse", "wsum", "evict_idx")},
                    **{n: U.to_np(st[n]) for n in ("k_cache", "v_cache", "scores", "token_pos")}})
    for n in res[0]:
        np.testing.assert_array_equal(res[1][n], res[0][n], err_msg=n)


@pytest.mark.parametrize("shape", [(8, 32, 8, 64, 4096, 1, "bf16"), (1, 8, 2, 128, 300, 70, "bf16")])
def test_graph_replays_match_eager(shape):
    """The chunk step captured in a HIP graph and replayed three times (the
    state advancing each time, with eager work and synchronisation between
    replays) gives the same bits as the same steps run eagerly."""
    B, Hq, Hkv, d, M, T, dt = shape
    wl = W.custom("graph", B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=T, dtype=dt, heavy_frac=0.02)
    say(f"graph replay {wl.describe()}")
    x = W.make_inputs(wl, seed=5)
    tdt = torch.bfloat16
    q, kn, vn = (U.to_dev(x[n], tdt) for n in ("q", "k_new", "v_new"))
    pos0, scale = int(x["pos0"]), float(x["scale"])
    sg, se = U.device_state(x, dt), U.device_state(x, dt)
    bg = H.alloc_step(B, Hq, Hkv, T, M, d, tdt)
    be = H.alloc_step(B, Hq, Hkv, T, M, d, tdt)
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        H.step(sg, q, kn, vn, bg, pos0, scale)
    torch.cuda.synchronize()          # capture does not run the step
    for r in range(3):
        graph.replay()
        H.step(se, q, kn, vn, be, pos0, scale)
        torch.cuda.synchronize()
        for n in ("out", "lse", "wsum", "evict_idx"):
            np.testing.assert_array_equal(U.to_np(bg[n]), U.to_np(be[n]), err_msg=f"replay {r} {n}")
        for n in ("k_cache", "v_cache", "scores", "token_pos"):
            np.testing.assert_array_equal(U.to_np(sg[n]), U.to_np(se[n]), err_msg=f"replay {r} {n}")
