"""Pins of the float64 oracle against computations that are not the oracle.

CPU only. Each pin is a different route to the same numbers (brute force,
torch's SDPA, the paper's two alternative summed-weight algorithms), a closed
form, or an invariant the mathematics fixes. ``test_planted_mistakes`` shows
that plausible mistakes in the oracle are caught by at least one pin.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from oracle import h2o_oracle as O
from paper_2608_19920_amd import workloads as W
import _pins as P

TINY = [  # B, Hq, Hkv, d, M, T
    (1, 1, 1, 4, 3, 1),
    (1, 2, 1, 8, 5, 3),
    (2, 4, 2, 4, 7, 4),
    (1, 3, 1, 6, 0, 4),      # no cache slots: plain causal attention
    (1, 2, 2, 5, 16, 2),
]


def _inputs(B, Hq, Hkv, d, M, T, seed=0, dtype="f32", heavy=0.0):
    w = W.custom(B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=T, dtype=dtype, heavy_frac=heavy)
    return W.make_inputs(w, seed)


def _args(x):
    return x["q"], x["k_cache"], x["v_cache"], x["k_new"], x["v_new"]


# --------------------------------------------------------------- attention
@pytest.mark.parametrize("shape", TINY)
def test_brute_force(shape):
    x = _inputs(*shape, seed=sum(shape))
    o, l, w = oracle.sdpa_chunk(*_args(x), x["scale"])
    bo, bl, bw = P.brute_sdpa(*_args(x), x["scale"])
    np.testing.assert_allclose(o, bo, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(l, bl, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(w, bw, rtol=1e-12, atol=1e-13)


def test_brute_force_bf16_heavy_hitters():
    x = _inputs(1, 4, 2, 8, 12, 3, seed=7, dtype="bf16", heavy=0.25)
    o, l, w = oracle.sdpa_chunk(*_args(x), x["scale"])
    bo, bl, bw = P.brute_sdpa(*_args(x), x["scale"])
    np.testing.assert_allclose(o, bo, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(l, bl, rtol=1e-13)
    np.testing.assert_allclose(w, bw, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("shape", [(2, 6, 2, 16, 40, 9), (1, 7, 1, 32, 70, 33),
                                   (1, 4, 4, 64, 130, 17)])
def test_torch_sdpa(shape):
    x = _inputs(*shape, seed=3, dtype="bf16", heavy=0.05)
    o, l, _ = oracle.sdpa_chunk(*_args(x), x["scale"])
    to, tl = P.torch_sdpa(*_args(x), x["scale"])
    np.testing.assert_allclose(o, to, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(l, tl, rtol=1e-13)


def test_special_case_no_cache_is_causal_attention():
    x = _inputs(1, 2, 1, 16, 0, 11, seed=5)
    o, _, _ = oracle.sdpa_chunk(*_args(x), x["scale"])
    F = torch.nn.functional
    K = torch.from_numpy(x["k_new"][0, 0].astype(np.float64))
    V = torch.from_numpy(x["v_new"][0, 0].astype(np.float64))
    for g in range(2):
        Q = torch.from_numpy(x["q"][0, g].astype(np.float64))
        ref = F.scaled_dot_product_attention(Q[None], K[None], V[None], is_causal=True,
                                             scale=float(x["scale"]))[0]
        np.testing.assert_allclose(o[0, g], ref.numpy(), rtol=1e-12, atol=1e-13)


def test_special_case_single_query_is_unmasked_attention():
    x = _inputs(1, 4, 2, 16, 50, 1, seed=6)
    o, _, _ = oracle.sdpa_chunk(*_args(x), x["scale"])
    F = torch.nn.functional
    for hq in range(4):
        h = hq // 2
        K = torch.from_numpy(np.concatenate([x["k_cache"][0, h], x["k_new"][0, h]]).astype(np.float64))
        V = torch.from_numpy(np.concatenate([x["v_cache"][0, h], x["v_new"][0, h]]).astype(np.float64))
        Q = torch.from_numpy(x["q"][0, hq].astype(np.float64))
        ref = F.scaled_dot_product_attention(Q[None], K[None], V[None], scale=float(x["scale"]))[0]
        np.testing.assert_allclose(o[0, hq], ref.numpy(), rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("G,M,T", [(1, 10, 4), (3, 37, 9), (7, 5, 5)])
def test_closed_form_zero_keys(G, M, T):
    x = _inputs(1, 2 * G, 2, 8, M, T, seed=11)
    kc = np.zeros_like(x["k_cache"])
    kn = np.zeros_like(x["k_new"])
    o, l, w = oracle.sdpa_chunk(x["q"], kc, x["v_cache"], kn, x["v_new"], x["scale"])
    for h in range(2):
        V = np.concatenate([x["v_cache"][0, h], x["v_new"][0, h]]).astype(np.float64)
        for i in range(T):
            for g in range(G):
                np.testing.assert_allclose(o[0, h * G + g, i], V[:M + i + 1].mean(axis=0),
                                           rtol=1e-12, atol=1e-13)
                assert abs(l[0, h * G + g, i] - np.log(M + i + 1)) < 1e-13
        inv = np.array([1.0 / (M + i + 1) for i in range(T)])
        np.testing.assert_allclose(w[0, h, :M], G * inv.sum(), rtol=1e-13)
        for t in range(T):
            np.testing.assert_allclose(w[0, h, M + t], G * inv[t:].sum(), rtol=1e-13)


@pytest.mark.parametrize("shape", [(2, 8, 2, 16, 64, 16), (1, 7, 1, 32, 33, 20)])
def test_invariants(shape):
    B, Hq, Hkv, d, M, T = shape
    G = Hq // Hkv
    x = _inputs(*shape, seed=12, dtype="bf16", heavy=0.1)
    o, l, w = oracle.sdpa_chunk(*_args(x), x["scale"])
    # every query row's weights sum to one  =>  per KV head, sum_j w = T*G
    np.testing.assert_allclose(w.sum(axis=-1), T * G, rtol=1e-13)
    assert (w >= 0).all()
    assert (w[..., :M] <= G * T * (1 + 1e-13)).all()
    for t in range(T):                    # chunk key t is seen by queries t..T-1
        assert (w[..., M + t] <= G * (T - t) * (1 + 1e-13)).all()
    assert np.isfinite(o).all() and np.isfinite(l).all()


@pytest.mark.parametrize("rt,ct", [(1, 1), (2, 3), (3, 7), (5, 64), (64, 5)])
def test_mapreduce_algorithm(rt, ct):
    x = _inputs(1, 4, 2, 8, 23, 6, seed=13, dtype="bf16", heavy=0.1)
    o, _, w = oracle.sdpa_chunk(*_args(x), x["scale"])
    mo, mw = P.mapreduce_wsum(*_args(x), x["scale"], rt, ct)
    np.testing.assert_allclose(mw, w, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(mo, o, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("shape", [(1, 4, 2, 8, 23, 6), (2, 3, 1, 16, 50, 12)])
def test_transposed_identity(shape):
    x = _inputs(*shape, seed=14, dtype="bf16", heavy=0.1)
    _, _, w = oracle.sdpa_chunk(*_args(x), x["scale"])
    tw = P.transposed_wsum(*_args(x), x["scale"])
    np.testing.assert_allclose(tw, w, rtol=1e-11, atol=1e-12)


def test_cache_slot_permutation():
    x = _inputs(1, 4, 2, 16, 31, 7, seed=15, dtype="bf16", heavy=0.1)
    o, l, w = oracle.sdpa_chunk(*_args(x), x["scale"])
    perm = np.random.default_rng(0).permutation(31)
    o2, l2, w2 = oracle.sdpa_chunk(x["q"], x["k_cache"][:, :, perm], x["v_cache"][:, :, perm],
                                   x["k_new"], x["v_new"], x["scale"])
    np.testing.assert_allclose(o2, o, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(l2, l, rtol=1e-13)
    np.testing.assert_allclose(w2[..., :31], w[..., perm], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(w2[..., 31:], w[..., 31:], rtol=1e-12, atol=1e-14)


def test_gqa_equals_sum_of_replicated_heads():
    """Group of G query heads on one KV head == G separate heads (G=1) whose
    KV head is a copy, summed: pins the contiguous hq // G mapping and the
    group sum of the per-head (B, Hq, N_k) arrays."""
    G, Hkv = 3, 2
    x = _inputs(2, G * Hkv, Hkv, 8, 19, 5, seed=16)
    o, l, w = oracle.sdpa_chunk(*_args(x), x["scale"])
    rep = lambda a: np.repeat(a, G, axis=1)           # KV head h -> q heads hG..hG+G-1
    o1, l1, w1 = oracle.sdpa_chunk(x["q"], rep(x["k_cache"]), rep(x["v_cache"]),
                                   rep(x["k_new"]), rep(x["v_new"]), x["scale"])
    np.testing.assert_allclose(o1, o, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(w1.reshape(2, Hkv, G, -1).sum(axis=2), w, rtol=1e-13)
    bo, bl, bw = P.brute_sdpa(x["q"][:1, :G], x["k_cache"][:1, :1], x["v_cache"][:1, :1],
                              x["k_new"][:1, :1], x["v_new"][:1, :1], x["scale"])
    np.testing.assert_allclose(w[:1, :1], bw, rtol=1e-12)


# ---------------------------------------------------------------- scores
def _f32_round_exact(fr: Fraction) -> np.float32:
    """Round an exact rational to float32, nearest with ties to even."""
    c = np.float32(float(fr))
    cands = {c, np.nextafter(c, np.float32(np.inf)), np.nextafter(c, np.float32(-np.inf))}
    best = min(cands, key=lambda v: (abs(Fraction(float(v)) - fr),
                                     int(np.array(v).view(np.uint32)) & 1))
    return np.float32(best)


def test_accumulate_is_one_float32_rounding():
    rng = np.random.default_rng(1)
    s = rng.standard_exponential((3, 2, 200)).astype(np.float32)
    s[0, 0, :5] = [0.0, 1e-30, 3.0e38, 1.0, 2 ** -20]
    w = rng.standard_exponential((3, 2, 210)) * 10 ** rng.uniform(-8, 3, (3, 2, 210))
    w = w.astype(np.float32)
    acc = oracle.accumulate_scores(s, w)
    assert acc.dtype == np.float32 and acc.shape == s.shape
    for idx in np.ndindex(s.shape):
        exact = Fraction(float(s[idx])) + Fraction(float(w[idx[:-1] + (idx[-1],)]))
        assert acc[idx] == _f32_round_exact(exact), idx


@pytest.mark.parametrize("M,k,quant", [(50, 7, None), (300, 64, None), (300, 64, 4),
                                       (33, 1, None), (33, 1, 1), (40, 40, 2), (40, 0, None),
                                       (1000, 999, 3)])
def test_bottomk_brute_force(M, k, quant):
    rng = np.random.default_rng(M + k)
    s = rng.standard_exponential((3, 4, M)).astype(np.float32)
    if quant is not None:                       # many exact ties: multiples of 2^-quant
        s = (np.floor(s * 2 ** quant) / 2 ** quant).astype(np.float32)
    e = oracle.bottomk(s, k)
    np.testing.assert_array_equal(e, P.brute_bottomk(s, k))
    for r in np.ndindex(s.shape[:-1]):
        sel = e[r]
        assert len(set(sel.tolist())) == k and (np.diff(sel) > 0).all()
        if 0 < k < M:
            rest = np.setdiff1d(np.arange(M), sel)
            assert s[r][sel].max() <= s[r][rest].min()
            tau = s[r][sel].max()                   # ties at the threshold: lower slots first
            if (s[r][rest] == tau).any():
                assert sel[s[r][sel] == tau].max() < rest[s[r][rest] == tau].min()


def test_bottomk_signed_zero_is_a_tie():
    s = np.array([[1.0, -0.0, 0.0, 2.0, -0.0]], np.float32)
    np.testing.assert_array_equal(oracle.bottomk(s, 2), [[1, 2]])
    np.testing.assert_array_equal(oracle.bottomk(s, 3), [[1, 2, 4]])


# ---------------------------------------------------------------- insert
def _scatter_torch(buf, idx, src):
    """buf.scatter(2, index broadcast along d, src) as stated for the cache buffers."""
    t = torch.from_numpy(buf.copy())
    ix = torch.from_numpy(idx.astype(np.int64))
    if t.dim() == 4:
        ix = ix.unsqueeze(-1).expand(-1, -1, -1, t.shape[-1])
    return t.scatter(2, ix, torch.from_numpy(src.copy())).numpy()


def _gather_torch(buf, idx):
    t = torch.from_numpy(buf.copy())
    ix = torch.from_numpy(idx.astype(np.int64))
    if t.dim() == 4:
        ix = ix.unsqueeze(-1).expand(-1, -1, -1, t.shape[-1])
    return t.gather(2, ix).numpy()


def test_insert_is_scatter_and_round_trips():
    x = _inputs(2, 4, 2, 8, 40, 9, seed=21, dtype="bf16")
    out, lse, w = oracle.sdpa_chunk(*_args(x), x["scale"])
    acc = oracle.accumulate_scores(x["scores"], w)
    kc, vc, sc, tp, e = oracle.evict_insert(x["k_cache"], x["v_cache"], acc, x["token_pos"],
                                            x["k_new"], x["v_new"], w, 9, int(x["pos0"]))
    np.testing.assert_array_equal(e, P.brute_bottomk(acc, 9))
    np.testing.assert_array_equal(kc, _scatter_torch(x["k_cache"], e, x["k_new"]))
    np.testing.assert_array_equal(vc, _scatter_torch(x["v_cache"], e, x["v_new"]))
    # inverse recurrence: keys = scatter(keys', index, gather(keys, index))
    delta = _gather_torch(x["k_cache"], e)
    np.testing.assert_array_equal(_scatter_torch(kc, e, delta), x["k_cache"])
    # untouched slots keep their accumulated score; inserted ones start at w[M+i]
    newsc = w[..., 40:].astype(np.float32)
    np.testing.assert_array_equal(sc, _scatter_torch(acc, e, newsc))
    np.testing.assert_array_equal(
        tp, _scatter_torch(x["token_pos"], e,
                           np.broadcast_to(int(x["pos0"]) + np.arange(9, dtype=np.int32),
                                           (2, 2, 9)).copy()))
    lhs = sc.astype(np.float64).sum(axis=-1)
    rhs = (acc.astype(np.float64).sum(axis=-1)
           - np.take_along_axis(acc, e, -1).astype(np.float64).sum(axis=-1)
           + newsc.astype(np.float64).sum(axis=-1))
    np.testing.assert_allclose(lhs, rhs, rtol=1e-12)


def test_insert_requires_k_equal_T():
    x = _inputs(1, 2, 1, 4, 10, 3, seed=1)
    _, _, w = oracle.sdpa_chunk(*_args(x), x["scale"])
    with pytest.raises(ValueError):
        oracle.evict_insert(x["k_cache"], x["v_cache"], x["scores"], None,
                            x["k_new"], x["v_new"], w, 2, 10)


def test_decode_trajectory_runs_step_by_step():
    w = W.custom(B=1, Hq=4, Hkv=2, d=8, M=12, T=1, dtype="bf16", heavy_frac=0.1, steps=4)
    x = W.make_inputs(w, 2)
    res = oracle.decode(x["k_cache"], x["v_cache"], x["scores"], x["token_pos"],
                        x["q_steps"], x["k_new_steps"], x["v_new_steps"], int(x["pos0"]),
                        x["scale"])
    assert len(res) == 4
    for s, r in enumerate(res):
        np.testing.assert_allclose(r["wsum"].sum(-1), 2.0, rtol=1e-13)   # T*G = 1*2
        for b, h in np.ndindex(1, 2):
            slot = r["evict_idx"][b, h, 0]
            assert r["token_pos"][b, h, slot] == int(x["pos0"]) + s
            np.testing.assert_array_equal(r["k_cache"][b, h, slot], x["k_new_steps"][s, b, h, 0])


# ------------------------------------------------------- planted mistakes
def _pin_failures(monkeypatch_ctx):
    """Run a small battery of pins; return the names of those that fail."""
    fails = []
    x = _inputs(1, 4, 2, 6, 9, 4, seed=31, dtype="bf16", heavy=0.2)
    try:
        o, l, w = oracle.sdpa_chunk(*_args(x), x["scale"])
        bo, bl, bw = P.brute_sdpa(*_args(x), x["scale"])
        if not (np.allclose(o, bo, rtol=1e-10, atol=1e-12) and np.allclose(l, bl, rtol=1e-10)
                and np.allclose(w, bw, rtol=1e-10, atol=1e-12)):
            fails.append("brute")
        if not np.allclose(w.sum(-1), 4 * 2, rtol=1e-12):
            fails.append("rowsum")
    except Exception:
        fails.append("attention-crash")
    s = np.floor(np.random.default_rng(3).standard_exponential((2, 30)) * 4).astype(np.float32) / 4
    try:
        if not np.array_equal(oracle.bottomk(s, 9), P.brute_bottomk(s, 9)):
            fails.append("bottomk")
    except Exception:
        fails.append("bottomk-crash")
    return fails


def test_planted_mistakes_are_caught(monkeypatch):
    assert _pin_failures(None) == []
    mutants = {}

    def off_by_one(M, T):                    # chunk key t visible only for t < i
        i = np.arange(T)[:, None]
        j = np.arange(M + T)[None, :]
        return (j < M) | ((j - M) < i)
    mutants["mask off by one"] = ("visible", off_by_one)

    def head_drop_max(Qh, K, V, allowed, scale):   # lse missing its max term
        A = np.where(allowed, scale * (Qh @ K.T), -np.inf)
        amax = A.max(axis=1, keepdims=True)
        lam = np.log(np.exp(A - amax).sum(axis=1))
        Mw = np.exp(A - lam[:, None])
        return Mw @ V, lam, Mw.sum(axis=0)
    mutants["dropped max in lse"] = ("_head", head_drop_max)

    def head_no_scale(Qh, K, V, allowed, scale):   # forgot d^-1/2
        return O.__dict__["_orig_head"](Qh, K, V, allowed, 1.0)
    mutants["missing scale"] = ("_head", head_no_scale)

    def head_transposed_sum(Qh, K, V, allowed, scale):   # sums over keys, not queries
        Y, lam, col = O.__dict__["_orig_head"](Qh, K, V, allowed, scale)
        A = np.where(allowed, scale * (Qh @ K.T), -np.inf)
        Mw = np.exp(A - lam[:, None])
        s = np.zeros_like(col)
        s[:Mw.shape[0]] = Mw.sum(axis=1)
        return Y, lam, s
    mutants["summed along the wrong axis"] = ("_head", head_transposed_sum)

    def bottomk_largest(scores, k):
        return O.__dict__["_orig_bottomk"](-np.asarray(scores, np.float32), k)
    mutants["evicts largest"] = ("bottomk", bottomk_largest)

    def bottomk_high_index_ties(scores, k):
        s = np.asarray(scores, np.float32)
        M = s.shape[-1]
        out = []
        for row in s.reshape(-1, M):
            order = np.lexsort((-np.arange(M), row))
            out.append(np.sort(order[:k]))
        return np.array(out, np.int32).reshape(*s.shape[:-1], k)
    mutants["ties evict higher slot"] = ("bottomk", bottomk_high_index_ties)

    monkeypatch.setitem(O.__dict__, "_orig_head", O._head)
    monkeypatch.setitem(O.__dict__, "_orig_bottomk", O.bottomk)
    for name, (attr, fn) in mutants.items():
        with monkeypatch.context() as m:
            m.setattr(O, attr, fn)
            if attr == "bottomk":
                m.setattr(oracle, "bottomk", fn)
            fails = _pin_failures(None)
        assert fails, f"planted mistake not caught: {name}"

    # a wrong GQA head mapping (strided instead of contiguous) is caught too
    orig = O.sdpa_chunk

    def strided(q, *a, **k):
        B, Hq, T, d = q.shape
        Hkv = a[0].shape[1]
        G = Hq // Hkv
        perm = np.array([(hq % G) * Hkv + hq // G for hq in range(Hq)])
        o, l, w = orig(q[:, perm], *a, **k)
        return o, l, w
    with monkeypatch.context() as m:
        m.setattr(oracle, "sdpa_chunk", strided)
        assert _pin_failures(None), "strided head mapping not caught"


# ------------------------------------------------------ score variants
def _acc_state(B, H, M, seed, quant=None):
    rng = np.random.default_rng(seed)
    s = rng.standard_exponential((B, H, M)).astype(np.float32)
    if quant is not None:
        s = (np.floor(s * quant) / quant).astype(np.float32)
    tp = rng.integers(0, 1000, size=(B, H, M)).astype(np.int32)
    return s, tp


def test_norm_keys_brute_force():
    """h2o_norm ranks phi / (t - token_pos), one float32 division per slot:
    each key equals the float32 rounding of the exact quotient."""
    s, tp = _acc_state(2, 3, 40, 0)
    t = 1500
    keys = oracle.selection_keys(s, tp, "h2o_norm", t)
    for idx in np.ndindex(s.shape):
        exact = float(s[idx]) / float(t - int(tp[idx]))   # float64: the quotient rounds once more
        assert keys[idx] == np.float32(exact)
    k = 7
    ref = np.sort(np.lexsort((np.arange(40), keys[1, 2].astype(np.float64)))[:k])
    np.testing.assert_array_equal(oracle.bottomk(keys, k)[1, 2], ref)


def test_norm_with_equal_ages_is_h2o():
    """Dividing every score by the same power of two keeps the ranking."""
    s, _ = _acc_state(2, 2, 64, 1, quant=8)
    tp = np.full(s.shape, 100, np.int32)
    a = oracle.bottomk(oracle.selection_keys(s, tp, "h2o_norm", 100 + 16), 9)
    np.testing.assert_array_equal(a, oracle.bottomk(s, 9))


def test_norm_prefers_evicting_old_slots():
    """Two slots with equal scores: the older one (larger age) has the smaller
    normalised score and is evicted first."""
    s = np.ones((1, 1, 4), np.float32)
    tp = np.array([[[50, 10, 60, 40]]], np.int32)
    idx = oracle.bottomk(oracle.selection_keys(s, tp, "h2o_norm", 70), 1)
    assert idx[0, 0, 0] == 1


def test_orig_keys_are_exact_batch_sums():
    """h2o_orig: with scores on a grid of 1/8 the float32 batch sums are exact,
    so they equal integer arithmetic; one slot set serves every batch entry."""
    s, tp = _acc_state(5, 3, 50, 2, quant=8)
    keys = oracle.selection_keys(s, tp, "h2o_orig", 0)
    exact = (np.round(s.astype(np.float64) * 8).astype(np.int64).sum(axis=0)) / 8.0
    np.testing.assert_array_equal(keys.astype(np.float64), exact)
    B, H, M = s.shape
    T = 4
    kc = np.zeros((B, H, M, 8), np.float32)
    kn = np.ones((B, H, T, 8), np.float32)
    w = np.zeros((B, H, M + T))
    *_, idx = oracle.evict_insert(kc, kc, s, tp, kn, kn, w, T, 1000, "h2o_orig")
    for b in range(B):
        np.testing.assert_array_equal(idx[b], oracle.bottomk(keys, T))


def test_orig_with_one_batch_entry_is_h2o():
    s, tp = _acc_state(1, 4, 33, 3)
    np.testing.assert_array_equal(oracle.bottomk(oracle.selection_keys(s, tp, "h2o_orig", 0), 5),
                                  oracle.bottomk(s, 5)[0])


def test_variants_insert_like_h2o():
    """The variants change which slots are evicted, not what is written there:
    new keys/values, the chunk key's own summed weight, token position pos0+i."""
    rng = np.random.default_rng(4)
    B, H, M, T, d = 2, 2, 20, 3, 8
    kc = rng.standard_normal((B, H, M, d)).astype(np.float32)
    vc = rng.standard_normal((B, H, M, d)).astype(np.float32)
    kn = rng.standard_normal((B, H, T, d)).astype(np.float32)
    vn = rng.standard_normal((B, H, T, d)).astype(np.float32)
    s, tp = _acc_state(B, H, M, 5)
    w = rng.random((B, H, M + T))
    for pol in ("h2o_norm", "h2o_orig"):
        kc2, vc2, sc2, tp2, idx = oracle.evict_insert(kc, vc, s, tp, kn, kn * 0 + vn, w, T, 2000, pol)
        for b in range(B):
            for h in range(H):
                e = idx[b, h]
                np.testing.assert_array_equal(kc2[b, h, e], kn[b, h])
                np.testing.assert_array_equal(sc2[b, h, e], w[b, h, M:].astype(np.float32))
                np.testing.assert_array_equal(tp2[b, h, e], 2000 + np.arange(T))
                keep = np.setdiff1d(np.arange(M), e)
                np.testing.assert_array_equal(kc2[b, h, keep], kc[b, h, keep])
                np.testing.assert_array_equal(sc2[b, h, keep], s[b, h, keep])


def test_variant_mistakes_are_caught(monkeypatch):
    """Plausible slips in the variants fail the pins above."""
    orig = O.selection_keys

    def age_off_by_one(scores, token_pos, policy, t):
        if policy == "h2o_norm":
            return orig(scores, token_pos, policy, t + 1)
        return orig(scores, token_pos, policy, t)

    def sum_over_heads(scores, token_pos, policy, t):
        if policy == "h2o_orig":
            s = np.asarray(scores, np.float32)
            return np.broadcast_to(s.sum(axis=1, dtype=np.float32)[:, None], s.shape)[0].copy()
        return orig(scores, token_pos, policy, t)

    for fn, test in ((age_off_by_one, test_norm_keys_brute_force),
                     (sum_over_heads, test_orig_keys_are_exact_batch_sums)):
        with monkeypatch.context() as m:
            m.setattr(O, "selection_keys", fn)
            m.setattr(oracle, "selection_keys", fn)
            with pytest.raises(AssertionError):
                test()


# ------------------------------------------- the paper's order: insert first
def _position_state(B, Hq, Hkv, d, M, T, seed, pos0=500, dtype="f32"):
    """A cache whose slots hold tokens before pos0, except T slots (scattered)
    that hold the chunk at positions pos0 .. pos0+T-1, in slot order."""
    rng = np.random.default_rng(seed)
    x = _inputs(B, Hq, Hkv, d, M, T, seed=seed, dtype=dtype)
    tp = rng.integers(0, pos0, size=(B, Hkv, M)).astype(np.int32)
    ev = np.stack([np.stack([np.sort(rng.choice(M, T, replace=False)) for _ in range(Hkv)])
                   for _ in range(B)])
    kc, vc = x["k_cache"].copy(), x["v_cache"].copy()
    for b in range(B):
        for h in range(Hkv):
            kc[b, h, ev[b, h]] = x["k_new"][b, h]
            vc[b, h, ev[b, h]] = x["v_new"][b, h]
            tp[b, h, ev[b, h]] = pos0 + np.arange(T)
    return x, kc, vc, tp, ev, pos0


@pytest.mark.parametrize("shape", [(1, 2, 1, 4, 6, 2), (2, 4, 2, 5, 9, 3), (1, 3, 3, 8, 5, 5)])
def test_sdpa_cache_brute_force(shape):
    """Brute force with arbitrary (non-monotone, repeated, future) positions,
    including query rows that see no slot at all."""
    B, Hq, Hkv, d, M, T = shape
    rng = np.random.default_rng(sum(shape))
    x = _inputs(*shape, seed=1)
    pos0 = 10
    tp = rng.integers(pos0 - 3, pos0 + T + 2, size=(B, Hkv, M)).astype(np.int32)
    tp[0, 0, :] = pos0 + 1                 # head (0, 0): query 0 sees nothing
    o, l, w = oracle.sdpa_cache(x["q"], x["k_cache"], x["v_cache"], tp, pos0, x["scale"])
    bo, bl, bw = P.brute_sdpa_positions(x["q"], x["k_cache"], x["v_cache"], tp, pos0, x["scale"])
    np.testing.assert_allclose(o, bo, rtol=1e-12, atol=1e-13)
    np.testing.assert_array_equal(np.isneginf(l), np.isneginf(bl))
    fin = np.isfinite(bl)
    np.testing.assert_allclose(l[fin], bl[fin], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(w, bw, rtol=1e-12, atol=1e-13)
    assert np.isneginf(l[0, 0, 0]) and not np.any(o[0, 0, 0])


@pytest.mark.parametrize("shape", [(2, 6, 2, 16, 40, 9), (1, 8, 2, 32, 130, 17)])
def test_sdpa_cache_torch(shape):
    x, kc, vc, tp, _, pos0 = _position_state(*shape, seed=5, dtype="bf16")
    o, l, _ = oracle.sdpa_cache(x["q"], kc, vc, tp, pos0, x["scale"])
    to, tl = P.torch_sdpa_positions(x["q"], kc, vc, tp, pos0, x["scale"])
    np.testing.assert_allclose(o, to, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(l, tl, rtol=1e-13)


@pytest.mark.parametrize("shape", [(1, 2, 1, 8, 12, 3), (2, 8, 2, 16, 50, 7)])
def test_sdpa_cache_is_attention_over_cache_minus_chunk_slots_then_chunk(shape):
    """With the chunk written into slots E and every other slot older than the
    chunk, the position mask is the attend-over-[cache || chunk] rule of
    ``sdpa_chunk`` applied to the slots outside E followed by the chunk: same
    outputs, and the summed weights map slot for slot."""
    B, Hq, Hkv, d, M, T = shape
    x, kc, vc, tp, ev, pos0 = _position_state(*shape, seed=9)
    o, l, w = oracle.sdpa_cache(x["q"], kc, vc, tp, pos0, x["scale"])
    for b in range(B):
        for h in range(Hkv):
            keep = np.setdiff1d(np.arange(M), ev[b, h])
            sub = lambda a: a[b:b + 1, h:h + 1]
            G = Hq // Hkv
            qs = x["q"][b:b + 1, h * G:(h + 1) * G]
            co, cl, cw = oracle.sdpa_chunk(qs, sub(kc)[:, :, keep], sub(vc)[:, :, keep],
                                           sub(x["k_new"]), sub(x["v_new"]), x["scale"])
            np.testing.assert_allclose(o[b, h * G:(h + 1) * G], co[0], rtol=1e-12, atol=1e-13)
            np.testing.assert_allclose(l[b, h * G:(h + 1) * G], cl[0], rtol=1e-13)
            np.testing.assert_allclose(w[b, h, keep], cw[0, 0, :len(keep)], rtol=1e-12,
                                       atol=1e-14)
            np.testing.assert_allclose(w[b, h, ev[b, h]], cw[0, 0, len(keep):], rtol=1e-12,
                                       atol=1e-14)


def test_sdpa_cache_slot_permutation():
    x, kc, vc, tp, _, pos0 = _position_state(2, 4, 2, 8, 20, 4, seed=2)
    perm = np.random.default_rng(0).permutation(20)
    o, l, w = oracle.sdpa_cache(x["q"], kc, vc, tp, pos0, x["scale"])
    po, pl, pw = oracle.sdpa_cache(x["q"], kc[:, :, perm], vc[:, :, perm], tp[:, :, perm], pos0,
                                   x["scale"])
    np.testing.assert_allclose(po, o, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(pl, l, rtol=1e-13)
    np.testing.assert_allclose(pw, w[:, :, perm], rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("policy", ["h2o", "h2o_norm", "h2o_orig"])
def test_insert_first_step_bookkeeping(policy):
    """The evicted slots are the bottom T of the ranking before the chunk
    (t = pos0); they hold the chunk with positions pos0+i and score 0 + their
    own summed weight; all other slots add their summed weight; every query
    sees its own key, so the weights sum to T*G."""
    B, Hq, Hkv, d, M, T = 2, 4, 2, 8, 30, 5
    x = _inputs(B, Hq, Hkv, d, M, T, seed=4)
    rng = np.random.default_rng(4)
    tp = rng.integers(0, 400, size=(B, Hkv, M)).astype(np.int32)
    pos0 = 400
    r = oracle.h2o_step_insert_first(x["k_cache"], x["v_cache"], x["scores"], tp, x["q"],
                                     x["k_new"], x["v_new"], pos0, x["scale"], policy)
    s0 = np.asarray(x["scores"], np.float32)
    if policy == "h2o":
        keys = s0
    elif policy == "h2o_norm":
        keys = (s0 / (pos0 - tp).astype(np.float32)).astype(np.float32)
    else:
        keys = s0.sum(axis=0, dtype=np.float32)[None].repeat(B, 0)
    w32 = r["wsum"].astype(np.float32)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hkv):
            ref = np.sort(np.lexsort((np.arange(M), keys[b, h].astype(np.float64)))[:T])
            e = r["evict_idx"][b, h]
            np.testing.assert_array_equal(e, ref)
            np.testing.assert_array_equal(r["token_pos"][b, h, e], pos0 + np.arange(T))
            np.testing.assert_array_equal(r["k_cache"][b, h, e], x["k_new"][b, h])
            np.testing.assert_array_equal(r["scores"][b, h, e], w32[b, h, e])
            keep = np.setdiff1d(np.arange(M), e)
            np.testing.assert_array_equal(r["scores"][b, h, keep], s0[b, h, keep] + w32[b, h, keep])
            assert abs(r["wsum"][b, h].sum() - T * G) < 1e-11
            # query i sees exactly the slots older than the chunk and chunk keys <= i
            assert np.all(r["wsum"][b, h, e[1:]] <= G * (T - np.arange(1, T)) + 1e-12)


def test_insert_first_mistakes_are_caught(monkeypatch):
    """A strict inequality in the position mask, a shifted P, or scores that are
    not reset when a slot is overwritten, each fail a pin above."""
    orig_vis, orig_step = O.visible_by_position, O.h2o_step_insert_first

    def strict(tp, pos0, T):
        return np.asarray(tp, np.int64)[None, :] < pos0 + np.arange(T)[:, None]

    def shifted(tp, pos0, T):
        return orig_vis(tp, pos0 + 1, T)

    def no_reset(k_cache, v_cache, scores, token_pos, q, k_new, v_new, pos0, scale=None,
                 policy="h2o"):
        r = orig_step(k_cache, v_cache, scores, token_pos, q, k_new, v_new, pos0, scale, policy)
        s = np.asarray(scores, np.float32)
        for b in range(s.shape[0]):
            for h in range(s.shape[1]):
                e = r["evict_idx"][b, h]
                r["scores"][b, h, e] = s[b, h, e] + r["wsum"][b, h, e].astype(np.float32)
        return r

    cases = [("visible_by_position", strict, lambda: test_sdpa_cache_brute_force((1, 2, 1, 4, 6, 2))),
             ("visible_by_position", shifted,
              lambda: test_sdpa_cache_is_attention_over_cache_minus_chunk_slots_then_chunk(
                  (1, 2, 1, 8, 12, 3))),
             ("h2o_step_insert_first", no_reset, lambda: test_insert_first_step_bookkeeping("h2o"))]
    for name, fn, test in cases:
        with monkeypatch.context() as m:
            m.setattr(O, name, fn)
            m.setattr(oracle, name, fn)
            with pytest.raises(AssertionError):
                test()


# ----------------------------------------------- backward and delta encoding
BWD_SHAPES = [(1, 2, 1, 4, 5, 3), (2, 4, 2, 8, 7, 4), (1, 3, 1, 6, 0, 4), (1, 4, 2, 16, 33, 9)]


def _dout(x, seed):
    return np.random.default_rng(seed).standard_normal(x["q"].shape)


@pytest.mark.parametrize("shape", BWD_SHAPES)
def test_backward_matches_torch_autograd(shape):
    x = _inputs(*shape, seed=sum(shape))
    do = _dout(x, 1)
    got = oracle.sdpa_chunk_backward(*_args(x), do, x["scale"])
    ref = P.torch_attention_grads(*_args(x), do, x["scale"])
    for a, r, n in zip(got, ref, ("dq", "dk_cache", "dv_cache", "dk_new", "dv_new")):
        np.testing.assert_allclose(a, r, rtol=1e-11, atol=1e-12, err_msg=n)


def test_backward_cache_mode_matches_torch_autograd():
    B, Hq, Hkv, d, M, T = 2, 4, 2, 8, 12, 3
    x = _inputs(B, Hq, Hkv, d, M, T, seed=3)
    rng = np.random.default_rng(3)
    tp = rng.integers(95, 105, size=(B, Hkv, M)).astype(np.int32)
    tp[:, :, 0] = 100                      # every query sees at least slot 0
    do = _dout(x, 2)
    got = oracle.sdpa_chunk_backward(x["q"], x["k_cache"], x["v_cache"], None, None, do,
                                     x["scale"], token_pos=tp, pos0=100)
    ref = P.torch_attention_grads(x["q"], x["k_cache"], x["v_cache"], None, None, do,
                                  x["scale"], token_pos=tp, pos0=100)
    for a, r in zip(got[:3], ref[:3]):
        np.testing.assert_allclose(a, r, rtol=1e-11, atol=1e-12)
    assert got[3] is None and got[4] is None


def test_backward_finite_differences():
    """Central differences of the forward oracle's loss sum(dout * out)."""
    x = _inputs(1, 2, 1, 3, 3, 2, seed=5)
    do = _dout(x, 5)
    grads = oracle.sdpa_chunk_backward(*_args(x), do, x["scale"])
    names = ("q", "k_cache", "v_cache", "k_new", "v_new")
    loss = lambda xx: float((do * oracle.sdpa_chunk(*_args(xx), x["scale"])[0]).sum())
    h = 1e-6
    for n, gr in zip(names, grads):
        base = {k: np.asarray(v, np.float64) for k, v in x.items() if k in names}
        for idx in np.ndindex(base[n].shape):
            up, dn = dict(x), dict(x)
            up[n] = base[n].copy(); up[n][idx] += h
            dn[n] = base[n].copy(); dn[n][idx] -= h
            fd = (loss(up) - loss(dn)) / (2 * h)
            assert abs(fd - gr[idx]) <= 1e-6 * max(1.0, abs(fd)), (n, idx, fd, gr[idx])


@pytest.mark.parametrize("shape", BWD_SHAPES)
def test_backward_invariants(shape):
    """Softmax is invariant to a common shift of a row's scores, so the key
    gradients of a KV head sum to zero; the weights of a row sum to one, so the
    value gradients sum to the sum of the output gradients of the group."""
    B, Hq, Hkv, d, M, T = shape
    x = _inputs(*shape, seed=7)
    do = _dout(x, 7)
    dq, dkc, dvc, dkn, dvn = oracle.sdpa_chunk_backward(*_args(x), do, x["scale"])
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hkv):
            sk = dkc[b, h].sum(0) + dkn[b, h].sum(0)
            assert np.abs(sk).max() < 1e-12
            sv = dvc[b, h].sum(0) + dvn[b, h].sum(0)
            np.testing.assert_allclose(sv, do[b, h * G:(h + 1) * G].sum((0, 1)), rtol=1e-12,
                                       atol=1e-12)


def test_kv_delta_round_trip():
    """The recurrence of the KV buffers and its inverse (Eq. recurrence-reverse):
    keys' = scatter(keys, index, new) and keys = scatter(keys', index,
    gather(keys, index)), bit for bit."""
    rng = np.random.default_rng(0)
    B, H, M, k, d = 2, 3, 40, 7, 8
    keys = rng.standard_normal((B, H, M, d)).astype(np.float32)
    new = rng.standard_normal((B, H, k, d)).astype(np.float32)
    idx = np.stack([np.stack([np.sort(rng.choice(M, k, replace=False)) for _ in range(H)])
                    for _ in range(B)]).astype(np.int32)
    delta = oracle.kv_gather(keys, idx)
    after = oracle.kv_scatter(keys, idx, new)
    np.testing.assert_array_equal(oracle.kv_gather(after, idx), new)
    np.testing.assert_array_equal(oracle.kv_scatter(after, idx, delta), keys)
    # the same as torch's gather/scatter along the slot axis
    np.testing.assert_array_equal(_gather_torch(keys, idx), delta)
    np.testing.assert_array_equal(_scatter_torch(keys, idx, new), after)


def test_backward_mistakes_are_caught(monkeypatch):
    orig = O._head_backward

    def no_centering(Qh, K, V, allowed, scale, dO):
        A = np.where(allowed, scale * (Qh @ K.T), -np.inf)
        Pm = np.exp(A - A.max(1, keepdims=True)); Pm /= Pm.sum(1, keepdims=True)
        dA = Pm * (dO @ V.T)                           # missing the - <p, g> term
        return scale * dA @ K, scale * dA.T @ Qh, Pm.T @ dO

    def no_scale_dk(Qh, K, V, allowed, scale, dO):
        dQ, dK, dV = orig(Qh, K, V, allowed, scale, dO)
        return dQ, dK / scale, dV

    for fn in (no_centering, no_scale_dk):
        with monkeypatch.context() as m:
            m.setattr(O, "_head_backward", fn)
            with pytest.raises(AssertionError):
                test_backward_matches_torch_autograd((2, 4, 2, 8, 7, 4))


# --------------------------------------------- the step's wiring, worked by hand
# One-hot keys make every logit a chosen number: with key j = e_j, scale 1 and
# query i = (ln a_i0, ln a_i1, ...), the logit of (i, j) is ln a_ij, so the
# softmax weights are a_ij / sum_j' a_ij' (exact rationals) and everything the
# step computes can be written down with fractions. Rows are chosen to sum to
# powers of two, so every weight and score below is exact in float32.
def _onehot_case():
    """B1 Hq2 Hkv1 (G2), M5, T2, d7: integer weights a[g, i, j] over the keys
    row i sees (cache slots 0..4, chunk key t <= i); prior scores S0; values
    V[j] = j + 1 (cache) and 10 + t (chunk keys)."""
    M, T, G = 5, 2, 2
    a = {
        (0, 0): [1, 1, 1, 1, 2, 2],
        (0, 1): [2, 1, 1, 1, 1, 1, 1],
        (1, 0): [1, 2, 1, 1, 1, 2],
        (1, 1): [8, 1, 1, 1, 1, 2, 2],
    }
    d = M + T
    q = np.zeros((1, G, T, d))
    for (g, i), row in a.items():
        q[0, g, i, :len(row)] = np.log(np.array(row, np.float64))
    keys = np.eye(d)
    kc, kn = keys[None, None, :M], keys[None, None, M:]
    vc = np.arange(1, M + 1, dtype=np.float64)[None, None, :, None] * np.ones((1, 1, M, d))
    vn = (10 + np.arange(T, dtype=np.float64))[None, None, :, None] * np.ones((1, 1, T, d))
    s0 = np.array([[[0.0625, 1.0, 0.75, 0.5, 0.25]]], np.float32)
    tp = np.array([[[7, 3, 9, 1, 4]]], np.int32)
    return dict(a=a, M=M, T=T, G=G, q=q, kc=kc, vc=vc, kn=kn, vn=vn, s0=s0, tp=tp, pos0=20)


def _onehot_expected(c):
    """The step's results by exact rational arithmetic (no oracle code)."""
    M, T, G, a = c["M"], c["T"], c["G"], c["a"]
    vals = [Fraction(j + 1) for j in range(M)] + [Fraction(10 + t) for t in range(T)]
    w = [Fraction(0)] * (M + T)
    out = np.zeros((G, T))
    lse = np.zeros((G, T))
    for (g, i), row in a.items():
        Z = sum(Fraction(x) for x in row)
        lse[g, i] = float(np.log(float(Z)))
        out[g, i] = float(sum(Fraction(x) / Z * vals[j] for j, x in enumerate(row)))
        for j, x in enumerate(row):
            w[j] += Fraction(x) / Z
    acc = [Fraction(float(c["s0"][0, 0, j])) + w[j] for j in range(M)]
    # bottom-T by (score, slot), ascending slots
    evict = sorted(sorted(range(M), key=lambda j: (acc[j], j))[:T])
    scores = [float(x) for x in acc]
    tp = [int(x) for x in c["tp"][0, 0]]
    for i, e in enumerate(evict):
        scores[e] = float(w[M + i])
        tp[e] = c["pos0"] + i
    return dict(w=[float(x) for x in w], acc=[float(x) for x in acc], evict=evict,
                scores=scores, tp=tp, out=out, lse=lse)


def _check_onehot_step(step_fn):
    """Runs ``step_fn`` (oracle.h2o_step's signature) on the worked case and
    compares with the exact results; returns the list of what differs."""
    c = _onehot_case()
    e = _onehot_expected(c)
    r = step_fn(c["kc"], c["vc"], c["s0"], c["tp"], c["q"], c["kn"], c["vn"], c["pos0"], 1.0)
    bad = []
    if not np.allclose(r["wsum"][0, 0], e["w"], rtol=1e-14, atol=0):
        bad.append("wsum")
    if not np.array_equal(np.asarray(r["scores_acc"])[0, 0], np.float32(e["acc"])):
        bad.append("accumulated scores")
    if not np.array_equal(r["evict_idx"][0, 0], e["evict"]):
        bad.append("evicted slots")
    if not np.array_equal(np.asarray(r["scores"])[0, 0], np.float32(e["scores"])):
        bad.append("scores after the insert")
    if not np.array_equal(r["token_pos"][0, 0], e["tp"]):
        bad.append("token positions")
    kc_new = np.array(c["kc"], copy=True)
    for i, slot in enumerate(e["evict"]):
        kc_new[0, 0, slot] = c["kn"][0, 0, i]
    if not np.array_equal(r["k_cache"], kc_new):
        bad.append("inserted keys")
    if not (np.allclose(r["out"][0, :, :, 0], e["out"], rtol=1e-14)
            and np.allclose(r["lse"][0], e["lse"], rtol=1e-14)):
        bad.append("out/lse")
    return bad


def test_step_worked_example_exact():
    """h2o_step on the worked case equals exact rational arithmetic: wsum
    sums each key's weight over both query heads and both queries (the chunk
    keys only over the queries that see them), the accumulated scores are
    S0 + wsum (Eq. h2o-score), the eviction is the bottom-2 of the
    *accumulated* scores - here {3, 4}, while the prior scores alone would
    evict {0, 4} - and chunk key i lands in the i-th smallest evicted slot
    with score wsum[M+i] (its own column sum) and position pos0 + i."""
    e = _onehot_expected(_onehot_case())
    assert e["evict"] == [3, 4]
    assert e["w"] == [1.0, 9 / 16, 7 / 16, 7 / 16, 9 / 16, 12 / 16, 4 / 16]
    assert e["scores"] == [1.0625, 1.5625, 1.1875, 0.75, 0.25]
    assert sum(e["w"]) == 4.0                     # T * G: every row sums to one
    assert _check_onehot_step(oracle.h2o_step) == []


def test_step_wiring_mistakes_are_caught(monkeypatch):
    """Mistakes in how h2o_step wires its parts fail the worked example."""
    orig_step = O.h2o_step

    def rank_prior(k_cache, v_cache, scores, token_pos, q, k_new, v_new, pos0, scale=None,
                   policy="h2o"):
        # ranks the scores before the chunk's weights are added
        out, lse, wsum = O.sdpa_chunk(q, k_cache, v_cache, k_new, v_new, scale)
        acc = O.accumulate_scores(scores, wsum)
        T = q.shape[2]
        idx = O.bottomk(scores, T)
        kc, vc = k_cache.copy(), v_cache.copy()
        sc, tp = acc.copy(), token_pos.copy()
        M = sc.shape[-1]
        for i, e in enumerate(idx[0, 0]):
            kc[0, 0, e] = k_new[0, 0, i]
            vc[0, 0, e] = v_new[0, 0, i]
            sc[0, 0, e] = np.float32(wsum[0, 0, M + i])
            tp[0, 0, e] = pos0 + i
        return dict(out=out, lse=lse, wsum=wsum, scores_acc=acc, evict_idx=idx, k_cache=kc,
                    v_cache=vc, scores=sc, token_pos=tp)

    def with_insert(mutate):
        def step(*a, **k):
            r = orig_step(*a, **k)
            mutate(r, a)
            return r
        return step

    def insert_zero(r, a):          # new slots start from 0
        for i, e in enumerate(r["evict_idx"][0, 0]):
            r["scores"][0, 0, e] = 0.0

    def insert_wrong_column(r, a):  # the first chunk columns instead of M + i
        for i, e in enumerate(r["evict_idx"][0, 0]):
            r["scores"][0, 0, e] = np.float32(r["wsum"][0, 0, i])

    def insert_reversed(r, a):      # new key i into the i-th largest evicted slot
        ev = r["evict_idx"][0, 0]
        M = r["scores"].shape[-1]
        for i, e in enumerate(ev[::-1]):
            r["scores"][0, 0, e] = np.float32(r["wsum"][0, 0, M + i])
            r["k_cache"][0, 0, e] = a[5][0, 0, i]

    def keep_prior_scores(r, a):    # the kept slots not accumulated
        keep = np.setdiff1d(np.arange(r["scores"].shape[-1]), r["evict_idx"][0, 0])
        r["scores"][0, 0, keep] = np.asarray(a[2], np.float32)[0, 0, keep]

    for name, fn in [("ranks prior scores", rank_prior),
                     ("inserted score 0", with_insert(insert_zero)),
                     ("inserted score from the wrong column", with_insert(insert_wrong_column)),
                     ("new keys in reversed slots", with_insert(insert_reversed)),
                     ("kept scores not accumulated", with_insert(keep_prior_scores))]:
        assert _check_onehot_step(fn), f"planted wiring mistake not caught: {name}"


def test_decode_threads_state_exact():
    """Two single-token steps by hand (one-hot keys, G1, M3): step 1 evicts
    slot 2 and writes key e3 there with score 1/2; step 2 must attend over that
    new state (e3 in slot 2) and, with slots 1 and 2 tied at 3/4, evict the
    lower slot 1. oracle.decode must thread the state from step to step."""
    d = 5
    keys = np.eye(d)
    kc = keys[None, None, :3].copy()
    vc = np.ones((1, 1, 3, d))
    s0 = np.array([[[0.5, 0.5, 0.25]]], np.float32)
    tp = np.array([[[0, 1, 2]]], np.int32)
    # step 1 sees e0 e1 e2 | e3 with weights 2 1 1 | 4 (sum 8)
    # step 2 sees e0 e1 e3 | e4 with weights 1 1 2 | 4 (sum 8); e2 is gone
    q1 = np.log(np.array([2, 1, 1, 4, 1], np.float64))
    q2 = np.log(np.array([1, 1, 1, 2, 4], np.float64))
    qs = np.stack([q1, q2])[:, None, None, None, :]
    kns = np.stack([keys[3], keys[4]])[:, None, None, None, :]
    vns = np.ones((2, 1, 1, 1, d))
    res = oracle.decode(kc, vc, s0, tp, qs, kns, vns, 3, 1.0)
    np.testing.assert_allclose(res[0]["wsum"][0, 0], [0.25, 0.125, 0.125, 0.5], rtol=1e-14)
    assert res[0]["evict_idx"][0, 0, 0] == 2
    np.testing.assert_array_equal(res[0]["scores"][0, 0], np.float32([0.75, 0.625, 0.5]))
    np.testing.assert_allclose(res[1]["wsum"][0, 0], [0.125, 0.125, 0.25, 0.5], rtol=1e-14)
    assert res[1]["evict_idx"][0, 0, 0] == 1                 # the tie goes to the lower slot
    np.testing.assert_array_equal(res[1]["scores"][0, 0], np.float32([0.875, 0.5, 0.75]))
    np.testing.assert_array_equal(res[1]["token_pos"][0, 0], [0, 4, 3])
    np.testing.assert_array_equal(res[1]["k_cache"][0, 0], keys[[0, 4, 3]])


# ------------------------------------------------- the metrics the gates use
def test_rel_err_hand_computed():
    """||x - ref|| / ||ref|| per slice, maximum over slices: slice 0 differs
    by (0, 0.5) against (3, 4) -> 0.1; slice 1 by (0, 0.2) against (1, 0)
    -> 0.2."""
    ref = np.array([[3.0, 4.0], [1.0, 0.0]])
    x = np.array([[3.0, 4.5], [1.0, 0.2]])
    assert oracle.rel_err(x, ref, axes=(-1,)) == pytest.approx(0.2, rel=1e-15)
    # over both axes: ||(0, .5, 0, .2)|| / ||(3, 4, 1, 0)|| = sqrt(.29 / 26)
    assert oracle.rel_err(x, ref, axes=(-2, -1)) == pytest.approx(np.sqrt(0.29 / 26), rel=1e-15)
    assert oracle.rel_err(ref, ref, axes=(-1,)) == 0.0


def test_elem_err_hand_computed():
    """|x - ref| / (|ref| + floor * max|ref|) per element: (0.5 / 4.000004)
    for the 4.0 entry of slice 0, 0.2 / (0 + 1e-6) for the 0.0 entry of
    slice 1, whose largest |ref| is 1."""
    ref = np.array([[3.0, 4.0], [1.0, 0.0]])
    x = np.array([[3.0, 4.5], [1.0, 2e-7]])
    assert oracle.elem_err(x, ref, axes=(-1,)) == pytest.approx(0.2, rel=1e-12)
    x2 = np.array([[3.0, 4.5], [1.0, 0.0]])
    assert oracle.elem_err(x2, ref, axes=(-1,)) == pytest.approx(0.5 / (4.0 + 4e-6), rel=1e-12)
    assert oracle.elem_err(np.zeros(3), np.zeros(3), axes=(-1,)) == 0.0
    assert oracle.elem_err(np.array([0, 1e-30, 0]), np.zeros(3), axes=(-1,)) == np.inf


def _skewed_head(seed=0):
    """One KV head with heavy hitters (a skewed wsum): the oracle's wsum and
    accumulated scores of B1 Hq4 Hkv1 d64 M2048 T256, 2 % heavy keys."""
    w = W.custom(B=1, Hq=4, Hkv=1, d=64, M=2048, T=256, dtype="bf16", heavy_frac=0.02)
    x = W.make_inputs(w, seed)
    _, _, ws = oracle.sdpa_chunk(*_args(x), x["scale"])
    return x, ws, oracle.accumulate_scores(x["scores"], ws)


def test_normwise_gate_misses_a_zeroed_tile_elementwise_gate_does_not():
    """Zeroing the summed weights of one 32-key tile of ordinary slots (no
    heavy hitter among them) passes a 2e-2 normwise check of the whole row -
    the heavy hitters dominate its norm - but fails the element-by-element
    check at the same tolerance, and changes the eviction."""
    x, ws, acc = _skewed_head()
    row = ws[0, 0, :2048]
    med = np.median(row)
    t0 = next(t for t in range(0, 2048, 32) if row[t:t + 32].max() < 4 * med)
    bad = ws.copy()
    bad[0, 0, t0:t0 + 32] = 0.0
    assert oracle.rel_err(bad, ws, axes=(-1,)) <= 2e-2
    assert oracle.elem_err(bad, ws, axes=(-1,)) > 2e-2
    bad_acc = oracle.accumulate_scores(x["scores"], bad)
    assert not np.array_equal(oracle.bottomk(bad_acc, 256), oracle.bottomk(acc, 256))


def test_eviction_band_accepts_near_ties_and_rejects_far_slots():
    """The band check: the oracle's own set is valid with no differences; a
    set that swaps the k-th slot with the (k+1)-th (a near tie, both inside a
    band of 1e-3 around the k-th score when they are that close) is valid; a
    set that swaps in a slot far above the threshold is not."""
    x, ws, acc = _skewed_head(1)
    k = 256
    s = acc[0, 0].astype(np.float64)
    own = oracle.bottomk(acc, k)[0, 0]
    n_diff, n_band, ok = oracle.eviction_agreement(own, s, k, 1e-3)
    assert (n_diff, ok) == (0, True) and n_band >= 1
    order = np.lexsort((np.arange(len(s)), s))
    # a near tie: the (k+1)-th score set 1e-4 above the k-th; an eviction
    # that takes it instead of the k-th slot is valid at a tolerance of 1e-3
    sn = s.copy()
    sn[order[k]] = s[order[k - 1]] * (1 + 1e-4)
    near = np.sort(np.concatenate([own[own != order[k - 1]], [order[k]]]))
    n_diff, n_band, ok = oracle.eviction_agreement(near, sn, k, 1e-3)
    assert n_diff == 1 and ok and n_band >= 2
    far = np.sort(np.concatenate([own[own != order[k - 1]], [order[-1]]]))   # the largest score
    n_diff, _, ok = oracle.eviction_agreement(far, s, k, 1e-3)
    assert n_diff == 1 and not ok
    # a slot a quarter above the threshold: outside the relative band, but
    # inside an absolute band of 4 * 2e-2 * max score (the heavy hitters
    # make that band wider than the threshold itself)
    tau = s[order[k - 1]]
    j = order[np.searchsorted(s[order], 1.25 * tau)]
    assert 1.2 * tau < s[j] <= tau + 4 * 2e-2 * s.max()
    mid = np.sort(np.concatenate([own[own != order[k - 1]], [j]]))
    n_diff, _, ok = oracle.eviction_agreement(mid, s, k, 1e-3)
    assert n_diff == 1 and not ok
