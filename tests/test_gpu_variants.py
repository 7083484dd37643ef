"""GPU parity of the eviction rankings h2o_norm and h2o_orig (Sec. "Variants
of Heavy-Hitter Oracle") through h2o_evict_insert_policy.

Given the same float32 scores, token positions and summed weights, the
selection and the insert are bit-exact against the oracle: the h2o_norm key
is one correctly rounded float32 division, the h2o_orig key a float32 sum in
increasing b, and both sides rank by (key, slot). The whole step with a
policy is checked the same way on the GPU's own accumulated scores, and its
eviction for validity against the oracle's float64-derived scores.
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

POLICIES = ["h2o", "h2o_norm", "h2o_orig"]
EVICT_SHAPES = [  # B, Hkv, M, T, d, dtype, quant (None: no forced ties)
    (1, 1, 1, 1, 64, "bf16", None),
    (3, 2, 37, 1, 64, "bf16", None),
    (8, 8, 4096, 1, 64, "bf16", 2),
    (2, 4, 300, 64, 128, "f32", None),
    (3, 2, 1000, 100, 64, "bf16", 3),
    (2, 8, 8192, 1024, 128, "bf16", None),
    (5, 1, 33, 33, 64, "f32", 0),
]


def _bits(a, dtype):
    return a if dtype == "f32" else W.bf16_bits_to_f32(W.f32_to_bf16_bits(a))


def _evict_inputs(B, Hkv, M, T, d, dtype, quant, seed):
    """Seeded float32 scores (forced ties and -0.0 when quant is set), token
    positions below pos0 (repeated when quant is set, so h2o_norm ties too),
    summed weights and cache/chunk rows exact in ``dtype``."""
    rng = np.random.Generator(np.random.PCG64(seed))
    f32 = np.float32
    sc = rng.standard_exponential((B, Hkv, M)).astype(f32)
    pos0 = 70000
    if quant is None:
        tp = rng.integers(0, pos0, size=(B, Hkv, M)).astype(np.int32)
    else:
        sc = (np.floor(sc * 2 ** quant) / 2 ** quant).astype(f32)
        sc.reshape(-1)[: min(3, sc.size)] = -0.0
        tp = rng.choice(np.arange(pos0 - 8, pos0, dtype=np.int32), size=(B, Hkv, M))
    x = dict(scores=sc, token_pos=tp, pos0=pos0,
             wsum=rng.standard_exponential((B, Hkv, M + T)).astype(f32))
    for n, r in (("k_cache", M), ("v_cache", M), ("k_new", T), ("v_new", T)):
        x[n] = _bits(rng.standard_normal((B, Hkv, r, d)).astype(f32), dtype)
    return x


def _run_evict(x, T, dtype, policy, with_pos=True):
    tdt = U.TDT[dtype]
    B, Hkv, M = x["scores"].shape
    st = dict(k_cache=U.to_dev(x["k_cache"], tdt), v_cache=U.to_dev(x["v_cache"], tdt),
              scores=U.to_dev(x["scores"], torch.float32),
              token_pos=U.to_dev(x["token_pos"], torch.int32) if with_pos else None)
    kn, vn = U.to_dev(x["k_new"], tdt), U.to_dev(x["v_new"], tdt)
    wsum = U.to_dev(x["wsum"], torch.float32)
    idx = torch.empty(B, Hkv, T, dtype=torch.int32, device=U.DEV)
    nbytes = H.h2o_evict_workspace_bytes(B, Hkv, M, T, policy)
    # a dirty workspace: its contents on entry must not matter
    ws = torch.full((max(nbytes, 16),), 0x7F, dtype=torch.uint8, device=U.DEV)
    H.h2o_evict_insert_policy(st["k_cache"], st["v_cache"], st["scores"], st["token_pos"], kn, vn,
                              wsum, idx, x["pos0"], policy, ws)
    torch.cuda.synchronize()
    out = {n: (None if t is None else U.to_np(t)) for n, t in st.items()}
    out["evict_idx"] = idx.cpu().numpy()
    return out


def _expect(x, T, policy, with_pos=True):
    kc, vc, sc, tp, idx = oracle.evict_insert(
        x["k_cache"], x["v_cache"], x["scores"], x["token_pos"] if with_pos else None,
        x["k_new"], x["v_new"], x["wsum"], T, x["pos0"], policy)
    return dict(k_cache=kc, v_cache=vc, scores=sc, token_pos=tp, evict_idx=idx)


def _assert_same(got, exp, tag):
    for n, e in exp.items():
        if e is None:
            assert got[n] is None, n
            continue
        np.testing.assert_array_equal(got[n], np.asarray(e, dtype=got[n].dtype),
                                      err_msg=f"{tag} {n}")


@pytest.mark.parametrize("policy", POLICIES)
@pytest.mark.parametrize("shape", EVICT_SHAPES)
def test_evict_policy_bit_exact(shape, policy):
    B, Hkv, M, T, d, dt, quant = shape
    say(f"evict {policy} B{B} Hkv{Hkv} M{M} T{T} d{d} {dt} quant {quant}")
    x = _evict_inputs(B, Hkv, M, T, d, dt, quant, seed=B * M + T)
    _assert_same(_run_evict(x, T, dt, policy), _expect(x, T, policy), policy)


@pytest.mark.parametrize("policy", ["h2o", "h2o_orig"])
def test_evict_policy_without_positions(policy):
    """token_pos is optional for the rankings that do not read it."""
    B, Hkv, M, T, d, dt = 3, 2, 500, 4, 64, "bf16"
    say(f"evict {policy} without token_pos")
    x = _evict_inputs(B, Hkv, M, T, d, dt, 1, seed=3)
    _assert_same(_run_evict(x, T, dt, policy, with_pos=False),
                 _expect(x, T, policy, with_pos=False), policy)


def test_policy_h2o_equals_evict_insert():
    """H2O_POLICY_H2O is h2o_evict_insert, bit for bit."""
    B, Hkv, M, T, d, dt = 2, 4, 700, 64, 128, "bf16"
    say("policy h2o vs h2o_evict_insert")
    x = _evict_inputs(B, Hkv, M, T, d, dt, 2, seed=9)
    got = _run_evict(x, T, dt, "h2o")
    tdt = U.TDT[dt]
    st = U.device_state(dict(x, q=None), dt)
    idx = torch.empty(B, Hkv, T, dtype=torch.int32, device=U.DEV)
    H.h2o_evict_insert(st["k_cache"], st["v_cache"], st["scores"], st["token_pos"],
                       U.to_dev(x["k_new"], tdt), U.to_dev(x["v_new"], tdt),
                       U.to_dev(x["wsum"], torch.float32), idx, x["pos0"])
    torch.cuda.synchronize()
    ref = {n: U.to_np(t) for n, t in st.items()}
    ref["evict_idx"] = idx.cpu().numpy()
    _assert_same(got, ref, "h2o")


def test_orig_sets_agree_over_batch():
    """h2o_orig evicts one slot set per kv head, the same for every b."""
    B, Hkv, M, T = 4, 3, 2048, 16
    say("orig: one slot set per head")
    x = _evict_inputs(B, Hkv, M, T, 64, "bf16", None, seed=21)
    idx = _run_evict(x, T, "bf16", "h2o_orig")["evict_idx"]
    assert (idx == idx[:1]).all()
    assert (np.diff(idx, axis=-1) > 0).all()


STEP_SHAPES = [  # B, Hq, Hkv, d, M, T, dtype
    (8, 32, 8, 64, 4096, 1, "bf16"),
    (2, 8, 2, 128, 700, 64, "bf16"),
    (2, 4, 2, 64, 300, 32, "f32"),
]


@pytest.mark.parametrize("policy", ["h2o_norm", "h2o_orig"])
@pytest.mark.parametrize("shape", STEP_SHAPES)
def test_step_with_policy(shape, policy):
    """A whole chunk step ranking by ``policy``: attention within tolerance of
    the oracle; eviction and insert bit-exact against the oracle run on the
    GPU's own accumulated scores; the evicted keys valid against the oracle's
    keys (Q15-style margin: near-ties only may differ)."""
    B, Hq, Hkv, d, M, T, dt = shape
    wl = W.custom("variant", B=B, Hq=Hq, Hkv=Hkv, d=d, M=M, T=T, dtype=dt, heavy_frac=0.02,
                  age_decay=8192.0)
    say(f"step {policy} {wl.describe()}")
    x = W.make_inputs(wl, seed=17)
    tdt = U.TDT[dt]
    q, kn, vn = (U.to_dev(x[n], tdt) for n in ("q", "k_new", "v_new"))
    st = U.device_state(x, dt)
    bufs = H.alloc_step(B, Hq, Hkv, T, M, d, tdt, policy=policy)
    pos0 = int(x["pos0"])
    H.step(st, q, kn, vn, bufs, pos0, float(x["scale"]), policy=policy)
    torch.cuda.synchronize()
    g_w = U.to_np(bufs["wsum"])
    o_out, o_lse, o_w = oracle.sdpa_chunk(x["q"], x["k_cache"], x["v_cache"], x["k_new"],
                                          x["v_new"], float(x["scale"]))
    U.check(dt, out=(U.to_np(bufs["out"]), o_out), wsum=(g_w, o_w))
    g_acc = oracle.accumulate_scores(x["scores"], g_w)
    kc, vc, sc, tp, idx = oracle.evict_insert(x["k_cache"], x["v_cache"], g_acc, x["token_pos"],
                                              x["k_new"], x["v_new"], g_w, T, pos0, policy)
    got = {n: U.to_np(st[n]) for n in ("k_cache", "v_cache", "scores", "token_pos")}
    got["evict_idx"] = bufs["evict_idx"].cpu().numpy()
    _assert_same(got, dict(k_cache=kc, v_cache=vc, scores=sc, token_pos=tp, evict_idx=idx),
                 policy)
    # against the oracle's own ranking: only near-ties may differ (the keys
    # are the scores divided by an exact age, or batch sums of non-negative
    # scores, so they carry the scores' relative error bound)
    o_keys = oracle.selection_keys(oracle.accumulate_scores(x["scores"], o_w), x["token_pos"],
                                   policy, pos0 + T)
    g_keys = oracle.selection_keys(g_acc, x["token_pos"], policy, pos0 + T)
    assert oracle.elem_err(g_keys, o_keys, (-1,)) <= U.SEL_TOL
    g_idx = got["evict_idx"][0] if policy == "h2o_orig" else got["evict_idx"]
    n_diff = 0
    for r, e in zip(o_keys.reshape(-1, M), g_idx.reshape(-1, T)):
        nd, _, ok = oracle.eviction_agreement(e, r, T, U.SEL_TOL)
        assert ok, "eviction outside the band around the oracle's k-th key"
        n_diff += nd
    say(f"  {n_diff} evicted slots differ from the oracle's (each inside the band)")
