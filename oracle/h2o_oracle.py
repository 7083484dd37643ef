"""Float64 CPU oracle for the H2O chunk step.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module. The HIP library
never calls it and shares no code with it.

What it computes is the plain definition of each step, one attention head at a
time, with numpy float64 matrix products as the only library primitive:

1. SDPA of the chunk's T queries against [cache keys || chunk keys]
   (Sec. "Sparse Attention. Key-Value Caching", Eq. main-sdpa and
   Eq. main-sdpa-comp): ``A = d^-1/2 Q K^T`` masked, ``M = softmax(A)`` along
   keys, ``Y = M V``. Every cache token precedes the chunk, so a query sees all
   cache slots; chunk key t is visible to chunk query i iff t <= i (the causal
   rule of Sec. "Discussion: SDPA Kernels for Sparse Attention").
2. The log-sum-exp of each query row, lambda = log(exp(A) 1)
   (Sec. "FlashAttention for Summed Attention Weights").
3. Summed attention weights sum_i m_{i,j} per key (Sec. "Variants of
   Heavy-Hitter Oracle", the H2O score increment; Sec. "Computing Summed
   Attention Weights in SDPA"), additionally summed over the q_g query heads
   that share one KV head (GQA, Sec. "Sparse Attention. Key-Value Caching"),
   because the score and the eviction are per KV head.
4. Score accumulation phi <- phi + sum_i m_{i,j} (Eq. h2o-score as a running
   sum over chunks), held in float32 storage: one IEEE float32 addition.
5. Eviction: per (b, kv-head), the k slots with the smallest score
   (Sec. "Variants of Heavy-Hitter Oracle"), ties broken by the lower slot
   index, returned in ascending slot order; or the ranking of one of the
   paper's two variants of the score, normalised by age (h2o_norm) or
   summed over the batch (h2o_orig).
6. Insert: scatter of the chunk's keys/values into the evicted slots along the
   slot axis (Sec. "Fine-Tuning for Sparse Attention", the linear recurrence;
   Sec. "Buffer Read/Write Access by torch.scatter, torch.gather"); new key i
   goes to the i-th smallest evicted slot, its score starts at its own summed
   weight from this chunk, its token position is pos0 + i.

The paper's own ordering of a chunk step (Sec. "Discussion: SDPA Kernels for
Sparse Attention") writes the chunk into the cache first and masks by token
position: ``sdpa_cache`` and ``h2o_step_insert_first`` below compute that
variant by the same plain definitions.

Readings of points the paper leaves open are listed in the repository's design
notes; the ones that change results are repeated at the functions below.
"""
from __future__ import annotations

from typing import Iterable, Optional, Sequence, Tuple

import numpy as np

F64 = np.float64


# ----------------------------------------------------------------- step 1: mask
def visible(M: int, T: int) -> np.ndarray:
    """Boolean [T, M+T]: may chunk query i attend key column j?

    Columns j < M are cache slots (all tokens precede the chunk: always
    visible). Column M+t is chunk key t, visible iff t <= i: the mask
    -inf * 1{P + i < t(j)} with t(j) = P + t.
    """
    i = np.arange(T)[:, None]
    j = np.arange(M + T)[None, :]
    return (j < M) | ((j - M) <= i)


# --------------------------------------------------------- steps 1-3 per head
def _head(Qh: np.ndarray, K: np.ndarray, V: np.ndarray, allowed: np.ndarray,
          scale: float) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """One query head: returns (Y [T,d], lambda [T], column sums [M+T])."""
    A = scale * (Qh @ K.T)                         # d^-1/2 Q K^T
    A = np.where(allowed, A, -np.inf)              # mask
    amax = A.max(axis=1, keepdims=True)            # finite: every row sees the cache
    lam = amax[:, 0] + np.log(np.exp(A - amax).sum(axis=1))
    Mw = np.exp(A - lam[:, None])                  # softmax rows; masked -> 0
    Y = Mw @ V
    return Y, lam, Mw.sum(axis=0)


def sdpa_chunk(q, k_cache, v_cache, k_new, v_new, scale: Optional[float] = None,
               heads: Optional[Iterable[Tuple[int, int]]] = None):
    """Attention of the chunk over [cache || chunk] with summed weights.

    Shapes: q [B,Hq,T,d]; k_cache, v_cache [B,Hkv,M,d]; k_new, v_new [B,Hkv,T,d].
    Query head hq uses KV head hq // (Hq/Hkv).

    Returns float64 (out [B,Hq,T,d], lse [B,Hq,T], wsum [B,Hkv,M+T]) where
    ``wsum[b,h,j] = sum over the group's query heads g and queries i of
    m^{(g)}_{i,j}``. With ``heads`` (a list of (b, kv-head)) only those heads
    are computed; the other entries are NaN.
    """
    q = np.asarray(q)
    B, Hq, T, d = q.shape
    Hkv, M = k_cache.shape[1], k_cache.shape[2]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    scale = float(scale)
    allowed = visible(M, T)
    out = np.full((B, Hq, T, d), np.nan, F64)
    lse = np.full((B, Hq, T), np.nan, F64)
    wsum = np.full((B, Hkv, M + T), np.nan, F64)
    if heads is None:
        heads = [(b, h) for b in range(B) for h in range(Hkv)]
    for b, h in heads:
        K = np.concatenate([k_cache[b, h], k_new[b, h]]).astype(F64)
        V = np.concatenate([v_cache[b, h], v_new[b, h]]).astype(F64)
        acc = np.zeros(M + T, F64)
        for g in range(G):
            hq = h * G + g
            Y, lam, col = _head(q[b, hq].astype(F64), K, V, allowed, scale)
            out[b, hq] = Y
            lse[b, hq] = lam
            acc += col
        wsum[b, h] = acc
    return out, lse, wsum


# ------------------------------------------------------------ step 4: scores
def accumulate_scores(scores, wsum) -> np.ndarray:
    """phi <- phi + summed weights of this chunk, for the M cache slots.

    Scores are stored in float32 and the update is one IEEE float32 addition
    of the stored score and the float32 value of the summed weight.
    """
    scores = np.asarray(scores, np.float32)
    M = scores.shape[-1]
    return scores + np.asarray(wsum)[..., :M].astype(np.float32)


# ---------------------------------------------------------- step 5: eviction
def bottomk(scores, k: int) -> np.ndarray:
    """Indices of the k smallest scores per row (last axis), ascending slots.

    Order is lexicographic on (score, slot): at equal scores the lower slot is
    evicted first. -0.0 and +0.0 compare equal. Scores must not be NaN.
    """
    s = np.asarray(scores, np.float32)
    lead, M = s.shape[:-1], s.shape[-1]
    if not 0 <= k <= M:
        raise ValueError("need 0 <= k <= M")
    flat = s.reshape(-1, M)
    res = np.empty((flat.shape[0], k), np.int32)
    slots = np.arange(M)
    for r in range(flat.shape[0]):
        row = flat[r].astype(F64) + 0.0                  # -0.0 -> +0.0
        order = np.lexsort((slots, row))                 # primary key: score
        res[r] = np.sort(order[:k])
    return res.reshape(*lead, k)


# ------------------------------------------------- the H2O score variants
POLICIES = ("h2o", "h2o_norm", "h2o_orig")


def selection_keys(scores, token_pos, policy: str, t: int) -> np.ndarray:
    """The float32 vector the eviction ranks, from the accumulated float32
    scores phi(b, h, j) (Sec. "Variants of Heavy-Hitter Oracle"):

      h2o       phi itself, per (b, kv-head)                        [B, H, M]
      h2o_norm  phi / (t - token_pos): the score divided by the slot's age,
                t being the number of tokens processed, this chunk
                included; one correctly rounded float32 division (the age
                is exact in float32)                                 [B, H, M]
      h2o_orig  the sum over the batch of phi, one slot set per kv-head;
                float32 additions in increasing b                    [H, M]
    """
    s = np.asarray(scores, np.float32)
    if policy == "h2o":
        return s.copy()
    if policy == "h2o_norm":
        if token_pos is None:
            raise ValueError("h2o_norm needs token positions")
        age = t - np.asarray(token_pos, np.int64)
        if (age < 1).any() or (age >= 1 << 24).any():
            raise ValueError("slot ages must be in [1, 2^24)")
        return (s / age.astype(np.float32)).astype(np.float32)
    if policy == "h2o_orig":
        acc = s[0].copy()
        for b in range(1, s.shape[0]):
            acc = (acc + s[b]).astype(np.float32)
        return acc
    raise ValueError(f"unknown policy {policy!r}")


# ------------------------------------------------------------ step 6: insert
def evict_insert(k_cache, v_cache, scores, token_pos, k_new, v_new, wsum,
                 k: int, pos0: int, policy: str = "h2o"):
    """Evict the k lowest-ranked slots per (b, kv-head) and insert the chunk.

    ``scores`` are the accumulated float32 scores; the ranking is that of
    ``selection_keys`` (h2o_orig: one slot set per kv-head, used for every b).
    Returns new copies (k_cache, v_cache, scores, token_pos, evict_idx);
    token_pos may be None except for h2o_norm.
    """
    T = k_new.shape[2]
    if k != T:
        raise ValueError("every chunk key is inserted: k must equal T")
    keys = selection_keys(scores, token_pos, policy, pos0 + T)
    idx = bottomk(keys, k)
    if policy == "h2o_orig":
        idx = np.broadcast_to(idx, (k_cache.shape[0],) + idx.shape).copy()
    kc, vc = k_cache.copy(), v_cache.copy()
    sc = np.asarray(scores, np.float32).copy()
    tp = None if token_pos is None else token_pos.copy()
    M = sc.shape[-1]
    B, H = sc.shape[0], sc.shape[1]
    newsc = np.asarray(wsum)[..., M:M + T].astype(np.float32)
    for b in range(B):
        for h in range(H):
            e = idx[b, h]
            kc[b, h, e] = k_new[b, h, :k]
            vc[b, h, e] = v_new[b, h, :k]
            sc[b, h, e] = newsc[b, h, :k]
            if tp is not None:
                tp[b, h, e] = pos0 + np.arange(k, dtype=np.int32)
    return kc, vc, sc, tp, idx


# --------------------------------------------------------------- whole step
def h2o_step(k_cache, v_cache, scores, token_pos, q, k_new, v_new, pos0: int,
             scale: Optional[float] = None, policy: str = "h2o"):
    """One chunk step: attend, accumulate, evict (ranking of ``policy``), insert.

    Returns dict with out, lse, wsum (float64), scores_acc (float32 scores after
    accumulation), evict_idx and the new cache state.
    """
    out, lse, wsum = sdpa_chunk(q, k_cache, v_cache, k_new, v_new, scale)
    acc = accumulate_scores(scores, wsum)
    T = q.shape[2]
    kc, vc, sc, tp, idx = evict_insert(k_cache, v_cache, acc, token_pos,
                                       k_new, v_new, wsum, T, pos0, policy)
    return dict(out=out, lse=lse, wsum=wsum, scores_acc=acc, evict_idx=idx,
                k_cache=kc, v_cache=vc, scores=sc, token_pos=tp)


# ------------------------------------- the paper's order: insert, then attend
def visible_by_position(token_pos_bh, pos0: int, T: int) -> np.ndarray:
    """Boolean [T, M]: may query i (token position pos0 + i) attend slot j?

    The causal mask of sparse attention (Sec. "Discussion: SDPA Kernels for
    Sparse Attention"): -inf * 1{P + i < t(b,h,j)} with P = pos0 and
    t(b,h,j) the token position stored for the slot, so the slot is visible
    iff t(b,h,j) <= pos0 + i.
    """
    tp = np.asarray(token_pos_bh, np.int64)
    return tp[None, :] <= pos0 + np.arange(T)[:, None]


def _head_masked(Qh: np.ndarray, K: np.ndarray, V: np.ndarray, allowed: np.ndarray,
                 scale: float) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """``_head`` for an arbitrary mask. A row that sees no key has no softmax:
    its output is 0, its lambda is -inf and it adds nothing to the column
    sums."""
    A = scale * (Qh @ K.T)
    A = np.where(allowed, A, -np.inf)
    some = allowed.any(axis=1)
    amax = np.where(some, A.max(axis=1), 0.0)[:, None]
    with np.errstate(divide="ignore"):
        lam = amax[:, 0] + np.log(np.exp(A - amax).sum(axis=1))
    Mw = np.where(some[:, None], np.exp(A - np.where(some, lam, 0.0)[:, None]), 0.0)
    return Mw @ V, lam, Mw.sum(axis=0)


def sdpa_cache(q, k_cache, v_cache, token_pos, pos0: int, scale: Optional[float] = None,
               heads: Optional[Iterable[Tuple[int, int]]] = None):
    """Attention of T queries (positions pos0 .. pos0+T-1) over the M cache
    slots alone, masked by the slots' token positions (``visible_by_position``);
    the chunk's own keys are expected in the cache already.

    Shapes: q [B,Hq,T,d]; k_cache, v_cache [B,Hkv,M,d]; token_pos [B,Hkv,M].
    Returns float64 (out [B,Hq,T,d], lse [B,Hq,T], wsum [B,Hkv,M]), wsum summed
    over the group's query heads as in ``sdpa_chunk``; ``heads`` as there.
    """
    q = np.asarray(q)
    B, Hq, T, d = q.shape
    Hkv, M = k_cache.shape[1], k_cache.shape[2]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    scale = float(scale)
    out = np.full((B, Hq, T, d), np.nan, F64)
    lse = np.full((B, Hq, T), np.nan, F64)
    wsum = np.full((B, Hkv, M), np.nan, F64)
    if heads is None:
        heads = [(b, h) for b in range(B) for h in range(Hkv)]
    for b, h in heads:
        allowed = visible_by_position(token_pos[b, h], pos0, T)
        K = np.asarray(k_cache[b, h], F64)
        V = np.asarray(v_cache[b, h], F64)
        acc = np.zeros(M, F64)
        for g in range(G):
            hq = h * G + g
            Y, lam, col = _head_masked(q[b, hq].astype(F64), K, V, allowed, scale)
            out[b, hq] = Y
            lse[b, hq] = lam
            acc += col
        wsum[b, h] = acc
    return out, lse, wsum


def h2o_step_insert_first(k_cache, v_cache, scores, token_pos, q, k_new, v_new,
                          pos0: int, scale: Optional[float] = None, policy: str = "h2o"):
    """One chunk step in the paper's order (Sec. "Sparse Attention. Key-Value
    Caching" with the mask of Sec. "Discussion: SDPA Kernels for Sparse
    Attention"):

    1. rank the slots by the scores after ``pos0`` tokens (t = pos0 for
       h2o_norm) and pick the T lowest (``bottomk``; h2o_orig: one set per
       kv-head);
    2. write chunk key/value i into the i-th picked slot, with token position
       pos0 + i and score 0 (Eq. h2o-score sums from the slot's own position);
    3. attend over the M slots with the token-position mask (``sdpa_cache``);
    4. add the summed weights to the scores of all M slots (one float32
       addition each).
    """
    T = q.shape[2]
    keys = selection_keys(scores, token_pos, policy, pos0)
    idx = bottomk(keys, T)
    if policy == "h2o_orig":
        idx = np.broadcast_to(idx, (k_cache.shape[0],) + idx.shape).copy()
    kc, vc = k_cache.copy(), v_cache.copy()
    sc = np.asarray(scores, np.float32).copy()
    tp = np.asarray(token_pos, np.int32).copy()
    B, H = sc.shape[0], sc.shape[1]
    for b in range(B):
        for h in range(H):
            e = idx[b, h]
            kc[b, h, e] = k_new[b, h]
            vc[b, h, e] = v_new[b, h]
            sc[b, h, e] = 0.0
            tp[b, h, e] = pos0 + np.arange(T, dtype=np.int32)
    out, lse, wsum = sdpa_cache(q, kc, vc, tp, pos0, scale)
    return dict(out=out, lse=lse, wsum=wsum, evict_idx=idx, scores_inserted=sc,
                k_cache=kc, v_cache=vc, scores=accumulate_scores(sc, wsum), token_pos=tp)


# ------------------------------------------- backward (fine-tuning) and deltas
def _head_backward(Qh, K, V, allowed, scale, dO):
    """Gradients of one query head's output Y = softmax(scale Q K^T, masked) V
    for the loss sum(dO * Y): returns (dQ [T,d], dK [Nk,d], dV [Nk,d]).

    The softmax vector-Jacobian product row by row: with p = softmax(a) and
    g = dL/dp, dL/da = p * (g - <p, g>). A row that sees no key has no
    gradient."""
    A = scale * (Qh @ K.T)
    A = np.where(allowed, A, -np.inf)
    some = allowed.any(axis=1)
    amax = np.where(some, A.max(axis=1), 0.0)[:, None]
    E = np.where(allowed, np.exp(A - amax), 0.0)
    Z = E.sum(axis=1, keepdims=True)
    P = np.where(some[:, None], E / np.where(Z > 0, Z, 1.0), 0.0)     # attention weights
    dV = P.T @ dO
    dP = dO @ V.T                                                      # dL/dP
    dA = P * (dP - (P * dP).sum(axis=1, keepdims=True))                # softmax VJP
    dQ = scale * (dA @ K)
    dK = scale * (dA.T @ Qh)
    return dQ, dK, dV


def sdpa_chunk_backward(q, k_cache, v_cache, k_new, v_new, dout, scale: Optional[float] = None,
                        token_pos=None, pos0: int = 0):
    """Gradients of the chunk attention's output for the loss sum(dout * out),
    the backward of the SDPA of a fine-tuning step (Sec. "Fine-Tuning for
    Sparse Attention"). The summed weights carry no gradient: they only steer
    the discrete eviction.

    Chunk mode (token_pos None): keys [cache || chunk] as in ``sdpa_chunk``;
    returns float64 (dq [B,Hq,T,d], dk_cache, dv_cache [B,Hkv,M,d], dk_new,
    dv_new [B,Hkv,T,d]). Cache mode (token_pos given): the keys are the cache
    slots with the token-position mask of ``sdpa_cache``; dk_new and dv_new
    are None. Gradients of a KV head sum over its group's query heads.
    """
    q = np.asarray(q)
    B, Hq, T, d = q.shape
    Hkv, M = k_cache.shape[1], k_cache.shape[2]
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    scale = float(scale)
    cache_mode = token_pos is not None
    Nk = M if cache_mode else M + T
    dq = np.zeros((B, Hq, T, d))
    dk = np.zeros((B, Hkv, Nk, d))
    dv = np.zeros((B, Hkv, Nk, d))
    for b in range(B):
        for h in range(Hkv):
            if cache_mode:
                K = np.asarray(k_cache[b, h], F64)
                V = np.asarray(v_cache[b, h], F64)
                allowed = visible_by_position(token_pos[b, h], pos0, T)
            else:
                K = np.concatenate([k_cache[b, h], k_new[b, h]]).astype(F64)
                V = np.concatenate([v_cache[b, h], v_new[b, h]]).astype(F64)
                allowed = visible(M, T)
            for g in range(G):
                hq = h * G + g
                gq, gk, gv = _head_backward(q[b, hq].astype(F64), K, V, allowed, scale,
                                            np.asarray(dout[b, hq], F64))
                dq[b, hq] = gq
                dk[b, h] += gk
                dv[b, h] += gv
    if cache_mode:
        return dq, dk, dv, None, None
    return dq, dk[:, :, :M], dv[:, :, :M], dk[:, :, M:], dv[:, :, M:]


def kv_gather(cache, idx) -> np.ndarray:
    """delta[b, h, i] = cache[b, h, idx[b, h, i]]: the rows a chunk's insert is
    about to overwrite, the delta encoding of the KV recurrence (Eq.
    recurrence-reverse, Sec. "Buffer Read/Write Access by torch.scatter,
    torch.gather")."""
    cache = np.asarray(cache)
    idx = np.asarray(idx)
    out = np.empty(idx.shape + cache.shape[3:], cache.dtype)
    for b in range(idx.shape[0]):
        for h in range(idx.shape[1]):
            out[b, h] = cache[b, h, idx[b, h]]
    return out


def kv_scatter(cache, idx, src) -> np.ndarray:
    """A copy of cache with cache[b, h, idx[b, h, i]] = src[b, h, i]: the insert
    of a chunk, and, with src = kv_gather(old cache, idx), its inverse."""
    out = np.array(cache, copy=True)
    idx = np.asarray(idx)
    for b in range(idx.shape[0]):
        for h in range(idx.shape[1]):
            out[b, h, idx[b, h]] = src[b, h]
    return out


def decode(k_cache, v_cache, scores, token_pos, q_steps, k_new_steps,
           v_new_steps, pos0: int, scale: Optional[float] = None):
    """Token generation: ``len(q_steps)`` chunk steps of length T (usually 1),
    positions pos0, pos0+T, ... Returns the list of per-step results."""
    res = []
    state = (k_cache, v_cache, scores, token_pos)
    for s in range(len(q_steps)):
        T = q_steps[s].shape[2]
        r = h2o_step(*state, q_steps[s], k_new_steps[s], v_new_steps[s],
                     pos0 + s * T, scale)
        res.append(r)
        state = (r["k_cache"], r["v_cache"], r["scores"], r["token_pos"])
    return res


# ------------------------------------------------------------------ metrics
def rel_err(x, ref, axes: Sequence[int]) -> float:
    """Max over slices of ||x - ref||_2 / ||ref||_2, the norm taken over `axes`."""
    x = np.asarray(x, F64)
    ref = np.asarray(ref, F64)
    num = np.sqrt(((x - ref) ** 2).sum(axis=tuple(axes)))
    den = np.sqrt((ref ** 2).sum(axis=tuple(axes)))
    return float((num / np.maximum(den, np.finfo(F64).tiny)).max())


def elem_err(x, ref, axes: Sequence[int], floor: float = 1e-6) -> float:
    """Max over elements of |x - ref| / (|ref| + floor * max|ref|), the maximum
    |ref| taken per slice over `axes`.

    The summed weight and the score are defined per key (Eq. h2o-score), so
    they are compared element by element: an element is held to a relative
    error, and only elements below ``floor`` times the largest of their slice
    to an absolute one. A slice whose reference is all zero must match
    exactly."""
    x = np.asarray(x, F64)
    ref = np.asarray(ref, F64)
    scale = np.abs(ref).max(axis=tuple(axes), keepdims=True)
    den = np.abs(ref) + floor * scale
    err = np.abs(x - ref)
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(den > 0, err / np.where(den > 0, den, 1.0), np.where(err > 0, np.inf, 0.0))
    return float(r.max()) if r.size else 0.0


def eviction_agreement(evicted, scores_ref, k: int, tol: float):
    """Compares a chosen eviction set with the oracle's for one row.

    ``evicted``: the k slots some computation evicted, from its own float32
    scores; ``scores_ref``: the oracle's accumulated scores of the row (all
    non-negative). If that computation's scores are within ``tol`` of the
    oracle's, relatively and element by element, then every slot it evicts
    has an oracle score of at most tau * (1 + tol) / (1 - tol) and every slot
    it keeps one of at least tau * (1 - tol) / (1 + tol), tau being the
    oracle's k-th smallest score (Sec. "Variants of Heavy-Hitter Oracle":
    the slots of smallest score are overwritten).

    Returns (n_diff, n_band, valid): the number of evicted slots outside the
    oracle's own eviction set, the number of oracle slots inside that band
    (the only ones that may trade places), and whether every evicted and
    every kept slot lies on its side of the band."""
    s = np.asarray(scores_ref, F64)
    M = s.shape[-1]
    ev = np.asarray(evicted, np.int64)
    own = bottomk(np.asarray(scores_ref, np.float32)[None], k)[0]
    if k == 0:
        return 0, 0, len(ev) == 0
    tau = float(np.sort(s)[k - 1])
    hi = tau * (1.0 + tol) / (1.0 - tol)
    lo = tau * (1.0 - tol) / (1.0 + tol)
    kept = np.setdiff1d(np.arange(M), ev)
    valid = (len(np.unique(ev)) == k and ev.min() >= 0 and ev.max() < M
             and bool((s[ev] <= hi).all()) and bool((s[kept] >= lo).all()))
    n_diff = int(len(np.setdiff1d(ev, own)))
    n_band = int(((s >= lo) & (s <= hi)).sum())
    return n_diff, n_band, valid
