"""Independent computations the oracle is pinned against (CPU, float64).

None of these call the oracle. Each is a different route to the same numbers:

* ``brute_sdpa``: pure-Python loops with ``math.fsum`` and ``math.exp``,
  softmax without max-shifting, head mapping written out per query head.
* ``torch_sdpa``: ``torch.nn.functional.scaled_dot_product_attention`` in
  float64 with an explicit boolean mask (library routine).
* ``mapreduce_wsum``: the tiled map-reduce of Sec. "FlashAttention for Summed
  Attention Weights": per tile lambda_{r,s} and F~_{r,s}, reduction of lambda
  along s with max + log1p(exp(-|a-b|)), then w_{r,s} = exp(lambda_{r,s} -
  lambda_r)^T F~_{r,s}, summed over r; the outputs y_{r,s} are combined with
  the matching rescaling.
* ``transposed_wsum``: the two-call identity of Sec. "Summed Attention Weights
  with FlexAttention": (y, lambda) = SDPA(Q, K, V), then
  (y~, lambda~) = SDPA_rev(K, Q, exp(-(lambda - mean lambda))) with the mask
  flipped, and w = exp(lambda~ - mean lambda) * y~. Both SDPA calls are torch's.
* ``brute_bottomk``: Python ``sorted`` on (score, slot) tuples.
"""
from __future__ import annotations

import math

import numpy as np
import torch


def brute_sdpa(q, kc, vc, kn, vn, scale):
    """Returns (out, lse, wsum) as float64 numpy arrays; tiny shapes only."""
    B, Hq, T, d = q.shape
    Hkv, M = kc.shape[1], kc.shape[2]
    G = Hq // Hkv
    out = np.zeros((B, Hq, T, d))
    lse = np.zeros((B, Hq, T))
    wsum = np.zeros((B, Hkv, M + T))
    for b in range(B):
        for h in range(Hkv):
            keys = [[float(x) for x in kc[b, h, j]] for j in range(M)] + \
                   [[float(x) for x in kn[b, h, t]] for t in range(T)]
            vals = [[float(x) for x in vc[b, h, j]] for j in range(M)] + \
                   [[float(x) for x in vn[b, h, t]] for t in range(T)]
            col_terms = [[] for _ in range(M + T)]
            for g in range(G):
                hq = h * G + g
                for i in range(T):
                    qi = [float(x) for x in q[b, hq, i]]
                    cols = list(range(M)) + [M + t for t in range(T) if t <= i]
                    a = {j: float(scale) * math.fsum(qi[c] * keys[j][c] for c in range(d))
                         for j in cols}
                    Z = math.fsum(math.exp(a[j]) for j in cols)
                    lse[b, hq, i] = math.log(Z)
                    p = {j: math.exp(a[j]) / Z for j in cols}
                    for c in range(d):
                        out[b, hq, i, c] = math.fsum(p[j] * vals[j][c] for j in cols)
                    for j in cols:
                        col_terms[j].append(p[j])
            for j in range(M + T):
                wsum[b, h, j] = math.fsum(col_terms[j])
    return out, lse, wsum


def _mask(M, T):
    # query i may see every cache slot and chunk keys t <= i
    m = torch.ones(T, M + T, dtype=torch.bool)
    m[:, M:] = torch.tril(torch.ones(T, T, dtype=torch.bool))
    return m


def _kv(kc, vc, kn, vn, b, h):
    K = torch.from_numpy(np.concatenate([kc[b, h], kn[b, h]]).astype(np.float64))
    V = torch.from_numpy(np.concatenate([vc[b, h], vn[b, h]]).astype(np.float64))
    return K, V


def _lse_torch(Q, K, mask, scale):
    A = scale * (Q @ K.T)
    A = A.masked_fill(~mask, float("-inf"))
    return torch.logsumexp(A, dim=-1)


def torch_sdpa(q, kc, vc, kn, vn, scale):
    """Output and lse of every head via torch's SDPA (float64, CPU)."""
    F = torch.nn.functional
    B, Hq, T, d = q.shape
    Hkv, M = kc.shape[1], kc.shape[2]
    G = Hq // Hkv
    mask = _mask(M, T)
    out = np.zeros((B, Hq, T, d))
    lse = np.zeros((B, Hq, T))
    for b in range(B):
        for h in range(Hkv):
            K, V = _kv(kc, vc, kn, vn, b, h)
            for g in range(G):
                Q = torch.from_numpy(q[b, h * G + g].astype(np.float64))
                out[b, h * G + g] = F.scaled_dot_product_attention(
                    Q[None], K[None], V[None], attn_mask=mask[None],
                    scale=float(scale))[0].numpy()
                lse[b, h * G + g] = _lse_torch(Q, K, mask, float(scale)).numpy()
    return out, lse


def transposed_wsum(q, kc, vc, kn, vn, scale):
    """Summed weights by the flipped second SDPA call (float64)."""
    F = torch.nn.functional
    B, Hq, T, d = q.shape
    Hkv, M = kc.shape[1], kc.shape[2]
    G = Hq // Hkv
    mask = _mask(M, T)
    w = np.zeros((B, Hkv, M + T))
    for b in range(B):
        for h in range(Hkv):
            K, V = _kv(kc, vc, kn, vn, b, h)
            for g in range(G):
                Q = torch.from_numpy(q[b, h * G + g].astype(np.float64))
                lam = _lse_torch(Q, K, mask, float(scale))            # (T,)
                lbar = lam.mean()
                vt = torch.exp(-(lam - lbar))[:, None]                 # (T, 1)
                # SDPA_rev: queries = keys, keys = queries, mask transposed
                yt = F.scaled_dot_product_attention(
                    K[None], Q[None], vt[None], attn_mask=mask.T[None],
                    scale=float(scale))[0, :, 0]
                lt = _lse_torch(K, Q, mask.T, float(scale))
                w[b, h] += (torch.exp(lt - lbar) * yt).numpy()
    return w


def _logaddexp_paper(a, b):
    """lambda_{s1 (+) s2} = max + log1p(exp(-|a - b|)), with -inf handled."""
    m = np.maximum(a, b)
    with np.errstate(invalid="ignore"):
        diff = np.where(np.isfinite(m), -np.abs(a - b), -np.inf)
    return np.where(np.isfinite(m), m + np.log1p(np.exp(diff)), m)


def mapreduce_wsum(q, kc, vc, kn, vn, scale, row_tile, col_tile):
    """Summed weights and outputs by the tiled map-reduce (float64).

    Returns (out, wsum). Tiles: rows I(r) of size row_tile over the T queries,
    columns J(s) of size col_tile over the M+T keys.
    """
    B, Hq, T, d = q.shape
    Hkv, M = kc.shape[1], kc.shape[2]
    G = Hq // Hkv
    N = M + T
    allowed = _mask(M, T).numpy()
    out = np.zeros((B, Hq, T, d))
    w = np.zeros((B, Hkv, N))
    rows = [np.arange(r0, min(r0 + row_tile, T)) for r0 in range(0, T, row_tile)]
    cols = [np.arange(c0, min(c0 + col_tile, N)) for c0 in range(0, N, col_tile)]
    for b in range(B):
        for h in range(Hkv):
            K = np.concatenate([kc[b, h], kn[b, h]]).astype(np.float64)
            V = np.concatenate([vc[b, h], vn[b, h]]).astype(np.float64)
            for g in range(G):
                Q = q[b, h * G + g].astype(np.float64)
                for I in rows:
                    lam_s, Ft_s, y_s = [], [], []
                    for J in cols:                              # map
                        A = scale * (Q[I] @ K[J].T)
                        A = np.where(allowed[np.ix_(I, J)], A, -np.inf)
                        mx = A.max(axis=1)
                        safe = np.where(np.isfinite(mx), mx, 0.0)
                        with np.errstate(divide="ignore"):
                            lam = safe + np.log(np.exp(A - safe[:, None]).sum(axis=1))
                        lam = np.where(np.isfinite(mx), lam, -np.inf)
                        lsafe = np.where(np.isfinite(lam), lam, 0.0)
                        Ft = np.exp(A - lsafe[:, None])          # F~_{r,s}
                        lam_s.append(lam)
                        Ft_s.append(Ft)
                        y_s.append(Ft @ V[J])                    # tile-normalised y_{r,s}
                    lam_r = lam_s[0]                             # reduce along s
                    y_r = y_s[0]
                    for s in range(1, len(cols)):
                        new = _logaddexp_paper(lam_r, lam_s[s])
                        a1 = np.exp(np.where(np.isfinite(lam_r), lam_r - new, -np.inf))
                        a2 = np.exp(np.where(np.isfinite(lam_s[s]), lam_s[s] - new, -np.inf))
                        y_r = a1[:, None] * y_r + a2[:, None] * y_s[s]
                        lam_r = new
                    out[b, h * G + g, I] = y_r
                    for s, J in enumerate(cols):                 # w_{r,s}
                        sc = np.exp(np.where(np.isfinite(lam_s[s]), lam_s[s] - lam_r, -np.inf))
                        w[b, h, J] += sc @ Ft_s[s]
    return out, w


def brute_bottomk(scores, k):
    s = np.asarray(scores, np.float32)
    M = s.shape[-1]
    flat = s.reshape(-1, M)
    res = []
    for row in flat:
        keyed = sorted((float(row[j]) + 0.0, j) for j in range(M))
        res.append(sorted(j for _, j in keyed[:k]))
    return np.array(res, np.int32).reshape(*s.shape[:-1], k)


def brute_sdpa_positions(q, kc, vc, tp, pos0, scale):
    """Attention over the cache slots masked by token position, by loops:
    query i (position pos0 + i) sees slot j iff tp[b,h,j] <= pos0 + i. A
    query that sees nothing gets out 0 and lse -inf. Returns float64
    (out, lse, wsum [B,Hkv,M]); tiny shapes only."""
    B, Hq, T, d = q.shape
    Hkv, M = kc.shape[1], kc.shape[2]
    G = Hq // Hkv
    out = np.zeros((B, Hq, T, d))
    lse = np.zeros((B, Hq, T))
    wsum = np.zeros((B, Hkv, M))
    for b in range(B):
        for h in range(Hkv):
            col_terms = [[] for _ in range(M)]
            for g in range(G):
                hq = h * G + g
                for i in range(T):
                    cols = [j for j in range(M) if int(tp[b, h, j]) <= pos0 + i]
                    if not cols:
                        lse[b, hq, i] = -math.inf
                        continue
                    qi = [float(x) for x in q[b, hq, i]]
                    a = {j: float(scale) * math.fsum(qi[c] * float(kc[b, h, j, c])
                                                     for c in range(d)) for j in cols}
                    Z = math.fsum(math.exp(a[j]) for j in cols)
                    lse[b, hq, i] = math.log(Z)
                    for c in range(d):
                        out[b, hq, i, c] = math.fsum(math.exp(a[j]) / Z * float(vc[b, h, j, c])
                                                     for j in cols)
                    for j in cols:
                        col_terms[j].append(math.exp(a[j]) / Z)
            for j in range(M):
                wsum[b, h, j] = math.fsum(col_terms[j])
    return out, lse, wsum


def torch_sdpa_positions(q, kc, vc, tp, pos0, scale):
    """Output and lse via torch's SDPA (float64, CPU) with the boolean mask
    built from token positions; every row must see at least one slot."""
    F = torch.nn.functional
    B, Hq, T, d = q.shape
    Hkv = kc.shape[1]
    G = Hq // Hkv
    out = np.zeros((B, Hq, T, d))
    lse = np.zeros((B, Hq, T))
    pos = torch.arange(T, dtype=torch.int64)[:, None] + int(pos0)
    for b in range(B):
        for h in range(Hkv):
            mask = torch.from_numpy(np.asarray(tp[b, h], np.int64))[None, :] <= pos
            K = torch.from_numpy(np.asarray(kc[b, h], np.float64))
            V = torch.from_numpy(np.asarray(vc[b, h], np.float64))
            for g in range(G):
                Q = torch.from_numpy(np.asarray(q[b, h * G + g], np.float64))
                out[b, h * G + g] = F.scaled_dot_product_attention(
                    Q[None], K[None], V[None], attn_mask=mask[None], scale=float(scale))[0].numpy()
                lse[b, h * G + g] = _lse_torch(Q, K, mask, float(scale)).numpy()
    return out, lse


def torch_attention_grads(q, kc, vc, kn, vn, dout, scale, token_pos=None, pos0=0):
    """Gradients of sum(dout * out) by torch autograd (float64, CPU) through an
    explicit masked softmax attention, head by head (GQA heads share the KV
    tensors, so their gradients add up by autograd itself)."""
    B, Hq, T, d = q.shape
    Hkv, M = kc.shape[1], kc.shape[2]
    G = Hq // Hkv
    t = lambda a: torch.tensor(np.asarray(a, np.float64), requires_grad=True)
    Q, KC, VC = t(q), t(kc), t(vc)
    cache_mode = token_pos is not None
    KN, VN = (None, None) if cache_mode else (t(kn), t(vn))
    loss = 0.0
    for b in range(B):
        for h in range(Hkv):
            if cache_mode:
                K, V = KC[b, h], VC[b, h]
                mask = torch.from_numpy(np.asarray(token_pos[b, h], np.int64))[None, :] <= \
                    (torch.arange(T)[:, None] + int(pos0))
            else:
                K = torch.cat([KC[b, h], KN[b, h]])
                V = torch.cat([VC[b, h], VN[b, h]])
                mask = _mask(M, T)
            for g in range(G):
                A = float(scale) * (Q[b, h * G + g] @ K.T)
                A = A.masked_fill(~mask, float("-inf"))
                P = torch.softmax(A, dim=-1)
                loss = loss + (torch.from_numpy(np.asarray(dout[b, h * G + g], np.float64)) *
                               (P @ V)).sum()
    loss.backward()
    g = lambda x: None if x is None else x.grad.numpy()
    return g(Q), g(KC), g(VC), g(KN), g(VN)
