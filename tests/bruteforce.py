"""Independent brute-force formulations used to pin the oracle on tiny inputs.

These are written as whole-matrix numpy / torch-autograd computations (explicit
L x L masks, full sorts, autograd gradients), deliberately different in form
from the oracle's per-row loops, so that a slip in either shows up as a
mismatch.  Test infrastructure only.
"""
from __future__ import annotations

import numpy as np
import torch


def blocks_of(positions, m):
    return np.asarray(positions) // m


def compress(K, punct, m, lam):
    """Eq. 6-8 via reshapes: K [B, L, Hkv, d] -> [B, Hkv, T, d]."""
    K = np.asarray(K, dtype=np.float64)
    B, L, H, d = K.shape
    T = L // m
    Kb = K[:, :T * m].reshape(B, T, m, H, d)
    w = np.asarray(punct, dtype=np.float64)[:, :T * m].reshape(B, T, m)
    m0 = Kb.mean(axis=2)                                            # [B, T, H, d]
    cnt = w.sum(axis=2)                                             # [B, T]
    mp_num = np.einsum("btm,btmhd->bthd", w, Kb)
    with np.errstate(invalid="ignore", divide="ignore"):
        mp = mp_num / cnt[:, :, None, None]
    fused = lam * m0 + (1.0 - lam) * mp
    out = np.where((cnt > 0)[:, :, None, None], fused, m0)
    return out.transpose(0, 2, 1, 3)


def group_scores(Q, Kc, scale):
    """[B, Hkv, Lq, T] sum over each group's heads of scale * q . M."""
    Q = np.asarray(Q, dtype=np.float64)
    B, Lq, Hq, d = Q.shape
    H = Kc.shape[1]
    G = Hq // H
    per_head = np.einsum("bihd,bgtd->bhgit", Q, Kc) * scale          # all (h, g) pairs
    out = np.zeros((B, H, Lq, Kc.shape[2]))
    for g in range(H):
        for hh in range(G):
            out[:, g] += per_head[:, g * G + hh, g]
    return out


def group_softmax_scores(Q, Kc, scale, m, Lk):
    """[B, Hkv, Lq, T] log of the summed per-head softmax probabilities, each
    head's softmax taken (with scipy) over the blocks strictly before the
    query's own block; -inf elsewhere."""
    from scipy.special import softmax
    Q = np.asarray(Q, dtype=np.float64)
    B, Lq, Hq, d = Q.shape
    H, T = Kc.shape[1], Kc.shape[2]
    G = Hq // H
    cur = (Lk - Lq + np.arange(Lq)) // m
    past = np.arange(T)[None, :] < cur[:, None]                     # [Lq, T]
    per_head = np.einsum("bihd,bgtd->bhgit", Q, Kc) * scale
    out = np.full((B, H, Lq, T), -np.inf)
    with np.errstate(divide="ignore"):
        for g in range(H):
            prob = np.zeros((B, Lq, T))
            for hh in range(G):
                logits = np.where(past[None], per_head[:, g * G + hh, g], -np.inf)
                rows = past.any(axis=1)
                prob[:, rows] += softmax(logits[:, rows], axis=-1)
            out[:, g] = np.where(past[None], np.log(prob), -np.inf)
    return out


def select(Q, Kc, m, top_k, n_init, window, scale, Lk, softmax_sum=False):
    """Algorithm 1 block selection by full lexsort of every row's score vector."""
    B, Lq = Q.shape[0], Q.shape[1]
    H, T = Kc.shape[1], Kc.shape[2]
    S = group_softmax_scores(Q, Kc, scale, m, Lk) if softmax_sum else group_scores(Q, Kc, scale)
    ksel = n_init + window // m + 1 + top_k
    out = -np.ones((B, H, Lq, ksel), dtype=np.int32)
    t_all = np.arange(T)
    for b in range(B):
        for g in range(H):
            for i in range(Lq):
                cur = (Lk - Lq + i) // m
                causal = t_all <= cur
                forced = causal & ((t_all < n_init) | (t_all >= cur - window // m))
                cand = np.nonzero(causal & ~forced)[0]
                order = np.lexsort((cand, -S[b, g, i, cand]))       # score desc, index asc
                picks = cand[order[:top_k]]
                final = np.union1d(np.nonzero(forced)[0], picks)
                out[b, g, i, :final.size] = final
    return out, S


def token_mask(sel, m, Lq, Lk):
    """Explicit [B, Hkv, Lq, Lk] boolean attention mask from block indices + causality."""
    B, H = sel.shape[0], sel.shape[1]
    T = Lk // m
    onehot = np.zeros((B, H, Lq, T + 1), dtype=bool)
    s = np.where(sel < 0, T, sel)
    np.put_along_axis(onehot, s.astype(np.int64), True, axis=3)
    blk = np.repeat(onehot[..., :T], m, axis=3)                     # [B, H, Lq, Lk]
    pos = (Lk - Lq) + np.arange(Lq)
    causal = np.arange(Lk)[None, :] <= pos[:, None]
    return blk & causal[None, None]


def attention(Q, K, V, sel, m, scale, dO=None):
    """Dense masked attention (and its autograd gradient) in float64 torch."""
    B, Lq, Hq, d = Q.shape
    Lk, H = K.shape[1], K.shape[2]
    G = Hq // H
    mask = torch.from_numpy(np.repeat(token_mask(np.asarray(sel), m, Lq, Lk), G, axis=1))
    q = torch.tensor(np.asarray(Q, dtype=np.float64), requires_grad=True)
    k = torch.tensor(np.asarray(K, dtype=np.float64), requires_grad=True)
    v = torch.tensor(np.asarray(V, dtype=np.float64), requires_grad=True)
    kk = k.repeat_interleave(G, dim=2)
    vv = v.repeat_interleave(G, dim=2)
    s = torch.einsum("bihd,bjhd->bhij", q, kk) * scale
    s = s.masked_fill(~mask, float("-inf"))
    lse = torch.logsumexp(s, dim=-1)                                 # [B, Hq, Lq]
    p = torch.exp(s - lse[..., None])
    o = torch.einsum("bhij,bjhd->bihd", p, vv)
    res = {"O": o.detach().numpy(), "LSE": lse.detach().numpy()}
    if dO is not None:
        (o * torch.tensor(np.asarray(dO, dtype=np.float64))).sum().backward()
        res.update(dQ=q.grad.numpy(), dK=k.grad.numpy(), dV=v.grad.numpy())
    return res
