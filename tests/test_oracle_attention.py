"""Pins of the oracle's sparse attention forward (Eq. 10-11) and backward."""
import numpy as np
import pytest
import torch

import oracle
from tests import bruteforce as bf


def _qkv(B, Lq, Lk, Hq, Hkv, d, seed, dyadic=False):
    rng = np.random.default_rng(seed)
    out = [rng.standard_normal(s).astype(np.float32) for s in
           ((B, Lq, Hq, d), (B, Lk, Hkv, d), (B, Lk, Hkv, d), (B, Lq, Hq, d))]
    if dyadic:      # multiples of 2^-8 so that +-2^-7 perturbations stay exact in float32
        out = [np.round(x * 256) / 256 for x in out]
    return out


def _select(Q, K, m, k, n_init, w, seed):
    Lk = K.shape[1]
    punct = (np.random.default_rng(seed).random((K.shape[0], Lk)) < 0.1).astype(np.uint8)
    Kc = oracle.compress(K, punct, m, 0.5)
    sel, _, _ = oracle.select(Q, Kc, m, k, n_init, w, Q.shape[-1] ** -0.5, Lk)
    return sel


def test_all_blocks_is_dense_causal_attention():
    """top-k covering every block reduces the method to dense causal attention (torch SDPA, fp64)."""
    B, L, Hq, Hkv, d, m = 2, 128, 4, 2, 16, 16
    Q, K, V, _ = _qkv(B, L, L, Hq, Hkv, d, 0)
    sel = _select(Q, K, m, L // m, 1, 0, 0)
    O, LSE = oracle.attn_fwd(Q, K, V, sel, m, d ** -0.5)
    q = torch.tensor(Q, dtype=torch.float64).transpose(1, 2)
    k = torch.tensor(K, dtype=torch.float64).transpose(1, 2).repeat_interleave(Hq // Hkv, dim=1)
    v = torch.tensor(V, dtype=torch.float64).transpose(1, 2).repeat_interleave(Hq // Hkv, dim=1)
    ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True).transpose(1, 2)
    np.testing.assert_allclose(O, ref.numpy(), atol=1e-12)
    s = torch.einsum("bhid,bhjd->bhij", q, k) * d ** -0.5
    s = s.masked_fill(torch.ones(L, L, dtype=torch.bool).triu(1), float("-inf"))
    np.testing.assert_allclose(LSE, torch.logsumexp(s, -1).numpy(), atol=1e-12)


@pytest.mark.parametrize("case", [
    # B, Lq, Lk, Hq, Hkv, d, m, k, n_init, w
    (1, 128, 128, 2, 1, 8, 16, 2, 1, 0),
    (2, 96, 96, 4, 2, 16, 8, 3, 1, 8),
    (1, 256, 256, 4, 1, 8, 32, 2, 2, 32),
    (2, 1, 256, 4, 2, 8, 16, 3, 1, 0),      # decode: one query at the last position
])
def test_bruteforce(case):
    B, Lq, Lk, Hq, Hkv, d, m, k, n_init, w = case
    Q, K, V, dO = _qkv(B, Lq, Lk, Hq, Hkv, d, sum(case))
    sel = _select(Q, K, m, k, n_init, w, 1)
    ref = bf.attention(Q, K, V, sel, m, d ** -0.5, dO=dO)
    O, LSE = oracle.attn_fwd(Q, K, V, sel, m, d ** -0.5)
    np.testing.assert_allclose(O, ref["O"], atol=1e-12)
    np.testing.assert_allclose(LSE, ref["LSE"], atol=1e-12)
    dQ, dK, dV = oracle.attn_bwd(Q, K, V, dO, sel, m, d ** -0.5)
    np.testing.assert_allclose(dQ, ref["dQ"], atol=1e-11)
    np.testing.assert_allclose(dK, ref["dK"], atol=1e-11)
    np.testing.assert_allclose(dV, ref["dV"], atol=1e-11)


def test_first_token_sees_only_itself():
    Q, K, V, _ = _qkv(1, 64, 64, 2, 1, 8, 3)
    sel = _select(Q, K, 16, 2, 1, 0, 3)
    O, LSE = oracle.attn_fwd(Q, K, V, sel, 16, 0.5)
    for h in range(2):
        np.testing.assert_allclose(O[0, 0, h], V[0, 0, 0], atol=1e-15)
        assert LSE[0, h, 0] == pytest.approx(0.5 * float(Q[0, 0, h].astype(np.float64) @ K[0, 0, 0]), abs=1e-12)


def test_convexity_and_lse_bound():
    B, L, Hq, Hkv, d, m = 1, 256, 2, 1, 16, 16
    Q, K, V, _ = _qkv(B, L, L, Hq, Hkv, d, 4)
    sel = _select(Q, K, m, 3, 1, 0, 4)
    O, LSE = oracle.attn_fwd(Q, K, V, sel, m, d ** -0.5)
    mask = bf.token_mask(sel, m, L, L)[0, 0]
    S = np.einsum("ihd,jd->hij", Q[0].astype(np.float64), K[0, :, 0].astype(np.float64)) * d ** -0.5
    for i in range(0, L, 5):
        vs = V[0, mask[i], 0]
        assert (O[0, i] >= vs.min(0) - 1e-12).all() and (O[0, i] <= vs.max(0) + 1e-12).all()
        for h in range(Hq):
            assert LSE[0, h, i] >= S[h, i, mask[i]].max() - 1e-12
            assert LSE[0, h, i] <= S[h, i, mask[i]].max() + np.log(mask[i].sum()) + 1e-12


def test_block_order_invariance():
    """The selected set is a set: permuting a row's block ids leaves O and LSE unchanged."""
    Q, K, V, dO = _qkv(1, 256, 256, 2, 1, 8, 5)
    sel = _select(Q, K, 16, 4, 1, 16, 5)
    rev = sel.copy()
    for i in range(256):
        n = int((sel[0, 0, i] >= 0).sum())
        rev[0, 0, i, :n] = sel[0, 0, i, :n][::-1]
    a = oracle.attn_fwd(Q, K, V, sel, 16, 0.3)
    b = oracle.attn_fwd(Q, K, V, rev, 16, 0.3)
    np.testing.assert_allclose(a[0], b[0], atol=1e-13)
    np.testing.assert_allclose(a[1], b[1], atol=1e-13)


def test_row_and_block_subsets():
    B, L, Hq, Hkv, d, m = 2, 128, 4, 2, 8, 16
    Q, K, V, dO = _qkv(B, L, L, Hq, Hkv, d, 6)
    sel = _select(Q, K, m, 2, 1, 0, 6)
    O, LSE = oracle.attn_fwd(Q, K, V, sel, m, 0.3)
    rows = np.array([0, 63, 64, 200, 255])
    Os, Ls = oracle.attn_fwd(Q, K, V, sel, m, 0.3, rows=rows)
    dQ, dK, dV = oracle.attn_bwd(Q, K, V, dO, sel, m, 0.3)
    dQs, _, _ = oracle.attn_bwd(Q, K, V, dO, sel, m, 0.3, rows=rows, want_dkv=False)
    blocks = np.array([0, 3, 8 + 1, 16 + 7, 31])                 # b*Hkv*T + g*T + t with T = 8
    _, dKs, dVs = oracle.attn_bwd(Q, K, V, dO, sel, m, 0.3, blocks=blocks, want_dq=False)
    for r, row in enumerate(rows):
        b, i = divmod(int(row), L)
        np.testing.assert_allclose(Os[r], O[b, i], atol=1e-14)
        np.testing.assert_allclose(Ls[r], LSE[b, :, i], atol=1e-14)
        np.testing.assert_allclose(dQs[r], dQ[b, i], atol=1e-13)
    for x, blk in enumerate(blocks):
        b, rem = divmod(int(blk), Hkv * 8)
        g, t = divmod(rem, 8)
        np.testing.assert_allclose(dKs[x], dK[b, t * m:(t + 1) * m, g], atol=1e-13)
        np.testing.assert_allclose(dVs[x], dV[b, t * m:(t + 1) * m, g], atol=1e-13)


def test_finite_differences():
    """Central differences of L = sum(dO * O) with the selection frozen (dyadic inputs, exact steps)."""
    B, L, Hq, Hkv, d, m = 1, 48, 2, 1, 4, 8
    Q, K, V, dO = _qkv(B, L, L, Hq, Hkv, d, 7, dyadic=True)
    sel = _select(Q, K, m, 2, 1, 0, 7)
    dQ, dK, dV = oracle.attn_bwd(Q, K, V, dO, sel, m, 0.5)
    eps = 2.0 ** -7
    loss = lambda q, k, v: float((oracle.attn_fwd(q, k, v, sel, m, 0.5)[0] * dO).sum())
    rng = np.random.default_rng(0)
    for name, X, G in (("Q", Q, dQ), ("K", K, dK), ("V", V, dV)):
        for _ in range(12):
            idx = tuple(int(rng.integers(s)) for s in X.shape)
            Xp, Xm = X.copy(), X.copy()
            Xp[idx] += eps
            Xm[idx] -= eps
            args_p = [Xp if n == name else A for n, A in (("Q", Q), ("K", K), ("V", V))]
            args_m = [Xm if n == name else A for n, A in (("Q", Q), ("K", K), ("V", V))]
            num = (loss(*args_p) - loss(*args_m)) / (2 * eps)
            assert G[idx] == pytest.approx(num, abs=2e-4, rel=2e-3), (name, idx)


def test_gradient_identities():
    """sum_j dS_ij = 0 gives sum over keys of dK = 0; sum_j P_ij = 1 gives sum dV = sum dO per group."""
    B, L, Hq, Hkv, d, m = 2, 256, 4, 2, 16, 16
    Q, K, V, dO = _qkv(B, L, L, Hq, Hkv, d, 8)
    sel = _select(Q, K, m, 3, 1, 16, 8)
    _, dK, dV = oracle.attn_bwd(Q, K, V, dO, sel, m, 0.25)
    np.testing.assert_allclose(dK.sum(axis=1), 0.0, atol=1e-11)
    dO_group = dO.astype(np.float64).reshape(B, L, Hkv, Hq // Hkv, d).sum(axis=(1, 3))
    np.testing.assert_allclose(dV.sum(axis=1), dO_group, atol=1e-10)
