"""Pins of the oracle at query positions inside a partial last block (a decode
step whose cache length is not a multiple of m): the explicit q_pos0 of the
selection and attention wrappers against brute force."""
import numpy as np
import pytest

import oracle
from tests import bruteforce as bf


@pytest.mark.parametrize("length,window,n_init,top_k", [(70, 0, 1, 3), (128, 16, 2, 2), (99, 32, 1, 10), (5, 0, 1, 2)])
def test_decode_position_in_partial_block(length, window, n_init, top_k):
    rng = np.random.default_rng(length)
    m, d, Hq, Hkv = 16, 8, 4, 2
    T_pad = -(-length // m)
    pad = T_pad * m
    q = rng.standard_normal((2, 1, Hq, d)).astype(np.float32)
    K = rng.standard_normal((2, pad, Hkv, d)).astype(np.float32)
    V = rng.standard_normal((2, pad, Hkv, d)).astype(np.float32)
    K[:, length:] = np.nan                      # past the cache length: never read
    V[:, length:] = np.nan
    punct = (rng.random((2, pad)) < 0.2).astype(np.uint8)
    Kc = bf.compress(np.nan_to_num(K), punct, m, 0.5)
    scale = d ** -0.5
    sel, kth, gap = oracle.select(q, Kc, m, top_k, n_init, window, scale, pad, q_pos0=length - 1)
    ref, _ = bf.select(q, Kc, m, top_k, n_init, window, scale, length)
    assert np.array_equal(sel, ref)
    O, LSE = oracle.attn_fwd(q, K, V, sel, m, scale, q_pos0=length - 1)
    for b in range(2):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            keys = [j for t in sel[b, g, 0] if t >= 0 for j in range(t * m, (t + 1) * m) if j < length]
            s = np.array([float(np.dot(q[b, 0, h].astype(np.float64), K[b, j, g].astype(np.float64))) for j in keys])
            s *= scale
            w = np.exp(s - s.max())
            o = (w[:, None] * V[b, keys, g].astype(np.float64)).sum(0) / w.sum()
            np.testing.assert_allclose(O[b, 0, h], o, rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(LSE[b, h, 0], s.max() + np.log(w.sum()), rtol=1e-12, atol=1e-12)
