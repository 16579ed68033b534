"""Pins of the oracle's SOFTMAX_SUM selection mode: Eq. 8's softmax per query
head, the group's heads combined by summing probabilities, each softmax over
the complete blocks before the query's own block."""
import itertools
import math

import numpy as np
import pytest

import oracle
from tests import bruteforce as bf

SM = oracle.SOFTMAX_SUM


def _case(B, L, Hq, Hkv, d, seed):
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((B, L, Hq, d)).astype(np.float32)
    K = rng.standard_normal((B, L, Hkv, d)).astype(np.float32)
    punct = (rng.random((B, L)) < 0.1).astype(np.uint8)
    return Q, K, punct


def _worked(a5=1.0):
    """Two heads, six blocks of two tokens, one query at position 11 (block 5).
    Representatives are unit vectors, so head h's logit of block t is q_h[t]
    (scale 1).  exp(logits) over blocks 0..4: head 0 = [1, 4, 2.5, 1, 1]
    (sum 19/2), head 1 = [100, 1, 2, 1, 1] (sum 105); a5 = exp(head 0's logit
    of the diagonal block 5), which the softmax must not see."""
    a = [1.0, 4.0, 2.5, 1.0, 1.0, a5]
    b = [100.0, 1.0, 2.0, 1.0, 1.0, 1.0]
    Q = np.zeros((1, 1, 2, 6), np.float32)
    Q[0, 0, 0] = np.log(a)
    Q[0, 0, 1] = np.log(b)
    Kc = np.eye(6)[None, None]                     # [1, 1, T = 6, d = 6]
    return Q, Kc


@pytest.mark.parametrize("a5", [1.0, 1000.0])
def test_worked_example_closed_form(a5):
    """Block 1 has p = 8/19 + 1/105 = 859/1995, block 2 has 5/19 + 2/105 = 563/1995,
    blocks 3 and 4 have 2/19 + 1/105 = 229/1995.  Summed logits would rank block 2
    first (log 2.5 + log 2 > log 4 + log 1); the softmax sum ranks block 1 first.
    Leaving block 0 (forced) out of the normaliser would also pick block 2, and
    so would letting the diagonal block in when its logit is large."""
    Q, Kc = _worked(a5)
    sel, kth, gap = oracle.select(Q, Kc, 2, 1, 1, 0, 1.0, 12, mode=SM)
    assert sel[0, 0, 0].tolist() == [0, 1, 5]
    assert kth[0, 0, 0] == pytest.approx(math.log(859 / 1995), abs=1e-6)
    assert gap[0, 0, 0] == pytest.approx(math.log(859 / 563), abs=1e-6)
    sel2, kth2, gap2 = oracle.select(Q, Kc, 2, 2, 1, 0, 1.0, 12, mode=SM)
    assert sel2[0, 0, 0].tolist() == [0, 1, 2, 5]
    assert kth2[0, 0, 0] == pytest.approx(math.log(563 / 1995), abs=1e-6)
    assert gap2[0, 0, 0] == pytest.approx(math.log(563 / 229), abs=1e-6)
    logit, _, _ = oracle.select(Q, Kc, 2, 1, 1, 0, 1.0, 12)
    assert logit[0, 0, 0].tolist() == [0, 2, 5]
    row = oracle.score_row(Q, Kc, 2, 1.0, 12, 0, 0, 0, mode=SM)
    np.testing.assert_allclose(np.exp(row[:5]), np.array([100 / 105 + 2 / 19, 859 / 1995, 563 / 1995,
                                                          229 / 1995, 229 / 1995]), rtol=1e-6)
    assert row[5] == -np.inf


CASES = [
    # B, L, Hq, Hkv, d, m, top_k, n_init, window
    (1, 64, 2, 1, 8, 4, 2, 1, 0),
    (2, 128, 4, 2, 16, 8, 3, 1, 8),
    (1, 256, 8, 2, 8, 8, 7, 3, 24),
    (1, 192, 2, 2, 4, 16, 5, 0, 16),
    (1, 128, 4, 1, 8, 4, 40, 1, 0),
]


@pytest.mark.parametrize("case", CASES)
def test_bruteforce(case):
    B, L, Hq, Hkv, d, m, k, n_init, w = case
    Q, K, punct = _case(B, L, Hq, Hkv, d, sum(case))
    Kc = oracle.compress(K, punct, m, 0.5)
    scale = d ** -0.5
    sel, kth, gap = oracle.select(Q, Kc, m, k, n_init, w, scale, L, mode=SM)
    ref, S = bf.select(Q, Kc, m, k, n_init, w, scale, L, softmax_sum=True)
    np.testing.assert_array_equal(sel, ref)
    for b, g, i in itertools.product(range(B), range(Hkv), range(0, L, 5)):
        cur = i // m
        t = np.arange(cur + 1)
        forced = (t < n_init) | (t >= cur - w // m)
        cs = np.sort(S[b, g, i, t[~forced]])[::-1]
        if cs.size == 0:
            assert np.isnan(kth[b, g, i])
            continue
        npick = min(k, cs.size)
        assert kth[b, g, i] == pytest.approx(cs[npick - 1], abs=1e-10)
        if cs.size > npick:
            assert gap[b, g, i] == pytest.approx(cs[npick - 1] - cs[npick], abs=1e-10)
        row = oracle.score_row(Q, Kc, m, scale, L, b, i, g, mode=SM)
        np.testing.assert_allclose(row[:cur], S[b, g, i, :cur], atol=1e-10)


def test_single_head_matches_summed_logits():
    """G = 1: softmax is monotone within a row, so the selection and the gaps
    equal those of the summed-logit mode (the score only shifts by the row's
    log normaliser)."""
    Q, K, punct = _case(2, 256, 2, 2, 8, 3)
    Kc = oracle.compress(K, punct, 8, 0.5)
    a, ka, ga = oracle.select(Q, Kc, 8, 5, 1, 8, 0.4, 256)
    b, kb, gb = oracle.select(Q, Kc, 8, 5, 1, 8, 0.4, 256, mode=SM)
    np.testing.assert_array_equal(a, b)
    ok = np.isfinite(ga)
    np.testing.assert_allclose(gb[ok], ga[ok], atol=1e-9)


def test_identical_heads_match_summed_logits():
    """Two heads with the same query have the same softmax, so the sum is twice
    one monotone function of the logit: same selection as summed logits."""
    Q, K, punct = _case(1, 256, 1, 1, 8, 4)
    Q2 = np.repeat(Q, 2, axis=2)
    Kc = oracle.compress(K, punct, 16, 0.5)
    a, _, _ = oracle.select(Q2, Kc, 16, 4, 1, 0, 0.4, 256)
    b, _, _ = oracle.select(Q2, Kc, 16, 4, 1, 0, 0.4, 256, mode=SM)
    np.testing.assert_array_equal(a, b)


def test_zero_query_head_has_no_say():
    """A head with q = 0 spreads 1/cur over blocks 0..cur-1, the same amount for
    every candidate, so the selection is that of the other head alone."""
    Q, K, punct = _case(1, 256, 2, 1, 8, 5)
    Q[:, :, 1] = 0.0
    Kc = oracle.compress(K, punct, 8, 0.5)
    a, _, _ = oracle.select(Q, Kc, 8, 3, 2, 16, 0.4, 256, mode=SM)
    b, _, _ = oracle.select(Q[:, :, :1], Kc, 8, 3, 2, 16, 0.4, 256, mode=SM)
    np.testing.assert_array_equal(a, b)


def test_head_permutation_within_group():
    Q, K, punct = _case(1, 128, 4, 2, 8, 6)
    Kc = oracle.compress(K, punct, 8, 0.5)
    a, _, _ = oracle.select(Q, Kc, 8, 4, 1, 8, 0.3, 128, mode=SM)
    b, _, _ = oracle.select(Q[:, :, [1, 0, 3, 2]], Kc, 8, 4, 1, 8, 0.3, 128, mode=SM)
    np.testing.assert_array_equal(a, b)


def test_decode_position_and_invariants():
    Q, K, punct = _case(2, 512, 4, 2, 8, 7)
    Kc = oracle.compress(K, punct, 32, 0.5)
    one, _, _ = oracle.select(Q[:, -1:], Kc, 32, 3, 1, 32, 0.35, 512, mode=SM)
    full, _, _ = oracle.select(Q, Kc, 32, 3, 1, 32, 0.35, 512, mode=SM)
    np.testing.assert_array_equal(one[:, :, 0], full[:, :, -1])
    for b, g, i in itertools.product(range(2), range(2), range(0, 512, 3)):
        row = full[b, g, i]
        valid = row[row >= 0]
        cur = i // 32
        assert (np.diff(valid) > 0).all() and valid.max() == cur
        assert valid.size == min(cur + 1, len(set(range(min(1, cur + 1))) | set(range(max(0, cur - 1), cur + 1))) + 3)
