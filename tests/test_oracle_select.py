"""Pins of the oracle's block selection (Eq. 8 logits, Algorithm 1 selection)."""
import itertools

import numpy as np
import pytest

import oracle
from tests import bruteforce as bf


def _case(B, L, Hq, Hkv, d, m, seed, p=0.1):
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((B, L, Hq, d)).astype(np.float32)
    K = rng.standard_normal((B, L, Hkv, d)).astype(np.float32)
    punct = (rng.random((B, L)) < p).astype(np.uint8)
    return Q, K, punct


CASES = [
    # B, L, Hq, Hkv, d, m, top_k, n_init, window
    (1, 64, 2, 1, 8, 4, 2, 1, 0),
    (2, 128, 4, 2, 16, 8, 3, 1, 8),
    (1, 256, 4, 1, 8, 16, 4, 2, 32),
    (2, 192, 2, 2, 4, 16, 5, 0, 16),
    (1, 256, 8, 2, 8, 8, 7, 3, 24),
    (1, 128, 1, 1, 8, 4, 40, 1, 0),    # top_k larger than any candidate set
]


@pytest.mark.parametrize("case", CASES)
def test_bruteforce(case):
    B, L, Hq, Hkv, d, m, k, n_init, w = case
    Q, K, punct = _case(B, L, Hq, Hkv, d, m, sum(case))
    Kc = oracle.compress(K, punct, m, 0.5)
    scale = d ** -0.5
    sel, kth, gap = oracle.select(Q, Kc, m, k, n_init, w, scale, L)
    ref, S = bf.select(Q, Kc, m, k, n_init, w, scale, L)
    np.testing.assert_array_equal(sel, ref)
    # kth / gap: the k-th best candidate score and its margin over the next one
    for b, g, i in itertools.product(range(B), range(Hkv), range(0, L, 7)):
        cur = i // m
        t = np.arange(cur + 1)
        forced = (t < n_init) | (t >= cur - w // m)
        cs = np.sort(S[b, g, i, t[~forced]])[::-1]
        if cs.size == 0:
            assert np.isnan(kth[b, g, i])
            continue
        npick = min(k, cs.size)
        assert kth[b, g, i] == pytest.approx(cs[npick - 1], abs=1e-12)
        if cs.size > npick:
            assert gap[b, g, i] == pytest.approx(cs[npick - 1] - cs[npick], abs=1e-12)
        else:
            assert np.isinf(gap[b, g, i])


@pytest.mark.parametrize("case", CASES)
def test_invariants(case):
    B, L, Hq, Hkv, d, m, k, n_init, w = case
    Q, K, punct = _case(B, L, Hq, Hkv, d, m, 100 + sum(case))
    Kc = oracle.compress(K, punct, m, 0.3)
    sel, _, _ = oracle.select(Q, Kc, m, k, n_init, w, d ** -0.5, L)
    ksel = n_init + w // m + 1 + k
    assert sel.shape == (B, Hkv, L, ksel)
    for b, g, i in itertools.product(range(B), range(Hkv), range(L)):
        row = sel[b, g, i]
        cur = i // m
        valid = row[row >= 0]
        assert (row[valid.size:] == -1).all()                     # padding only at the end
        assert (np.diff(valid) > 0).all()                         # ascending, no duplicates
        assert valid.min() >= 0 and valid.max() <= cur            # causal
        forced = set(range(min(n_init, cur + 1))) | set(range(max(0, cur - w // m), cur + 1))
        assert forced <= set(valid.tolist())                      # forced blocks always kept
        assert valid.size == min(cur + 1, len(forced) + k)        # size of the final set


def test_all_blocks_when_k_covers_candidates():
    Q, K, punct = _case(1, 256, 2, 1, 8, 16, 3)
    Kc = oracle.compress(K, punct, 16, 0.5)
    sel, _, _ = oracle.select(Q, Kc, 16, 16, 1, 0, 0.35, 256)
    for i in range(256):
        cur = i // 16
        assert sel[0, 0, i, :cur + 1].tolist() == list(range(cur + 1))


def test_head_permutation_within_group():
    """The group score sums over the group's heads, so their order does not matter."""
    Q, K, punct = _case(1, 256, 4, 2, 8, 8, 4)
    Kc = oracle.compress(K, punct, 8, 0.5)
    a, _, _ = oracle.select(Q, Kc, 8, 5, 1, 8, 0.3, 256)
    b, _, _ = oracle.select(Q[:, :, [1, 0, 3, 2]], Kc, 8, 5, 1, 8, 0.3, 256)
    np.testing.assert_array_equal(a, b)


def test_planted_block_is_selected():
    """Block t* whose keys all point along the query gets the strictly largest score."""
    rng = np.random.default_rng(5)
    L, m, d = 512, 16, 16
    Q = rng.standard_normal((1, L, 1, d)).astype(np.float32) * 0.01
    K = rng.standard_normal((1, L, 1, d)).astype(np.float32) * 0.01
    i, tstar = 500, 13
    Q[0, i, 0] = 1.0
    K[0, tstar * m:(tstar + 1) * m, 0] = 1.0
    punct = (rng.random((1, L)) < 0.2).astype(np.uint8)
    Kc = oracle.compress(K, punct, m, 0.5)
    sel, _, _ = oracle.select(Q, Kc, m, 1, 1, 0, d ** -0.5, L)
    assert sel[0, 0, i].tolist() == [0, tstar, i // m]


def test_zero_mask_selection_is_mean_pooling_selection():
    Q, K, _ = _case(1, 256, 2, 1, 8, 16, 6)
    zero = np.zeros((1, 256), np.uint8)
    Kc = oracle.compress(K, zero, 16, 0.5)
    mean = K.astype(np.float64).reshape(1, 16, 16, 1, 8).mean(axis=2).transpose(0, 2, 1, 3)
    sel, _, _ = oracle.select(Q, Kc, 16, 3, 1, 0, 0.35, 256)
    ref, _ = bf.select(Q, mean, 16, 3, 1, 0, 0.35, 256)
    np.testing.assert_array_equal(sel, ref)


def test_tiny_config_early_rows():
    """1024 tokens, m = 64, one init block, diagonal block, 2 free picks (4 slots)."""
    Q, K, punct = _case(1, 1024, 2, 1, 64, 64, 7)
    Kc = oracle.compress(K, punct, 64, 0.5)
    sel, _, _ = oracle.select(Q, Kc, 64, 2, 1, 0, 0.125, 1024)
    assert sel[0, 0, 0].tolist() == [0, -1, -1, -1]
    assert sel[0, 0, 64].tolist() == [0, 1, -1, -1]
    assert sel[0, 0, 128].tolist() == [0, 1, 2, -1]
    assert sel[0, 0, 200].tolist() == [0, 1, 2, 3]
    assert (sel[0, 0, 256:] >= 0).all()


def test_decode_position():
    """One query at the last position sees every block; its own block is forced."""
    Q, K, punct = _case(3, 512, 2, 1, 8, 64, 8)
    Kc = oracle.compress(K, punct, 64, 0.5)
    sel, _, _ = oracle.select(Q[:, -1:], Kc, 64, 3, 1, 0, 0.35, 512)
    full, _, _ = oracle.select(Q, Kc, 64, 3, 1, 0, 0.35, 512)
    np.testing.assert_array_equal(sel[:, :, 0], full[:, :, -1])
    assert (sel[:, :, 0, -1] == 7).all()


def test_row_subset_matches_full():
    Q, K, punct = _case(2, 256, 4, 2, 8, 16, 9)
    Kc = oracle.compress(K, punct, 16, 0.5)
    full, kth, gap = oracle.select(Q, Kc, 16, 4, 1, 16, 0.3, 256)
    rows = np.array([0, 17, 255, 256 + 3, 511])
    sub, skth, sgap = oracle.select(Q, Kc, 16, 4, 1, 16, 0.3, 256, rows=rows)
    for r, row in enumerate(rows):
        b, i = divmod(int(row), 256)
        np.testing.assert_array_equal(sub[r], full[b, :, i])
        np.testing.assert_array_equal(skth[r], kth[b, :, i])


def test_score_row():
    Q, K, punct = _case(1, 128, 4, 2, 8, 16, 10)
    Kc = oracle.compress(K, punct, 16, 0.5)
    S = bf.group_scores(Q, Kc, 0.3)
    np.testing.assert_allclose(oracle.score_row(Q, Kc, 16, 0.3, 128, 0, 77, 1), S[0, 1, 77], atol=1e-12)
