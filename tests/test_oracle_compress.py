"""Pins of the oracle's block representatives (Eq. 3, 6, 7, 8)."""
import json
import os

import numpy as np
import pytest

import oracle
from tests import bruteforce as bf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_example.json")


def _rand(shape, seed, ints=False):
    rng = np.random.default_rng(seed)
    if ints:
        return rng.integers(-8, 9, size=shape).astype(np.float32)
    return rng.standard_normal(shape).astype(np.float32)


@pytest.mark.parametrize("lam", ["0.5", "0.25", "1.0", "0.0"])
def test_worked_example(lam):
    """The paper's tokenised sentence: ids 11 and 13 are punctuation, m = 4."""
    g = json.load(open(GOLDEN))
    ids = np.array(g["token_ids"])
    mask = np.isin(ids, g["punctuation_ids"]).astype(np.uint8)
    assert mask.tolist() == g["expected_mask"]
    i = np.arange(ids.size, dtype=np.float32)
    K = np.stack([i, i * i], axis=-1)[None, :, None, :]              # [1, 12, 1, 2]
    Kc = oracle.compress(K, mask[None], g["block_size"], float(lam))
    np.testing.assert_array_equal(Kc[0, 0], np.array(g["expected"][lam]))


@pytest.mark.parametrize("lam", [0.0, 0.3, 0.5, 1.0])
def test_zero_mask_is_mean_pooling(lam):
    """No punctuation anywhere: the representative is the plain block mean."""
    K = _rand((2, 96, 3, 8), 1)
    Kc = oracle.compress(K, np.zeros((2, 96), np.uint8), 16, lam)
    ref = K.astype(np.float64).reshape(2, 6, 16, 3, 8).mean(axis=2).transpose(0, 2, 1, 3)
    np.testing.assert_allclose(Kc, ref, rtol=0, atol=1e-12)


def test_all_punct_is_mean_pooling():
    K = _rand((1, 64, 2, 4), 2)
    Kc = oracle.compress(K, np.ones((1, 64), np.uint8), 8, 0.37)
    ref = K.astype(np.float64).reshape(1, 8, 8, 2, 4).mean(axis=2).transpose(0, 2, 1, 3)
    np.testing.assert_allclose(Kc, ref, rtol=0, atol=1e-12)


def test_lambda_zero_is_punctuation_mean():
    K = _rand((1, 64, 1, 4), 3)
    mask = np.zeros((1, 64), np.uint8)
    mask[0, [1, 5, 6, 17, 40, 41, 42]] = 1
    Kc = oracle.compress(K, mask, 16, 0.0)
    Kd = K.astype(np.float64)[0, :, 0]
    np.testing.assert_allclose(Kc[0, 0, 0], Kd[[1, 5, 6]].mean(0), atol=1e-12)
    np.testing.assert_allclose(Kc[0, 0, 1], Kd[[17]].mean(0), atol=1e-12)
    np.testing.assert_allclose(Kc[0, 0, 2], Kd[[40, 41, 42]].mean(0), atol=1e-12)
    np.testing.assert_allclose(Kc[0, 0, 3], Kd[48:64].mean(0), atol=1e-12)   # fallback


def test_single_punct_token():
    """One punctuation token j in a block: M = lam * M0 + (1 - lam) * K_j."""
    K = _rand((1, 32, 1, 6), 4)
    mask = np.zeros((1, 32), np.uint8)
    mask[0, 21] = 1
    lam = 0.7
    Kc = oracle.compress(K, mask, 16, lam)
    Kd = K.astype(np.float64)[0, :, 0]
    np.testing.assert_allclose(Kc[0, 0, 1], lam * Kd[16:32].mean(0) + (1 - lam) * Kd[21], atol=1e-12)


def test_linearity_in_keys():
    """Fixed mask: compress(a K1 + b K2) = a compress(K1) + b compress(K2) (integer keys, exact)."""
    K1, K2 = _rand((2, 128, 2, 8), 5, ints=True), _rand((2, 128, 2, 8), 6, ints=True)
    mask = (np.random.default_rng(7).random((2, 128)) < 0.2).astype(np.uint8)
    lhs = oracle.compress(3 * K1 - 2 * K2, mask, 32, 0.5)
    rhs = 3 * oracle.compress(K1, mask, 32, 0.5) - 2 * oracle.compress(K2, mask, 32, 0.5)
    np.testing.assert_allclose(lhs, rhs, atol=1e-12)


def test_permutation_within_block():
    """Pooling is order-free inside a block: shuffling a block's tokens (with their mask bits) changes nothing."""
    K = _rand((1, 64, 2, 8), 8)
    mask = (np.random.default_rng(9).random((1, 64)) < 0.3).astype(np.uint8)
    perm = np.concatenate([np.random.default_rng(10).permutation(16) + 16 * t for t in range(4)])
    a = oracle.compress(K, mask, 16, 0.4)
    b = oracle.compress(K[:, perm], mask[:, perm], 16, 0.4)
    np.testing.assert_allclose(a, b, atol=1e-12)


@pytest.mark.parametrize("m", [4, 8, 16, 64])
def test_bruteforce(m):
    K = _rand((2, 256, 3, 16), 11 + m)
    mask = (np.random.default_rng(m).random((2, 256)) < 0.1).astype(np.uint8)
    for lam in (0.0, 0.25, 0.5, 1.0):
        np.testing.assert_allclose(oracle.compress(K, mask, m, lam), bf.compress(K, mask, m, lam),
                                   rtol=1e-12, atol=1e-12)
