"""Oracle pins for the punctuation indicator I(x_i in P) of Eq. 7 (Section 3.2)."""
import json
import os

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_example.json")


def test_worked_example_mask():
    """The paper's tokenised sentence: ids 11 (',') and 13 ('.') are the punctuation."""
    g = json.load(open(GOLDEN))
    mask = oracle.punct_mask(g["token_ids"], g["punctuation_ids"])
    assert mask.tolist() == g["expected_mask"]


def test_against_set_membership():
    rng = np.random.default_rng(0)
    for trial in range(20):
        ids = rng.integers(-5, 300, size=(3, 257), dtype=np.int32)
        pset = rng.choice(np.arange(-5, 300), size=int(rng.integers(0, 40)), replace=False).astype(np.int32)
        want = np.array([[1 if int(x) in set(pset.tolist()) else 0 for x in row] for row in ids], dtype=np.uint8)
        assert np.array_equal(oracle.punct_mask(ids, pset), want)


def test_special_cases():
    ids = np.arange(100, dtype=np.int32)
    assert oracle.punct_mask(ids, []).sum() == 0                        # empty set: no punctuation
    assert oracle.punct_mask(ids, ids).all()                            # every id is punctuation
    assert oracle.punct_mask(ids, [7, 7, 7]).tolist() == [int(i == 7) for i in range(100)]   # duplicates
    assert oracle.punct_mask(np.zeros(0, np.int32), [1]).shape == (0,)  # no tokens
    big = np.array([np.iinfo(np.int32).min, np.iinfo(np.int32).max, 0], dtype=np.int32)
    assert oracle.punct_mask(big, [np.iinfo(np.int32).max]).tolist() == [0, 1, 0]
