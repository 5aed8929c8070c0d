"""Pins of the random-selection baseline of the oracle (the component
ablation's random tokens at the same budget) -- CPU only.

The counter-based generator is checked against numpy's own Philox4x64-10
bit generator (an independent implementation of the same published
algorithm); the selection against a brute-force ordering; uniformity of the
subsets statistically."""
import numpy as np

import oracle as O


def test_philox_matches_numpy_philox_bit_generator():
    for key in ((5, 7), (0, 0), (2 ** 64 - 1, 12345)):
        bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                              counter=np.zeros(4, dtype=np.uint64))
        raw = bg.random_raw(4 * 6).reshape(6, 4)
        # numpy increments its counter before each block: blocks 1..6
        ctr = np.zeros((6, 4), np.uint64)
        ctr[:, 0] = np.arange(1, 7, dtype=np.uint64)
        np.testing.assert_array_equal(O.philox4x64_10(ctr, key), raw)


def test_philox_carries_across_counter_words():
    # a counter with a high word set equals numpy's after advancing past 2^64 blocks
    key = (9, 3)
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                          counter=np.array([2 ** 64 - 1, 4, 0, 0], dtype=np.uint64))
    raw = bg.random_raw(4)
    ctr = np.array([[0, 5, 0, 0]], np.uint64)
    np.testing.assert_array_equal(O.philox4x64_10(ctr, key)[0], raw)


def test_random_keys_grid_and_determinism():
    k = O.random_keys(11, 2, 3, 50)
    assert k.shape == (2, 3, 50) and k.dtype == np.float32
    assert (k >= 0).all() and (k < 1).all()
    assert np.all(k * 2.0 ** 24 == np.floor(k * 2.0 ** 24))      # on the 2^-24 grid
    np.testing.assert_array_equal(k, O.random_keys(11, 2, 3, 50))
    assert not np.array_equal(k, O.random_keys(12, 2, 3, 50))


def test_random_selection_is_the_top_keys_with_index_ties():
    rng = np.random.default_rng(0)
    keys = (rng.integers(0, 8, (3, 40)) / 8.0).astype(np.float32)   # many ties
    sel = O.random_selection(keys, 13)
    for f in range(3):
        order = sorted(range(40), key=lambda j: (-keys[f, j], j))[:13]
        np.testing.assert_array_equal(sel.retained[f], np.sort(order))
        assert len(sel.anchors) == 0


def test_random_subsets_are_uniform():
    # inclusion frequency of every position is k / N within 5 sigma over many seeds
    N, k, n = 24, 6, 3000
    hits = np.zeros(N)
    for seed in range(n // 10):
        keys = O.random_keys(seed, 1, 10, N)[0]
        for f in range(10):
            hits[O.random_selection(keys[f:f + 1], k).retained[0]] += 1
    p = k / N
    sd = np.sqrt(n * p * (1 - p))
    assert np.all(np.abs(hits - n * p) < 5 * sd), hits
