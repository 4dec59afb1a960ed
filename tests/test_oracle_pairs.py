"""Pins of the pair enumeration of oracle/pairs.py: brute force over all
ordered pairs, the per-key count identity, order, and the pair text."""
import itertools

import numpy as np

from oracle.pairs import candidate_pairs, pair_sequences


def table(n, n_keys, seed):
    r = np.random.default_rng(seed)
    lens = r.integers(0, 5, n)
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    return {"movie_id": r.integers(0, n_keys, n).astype(np.int32), "offsets": off,
            "tokens": r.integers(0, 50, int(off[-1])).astype(np.int32)}


def test_pairs_equal_brute_force_over_all_row_pairs():
    for seed in range(20):
        t = table(40, 6, seed)
        rows = np.sort(np.random.default_rng(seed + 100).choice(40, 25, replace=False))
        a, b = candidate_pairs(t, rows, "movie_id")
        want = [(int(x), int(y)) for x, y in itertools.combinations(rows, 2)
                if t["movie_id"][x] == t["movie_id"][y]]
        assert list(zip(a.tolist(), b.tolist())) == want    # combinations() yields (A, B) ascending


def test_pair_count_is_sum_of_key_group_pairs():
    t = table(500, 9, 3)
    rows = np.arange(500)
    a, _ = candidate_pairs(t, rows, "movie_id")
    _, counts = np.unique(t["movie_id"], return_counts=True)
    assert len(a) == int(np.sum(counts * (counts - 1) // 2))


def test_pairs_single_rows_and_distinct_keys_give_none():
    t = table(10, 1000, 4)
    t["movie_id"] = np.arange(10, dtype=np.int32)
    a, b = candidate_pairs(t, np.arange(10), "movie_id")
    assert len(a) == len(b) == 0
    a, b = candidate_pairs(t, np.array([3]), "movie_id")
    assert len(a) == 0


def test_pair_text_is_prefix_then_a_then_b():
    t = {"offsets": np.array([0, 2, 2, 5]), "tokens": np.array([7, 8, 9, 10, 11])}
    seqs = pair_sequences(t, [0, 0, 1], [1, 2, 2], [1, 2])
    assert [s.tolist() for s in seqs] == [[1, 2, 7, 8], [1, 2, 7, 8, 9, 10, 11], [1, 2, 9, 10, 11]]
