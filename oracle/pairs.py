"""Pairs of rows classified together: Q4 of Section 4 (the self-join
``FROM t A CROSS JOIN t B WHERE ... AND A.id = B.id AND A.review_id <
B.review_id`` with ``AI_IF([A.text, B.text], prompt)``; Fig. 4 discusses its
host-transfer cost).  Test infrastructure only (see the package docstring).

Readings (the query text leaves them open):
* the WHERE predicate applies to both sides: the pairs are those of the
  filtered table;
* ``A.id = B.id`` is equality of the pair key column (the movie id) and
  ``A.review_id < B.review_id`` orders the two rows of a pair by row id (the
  row id is the review id);
* the pair's text is the prompt prefix, then A's tokens, then B's tokens;
* output: the pairs whose AI_IF decision is 1, ascending by (A, B), and their
  COUNT.
"""
from __future__ import annotations

import numpy as np


def candidate_pairs(probe: dict, rows: np.ndarray, key_col: str):
    """(A rows, B rows) of every pair of selected rows with equal keys and
    A < B, ascending by (A, B)."""
    rows = np.asarray(rows, dtype=np.int64)
    keys = np.asarray(probe[key_col]).astype(np.int64)[rows]
    a_out, b_out = [], []
    for i in range(len(rows)):
        later = np.flatnonzero(keys[i + 1:] == keys[i]) + i + 1
        a_out.extend([int(rows[i])] * len(later))
        b_out.extend(int(rows[j]) for j in later)
    return np.asarray(a_out, dtype=np.int64), np.asarray(b_out, dtype=np.int64)


def pair_sequences(probe: dict, a_rows, b_rows, prefix) -> list:
    """Token sequence of each pair: prefix, A's tokens, B's tokens."""
    off, tok = probe["offsets"], probe["tokens"]
    pre = np.asarray(prefix, dtype=np.int64)
    return [np.concatenate([pre, tok[off[a]:off[a + 1]].astype(np.int64), tok[off[b]:off[b + 1]].astype(np.int64)])
            for a, b in zip(a_rows, b_rows)]
