"""Relational part of the oracle: WHERE masks, selection, PK-FK join, packing,
aggregates.  Test infrastructure only (see the package docstring).

Semantics follow Table 1 of the paper (Section 3.1): a WHERE clause becomes an
element-wise boolean mask over the column arrays; an aggregate is a reduction
over the rows the final mask keeps.  Comparisons are exact: integer columns
widened to int64, fp32 columns widened to fp64 and compared with the fp64
constant (IEEE semantics: NaN fails every ordered comparison and EQ, passes NE).
"""
from __future__ import annotations

import numpy as np

_CMP = {
    "lt": np.less, "le": np.less_equal, "gt": np.greater, "ge": np.greater_equal,
    "eq": np.equal, "ne": np.not_equal,
}


def eval_pred(cols: dict, pred) -> np.ndarray:
    """Boolean mask of one atom ``col op k`` or ``col IN (values)`` (Table 1, WHERE row)."""
    col = np.asarray(cols[pred.col])
    if col.dtype.kind == "f":
        if pred.op == "in":
            raise ValueError("IN is defined for integer columns only")
        return _CMP[pred.op](col.astype(np.float64), np.float64(pred.k))
    v = col.astype(np.int64)
    if pred.op == "in":
        m = np.zeros(v.shape, dtype=bool)
        for x in pred.values:
            m |= v == np.int64(x)
        return m
    return _CMP[pred.op](v, np.int64(pred.k))


def select(cols: dict, preds, n_rows: int) -> np.ndarray:
    """Row ids, ascending, of the rows satisfying the conjunction of ``preds``.

    The empty conjunction keeps every row."""
    m = np.ones(n_rows, dtype=bool)
    for p in preds:
        m &= eval_pred(cols, p)
    return np.flatnonzero(m).astype(np.int64)


def hash_join(probe: dict, build: dict, join, probe_rows: np.ndarray):
    """Inner PK-FK equi-join of the probe rows with the build rows that pass the
    build-side predicates (the reviews JOIN movies ON movie_id of Section 4).

    For each probe row, in ascending order, the build row with the same key is
    looked up; the probe row is kept when that row exists and passes.  Returns
    (kept probe rows, payload of the matched build row).  A duplicate build key
    among the passing build rows is an error (the key is a primary key)."""
    nb = len(build[join.build_key])
    passing = select(build, join.build_preds, nb)
    index = {}
    for b in passing:
        key = int(build[join.build_key][b])
        if key in index:
            raise ValueError("duplicate build key %d" % key)
        index[key] = int(b)
    keys = probe[join.probe_key]
    payload = build[join.payload]
    rows, pay = [], []
    for r in probe_rows:
        b = index.get(int(keys[r]))
        if b is not None:
            rows.append(int(r))
            pay.append(int(payload[b]))
    return np.asarray(rows, dtype=np.int64), np.asarray(pay, dtype=np.int64)


def sequences(probe: dict, rows: np.ndarray, prefix: np.ndarray) -> list:
    """Token sequence of each selected row: the prompt prefix followed by the
    row's own token list (the FROM-clause input arrays of Table 1, without the
    padding to a static length that the paper's prototype uses)."""
    off, tok = probe["offsets"], probe["tokens"]
    pre = np.asarray(prefix, dtype=np.int64)
    return [np.concatenate([pre, tok[off[r]:off[r + 1]].astype(np.int64)]) for r in rows]


def pack(seqs: list):
    """Concatenation of the sequences and their boundaries ``cu[i]..cu[i+1]``."""
    cu = np.zeros(len(seqs) + 1, dtype=np.int64)
    for i, s in enumerate(seqs):
        cu[i + 1] = cu[i] + len(s)
    flat = np.concatenate(seqs) if seqs else np.zeros(0, dtype=np.int64)
    return cu, flat


def group_avg_count(keys: np.ndarray, values: np.ndarray):
    """GROUP BY key: (key, COUNT(*), SUM(value), AVG(value)) for every key present,
    in ascending key order.  COUNT and SUM are exact integers; AVG is the fp64
    quotient SUM / COUNT."""
    keys = np.asarray(keys, dtype=np.int64)
    values = np.asarray(values, dtype=np.int64)
    uk = np.unique(keys)
    out_k, out_c, out_s, out_a = [], [], [], []
    for k in uk:
        sel = keys == k
        c = int(sel.sum())
        s = int(values[sel].sum())
        out_k.append(int(k))
        out_c.append(c)
        out_s.append(s)
        out_a.append(float(s) / float(c))
    return (np.asarray(out_k, dtype=np.int64), np.asarray(out_c, dtype=np.int64),
            np.asarray(out_s, dtype=np.int64), np.asarray(out_a, dtype=np.float64))


def count_by(keys: np.ndarray):
    """GROUP BY key COUNT(*), ascending key order, present keys only."""
    k, c, _, _ = group_avg_count(keys, np.zeros(len(keys), dtype=np.int64))
    return k, c


def sum_f32(values: np.ndarray) -> float:
    """SUM of an fp32 column over the kept rows (the float aggregate of the
    paper's running query, Table 1 SUM row and Figure 2): the exact sum of the
    values, rounded once to fp64 (math.fsum).  Non-finite values follow IEEE
    addition, whose result then does not depend on the order: NaN if any
    value is NaN or both infinities occur, else the infinity."""
    import math
    v = np.asarray(values, dtype=np.float32).astype(np.float64)
    if not np.isfinite(v).all():
        if np.isnan(v).any() or (np.isposinf(v).any() and np.isneginf(v).any()):
            return float("nan")
        return float("inf") if np.isposinf(v).any() else float("-inf")
    return math.fsum(v.tolist())

