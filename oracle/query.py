"""End-to-end oracle of one AI query.  Test infrastructure only.

Order of steps (Table 1 and Figure 2 of the paper, Section 3.1):
FROM (input arrays) -> WHERE (boolean mask, optional join) -> AI_IF (causal LM
forward per selected row, last-position label logits, decision) -> aggregate.
"""
from __future__ import annotations

import numpy as np

from .relational import select, hash_join, sequences, group_avg_count, count_by, sum_f32
from .transformer import label_logits


def relational(tables: dict, query):
    """Selected probe rows (ascending) and, for a join, the build payload per row."""
    probe = tables["probe"]
    rows = select(probe, query.preds, len(probe["id"]))
    payload = None
    if query.join is not None:
        rows, payload = hash_join(probe, tables["build"], query.join, rows)
    return rows, payload


def decide(logits: np.ndarray, query) -> np.ndarray:
    """Label value per row.

    binary_gt: 1 when the first label's logit is strictly greater than the
    second's (the ``score_yes > score_no`` filter of Figure 2), else 0.
    argmax: the label token id with the largest logit, ties to the lowest index."""
    logits = np.asarray(logits)
    if query.decision == "binary_gt":
        return (logits[:, 0] > logits[:, 1]).astype(np.int64)
    return np.asarray(query.labels, dtype=np.int64)[np.argmax(logits, axis=1)]


def margin(logits: np.ndarray, query) -> np.ndarray:
    """Distance of each row's decision from a tie."""
    logits = np.asarray(logits)
    if query.decision == "binary_gt":
        return np.abs(logits[:, 0] - logits[:, 1])
    s = np.sort(logits, axis=1)
    return s[:, -1] - s[:, -2]


def aggregate(tables: dict, rows: np.ndarray, payload, labels: np.ndarray, query) -> dict:
    """Final aggregate from per-row labels (the masked reduction of Table 1 and
    the ``jnp.where(filter, values, 0).sum()`` of Figure 2, as COUNT / GROUP BY)."""
    probe = tables["probe"]
    labels = np.asarray(labels, dtype=np.int64)
    if query.decision == "binary_gt":
        keep = labels == 1
        kept = rows[keep]
    else:
        keep = np.ones(len(rows), dtype=bool)
        kept = rows
    out = {"kept_ids": kept.astype(np.int64), "count": int(len(kept))}
    if query.agg == "avg_label_count_by":
        keys = probe[query.group_col][rows].astype(np.int64)
        out["groups"] = group_avg_count(keys, labels)
    elif query.agg == "count_by_payload":
        k, c = count_by(np.asarray(payload, dtype=np.int64)[keep])
        out["groups"] = (k, c, np.zeros_like(c), np.zeros(len(c)))
    elif query.agg == "sum_f32":
        out["sum"] = sum_f32(probe[query.group_col][kept])
    return out


def run_query(tables: dict, model: dict, query, sample=None) -> dict:
    """Runs the whole query.  ``sample`` (indices into the selected rows) limits
    the transformer to those rows; the aggregate is then not computed."""
    rows, payload = relational(tables, query)
    prefix = tables["prefix"][: query.n_prefix]
    res = {"rows": rows, "payload": payload}
    idx = np.arange(len(rows)) if sample is None else np.asarray(sample, dtype=np.int64)
    seqs = sequences(tables["probe"], rows[idx], prefix)
    lg = label_logits(model, seqs, query.labels)
    res.update(sample=idx, logits=lg, labels=decide(lg, query), margin=margin(lg, query),
               n_tokens=int(sum(len(s) for s in seqs)))
    if sample is None:
        res.update(aggregate(tables, rows, payload, res["labels"], query))
    return res

