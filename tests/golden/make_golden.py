"""Writes the oracle's expected results for the GPU parity tests.

    python -m tests.golden.make_golden tiny reviews [groupby1b join1b sweep3b sweep3b_head]

Calls only the seeded generators (synth) and the CPU oracle (oracle); no
value here comes from the device path.  For the small workloads every
selected row goes through the oracle.  For the large ones the relational
result is complete and the logits cover a seeded sample of at least 128
selected rows: the shortest and the longest sequence, seeded picks, and more
seeded picks until every outcome of the decision (both binary outcomes, or
every label of an argmax) appears among the sampled rows.

``sweep3b`` covers the 1 % and 10 % thresholds of the selectivity sweep on
the whole 1,048,576-row table with the 3B-class model.  ``sweep3b_head``
covers the 50 % and 100 % thresholds with the same model on the table's
first 8,192 rows (the whole-table runs at those thresholds take minutes of
device time each; their relational results are checked exactly on the whole
table by the device tests).
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from oracle.query import decide, margin, relational  # noqa: E402
from synth import WORKLOADS  # noqa: E402
from synth.gen import make_model, make_tables  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))
SAMPLE = 128          # sampled rows per query of a large workload
EXTRA = 32            # rows added per round while a decision outcome is missing
MAX_EXTRA_ROUNDS = 8
HEAD_ROWS = 8192      # rows of the sweep table in the sweep3b_head golden

# golden name -> (workload, query indices, table rows (None: whole table))
GOLDENS = {
    "tiny": ("tiny", (0,), None),
    "reviews": ("reviews", (0,), None),
    "groupby1b": ("groupby1b", (0,), None),
    "join1b": ("join1b", (0,), None),
    "sweep3b": ("sweep3b", (0, 1), None),
    "sweep3b_head": ("sweep3b", (2, 3), HEAD_ROWS),
}
SAMPLED = {"groupby1b", "join1b", "sweep3b", "sweep3b_head"}


def head_rows(tables: dict, n: int) -> dict:
    """The first n rows of a probe table (its token lists included)."""
    p = tables["probe"]
    off = p["offsets"][: n + 1]
    probe = {k: v[:n] for k, v in p.items() if k not in ("offsets", "tokens")}
    probe["offsets"] = off
    probe["tokens"] = p["tokens"][: int(off[-1])]
    return {"probe": probe, "build": tables.get("build"), "prefix": tables["prefix"]}


def outcomes(query) -> set:
    """Every value the decision can take."""
    return {0, 1} if query.decision == "binary_gt" else set(int(l) for l in query.labels)


def first_sample(lens: np.ndarray, k: int, rng) -> list:
    """Shortest, longest, then seeded picks: k distinct indices (all if fewer)."""
    n = len(lens)
    if n <= k:
        return list(range(n))
    pick = [int(np.argmin(lens)), int(np.argmax(lens))]
    seen = set(pick)
    while len(pick) < k:
        i = int(rng.integers(0, n))
        if i not in seen:
            seen.add(i)
            pick.append(i)
    return pick


def sampled_logits(tables, model, query, rows, seed):
    """Oracle logits of a stratified sample of the selected rows; returns the
    sorted sample indices and their logits, labels and margins."""
    lens = tables["probe"]["len"][rows] + query.n_prefix
    rng = np.random.default_rng(seed)
    pick = first_sample(lens, SAMPLE, rng)
    prefix = tables["prefix"][: query.n_prefix]
    lg = oracle.label_logits(model, oracle.sequences(tables["probe"], rows[pick], prefix), query.labels)
    want = outcomes(query)
    for _ in range(MAX_EXTRA_ROUNDS):
        if want <= set(decide(lg, query).tolist()) or len(pick) >= len(rows):
            break
        seen = set(pick)
        more = []
        while len(more) < EXTRA and len(seen) < len(rows):
            i = int(rng.integers(0, len(rows)))
            if i not in seen:
                seen.add(i)
                more.append(i)
        lg = np.concatenate([lg, oracle.label_logits(model, oracle.sequences(tables["probe"], rows[more], prefix),
                                                     query.labels)])
        pick += more
    order = np.argsort(pick)
    idx = np.asarray(pick, dtype=np.int64)[order]
    lg = lg[order]
    return idx, lg, decide(lg, query), margin(lg, query)


def make(name: str) -> str:
    wname, queries, n_head = GOLDENS[name]
    w = WORKLOADS[wname]
    t0 = time.time()
    tables = make_tables(w)
    if n_head is not None:
        tables = head_rows(tables, n_head)
    model = make_model(w.model)
    out = {}
    for qi in queries:
        q = w.queries[qi]
        p = f"q{qi}_"
        rows, payload = relational(tables, q)
        out[p + "rows"] = rows
        if payload is not None:
            out[p + "payload"] = payload
        if name in SAMPLED:
            idx, lg, lab, mg = sampled_logits(tables, model, q, rows, 1000 + qi)
            out[p + "sample"], out[p + "logits"], out[p + "labels"], out[p + "margin"] = idx, lg, lab, mg
            print(f"{name} q{qi}: {len(rows)} selected, {len(idx)} sampled, outcomes "
                  f"{sorted(set(lab.tolist()))}, {time.time() - t0:.0f}s", flush=True)
        else:
            res = oracle.run_query(tables, model, q)
            out[p + "sample"] = res["sample"]
            out[p + "logits"] = res["logits"]
            out[p + "labels"] = res["labels"]
            out[p + "margin"] = res["margin"]
            out[p + "kept_ids"] = res["kept_ids"]
            out[p + "count"] = np.array([res["count"]])
            out[p + "n_tokens"] = np.array([res["n_tokens"]])
            if "groups" in res:
                for j, g in enumerate(res["groups"]):
                    out[p + f"groups{j}"] = g
    path = os.path.join(HERE, f"{name}_oracle.npz")
    np.savez_compressed(path, **out)
    print(f"{name}: {time.time() - t0:.1f}s -> {path}", flush=True)
    return path


if __name__ == "__main__":
    for n in sys.argv[1:] or ["tiny", "reviews"]:
        make(n)
