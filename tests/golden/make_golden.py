"""Writes the oracle's expected results for the GPU parity tests.

    python -m tests.golden.make_golden tiny reviews [groupby1b join1b sweep3b]

Calls only the seeded generators (synth) and the CPU oracle (oracle); no
value here comes from the device path.  For the small workloads every
selected row goes through the oracle; for the large ones the relational
result is complete and the logits cover a seeded sample of the selected rows
(always including the shortest and the longest sequence).
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
from oracle.query import relational  # noqa: E402
from synth import WORKLOADS  # noqa: E402
from synth.gen import make_model, make_tables  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))
SAMPLE = {"groupby1b": 24, "join1b": 24, "sweep3b": 8}


def sample_rows(lens: np.ndarray, k: int, seed: int) -> np.ndarray:
    """k indices into the selected rows: shortest, longest, then seeded picks."""
    n = len(lens)
    if n <= k:
        return np.arange(n)
    pick = {int(np.argmin(lens)), int(np.argmax(lens))}
    rng = np.random.default_rng(seed)
    while len(pick) < k:
        pick.add(int(rng.integers(0, n)))
    return np.array(sorted(pick))


def make(name: str) -> str:
    w = WORKLOADS[name]
    t0 = time.time()
    tables = make_tables(w)
    model = make_model(w.model)
    out = {}
    for qi, q in enumerate(w.queries):
        if name == "sweep3b" and qi != 0:
            # the sweep's other thresholds only change the selection; their
            # relational results are checked exactly by the device tests
            continue
        rows, payload = relational(tables, q)
        lens = tables["probe"]["len"][rows] + q.n_prefix
        sample = None if name not in SAMPLE else sample_rows(lens, SAMPLE[name], 1000 + qi)
        res = oracle.run_query(tables, model, q, sample=sample)
        p = f"q{qi}_"
        out[p + "rows"] = rows
        out[p + "sample"] = res["sample"]
        out[p + "logits"] = res["logits"]
        out[p + "labels"] = res["labels"]
        out[p + "margin"] = res["margin"]
        if payload is not None:
            out[p + "payload"] = payload
        if sample is None:
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
