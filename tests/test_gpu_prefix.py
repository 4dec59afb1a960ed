"""Shared prompt prefix on the MFMA path (a prompted AI_IF, Table 1; the join
query of Section 4 puts a 32-token instruction before every review).

The device prefills the prefix once and every row attends to its kept keys and
values.  Pinned three ways:
* against the per-row computation on the device (AIQ_PLAN_UNSHARED_PREFIX):
  label logits bit-identical, for prefix lengths on both sides of the 64-key
  block edge, head dims 64 and 128, several chunks, and rows with no own token;
* against the oracle (prefix || row tokens, per sequence, fp64) within the
  bf16 tolerance, on a sample that includes the shortest and longest rows;
* token totals: the prefix counted once per selected row in both modes.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle.query import aggregate, decide, margin, relational
from paper_2608_10139_amd.device import DeviceModel, DeviceQuery
from synth.configs import ModelSpec, Pred, Query
from synth.gen import make_model
from tests._parity import TOL_BF16, check_labels

pytestmark = pytest.mark.gpu

MODELS = {
    "hd64": ModelSpec(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, d_ff=512, vocab=1000, act="swiglu",
                      dtype="bf16", weight_seed=21),
    "hd128": ModelSpec(n_layers=2, d_model=512, n_heads=4, n_kv_heads=2, d_ff=512, vocab=1000, act="swiglu",
                       dtype="bf16", weight_seed=22),
}
_M = {}


def say(*a):
    print(*a, flush=True)


def model(name):
    if name not in _M:
        m = make_model(MODELS[name])
        _M[name] = (m, DeviceModel(m))
    return _M[name]


def tables(n, seed, max_len=200, empty_every=0, vocab=1000):
    r = np.random.default_rng(seed)
    lens = r.integers(1, max_len + 1, size=n).astype(np.int32)
    if empty_every:
        lens[::empty_every] = 0
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    probe = {"id": np.arange(n, dtype=np.int32), "c": r.integers(0, 1000, n).astype(np.int32), "len": lens,
             "offsets": off, "tokens": r.integers(3, vocab, int(off[-1])).astype(np.int32)}
    prefix = r.integers(3, vocab, 64).astype(np.int32)
    return {"probe": probe, "build": None, "prefix": prefix}


def query(npre):
    return Query(preds=(Pred("c", "lt", 700),), labels=(1, 2), decision="binary_gt", agg="count", n_prefix=npre)


def run(t, m, dm, q, share, chunk_tokens=0):
    dq = DeviceQuery(t, m, q, dmodel=dm, share_prefix=share, chunk_tokens=chunk_tokens)
    dq.run()
    torch.cuda.synchronize()
    r = dq.results()
    dq.close()
    return r


def same_result(a, b):
    assert a["status"] == 0 and b["status"] == 0, (hex(a["status"]), hex(b["status"]))
    np.testing.assert_array_equal(a["sel_ids"], b["sel_ids"])
    assert a["n_tokens"] == b["n_tokens"]
    np.testing.assert_array_equal(a["logits"], b["logits"])
    np.testing.assert_array_equal(a["labels"], b["labels"])
    np.testing.assert_array_equal(a["kept_ids"], b["kept_ids"])
    assert a["count"] == b["count"]


@pytest.mark.parametrize("mname", ["hd64", "hd128"])
@pytest.mark.parametrize("npre", [1, 31, 32, 33, 64])
def test_shared_prefix_bitwise_equals_per_row(mname, npre):
    say(f"case: shared vs per-row prefix, model {mname}, prefix {npre}")
    m, dm = model(mname)
    t = tables(900, 100 + npre)
    q = query(npre)
    shared = run(t, m, dm, q, True)
    per_row = run(t, m, dm, q, False)
    say(f"  selected {shared['n_selected']} tokens {shared['n_tokens']}")
    rows, _ = relational(t, q)
    assert shared["n_tokens"] == int(t["probe"]["len"][rows].sum()) + npre * len(rows)
    same_result(shared, per_row)


@pytest.mark.parametrize("mname", ["hd64", "hd128"])
def test_shared_prefix_vs_oracle(mname):
    say(f"case: shared prefix vs oracle, model {mname}")
    m, dm = model(mname)
    t = tables(2000, 7)
    q = query(32)
    r = run(t, m, dm, q, True)
    rows, _ = relational(t, q)
    np.testing.assert_array_equal(r["sel_ids"], rows)
    lens = t["probe"]["len"][rows]
    rng = np.random.default_rng(3)
    sample = np.unique(np.concatenate([rng.integers(0, len(rows), 24), [int(np.argmin(lens)), int(np.argmax(lens))]]))
    seqs = oracle.sequences(t["probe"], rows[sample], t["prefix"][:32])
    lg = oracle.label_logits(m, seqs, q.labels)
    labels = r["labels"].copy()
    labels[sample] = check_labels(r["logits"][sample], r["labels"][sample], lg, decide(lg, q), margin(lg, q),
                                  TOL_BF16, "sample")
    agg = aggregate(t, rows, None, labels, q)
    np.testing.assert_array_equal(r["kept_ids"], agg["kept_ids"])
    assert r["count"] == agg["count"]


def test_shared_prefix_rows_without_tokens():
    """A row with an empty list is the prefix alone: classified from the
    prefix's last token in both modes, and by the oracle."""
    say("case: shared prefix, rows with empty lists")
    m, dm = model("hd64")
    t = tables(600, 11, empty_every=7)
    q = query(32)
    shared = run(t, m, dm, q, True)
    per_row = run(t, m, dm, q, False)
    same_result(shared, per_row)
    rows, _ = relational(t, q)
    lens = t["probe"]["len"][rows]
    empty = np.flatnonzero(lens == 0)
    assert len(empty) > 0
    sample = np.concatenate([empty[:4], np.flatnonzero(lens > 0)[:4]])
    seqs = oracle.sequences(t["probe"], rows[sample], t["prefix"][:32])
    lg = oracle.label_logits(m, seqs, q.labels)
    check_labels(shared["logits"][sample], shared["labels"][sample], lg, decide(lg, q), margin(lg, q), TOL_BF16,
                 "empty rows")
    # every empty row carries the same logits: those of the prefix alone
    e = shared["logits"][empty]
    assert np.all(e == e[0])


def test_shared_prefix_chunking_does_not_change_results():
    say("case: shared prefix, several chunks vs one")
    m, dm = model("hd64")
    t = tables(1500, 13)
    q = query(32)
    one = run(t, m, dm, q, True)
    many = run(t, m, dm, q, True, chunk_tokens=4096)
    same_result(one, many)
