"""The last layer for the last positions only (the label head reads one row
per sequence; in a causal decoder the last layer's rows after its q|k|v
projection feed no other position).  Pinned against:
* the full last layer on the device (AIQ_PLAN_FULL_LAST_LAYER): the same
  selection, logits within the bf16 tolerance, labels equal outside the tie
  band; for MHA and GQA (2, 3 and 4 query heads per key/value head), head
  dims 64 and 128;
* the oracle (fp64, per sequence) on a sample with the shortest and longest
  rows;
* itself across chunkings and across more sequences than one block of last
  positions holds (262,144): bit-identical, since every sequence's last
  position is computed alone;
* the prefill-only entry point, labels and full-vocabulary logits.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle.query import aggregate, decide, margin, relational
from paper_2608_10139_amd.device import DeviceModel, DevicePrefill, DeviceQuery
from synth.configs import ModelSpec, Pred, Query
from synth.gen import make_model
from tests._parity import TOL_BF16, check_labels

pytestmark = pytest.mark.gpu

MODELS = {
    "mha64": ModelSpec(n_layers=3, d_model=256, n_heads=4, n_kv_heads=4, d_ff=512, vocab=1000, act="swiglu",
                       dtype="bf16", weight_seed=31),
    "gqa64_rep4": ModelSpec(n_layers=2, d_model=512, n_heads=8, n_kv_heads=2, d_ff=512, vocab=1024, act="swiglu",
                            dtype="bf16", weight_seed=32),
    "gqa128_rep3": ModelSpec(n_layers=2, d_model=768, n_heads=6, n_kv_heads=2, d_ff=512, vocab=1000,
                             act="swiglu", dtype="bf16", weight_seed=33),
    "gqa128_rep2": ModelSpec(n_layers=2, d_model=512, n_heads=4, n_kv_heads=2, d_ff=512, vocab=1000,
                             act="swiglu", dtype="bf16", weight_seed=34),
}
_M = {}


def say(*a):
    print(*a, flush=True)


def model(name):
    if name not in _M:
        m = make_model(MODELS[name])
        _M[name] = (m, DeviceModel(m))
    return _M[name]


def tables(n, seed, max_len=200, min_len=1, vocab=1000, prefix=0):
    r = np.random.default_rng(seed)
    lens = r.integers(min_len, max_len + 1, size=n).astype(np.int32)
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    probe = {"id": np.arange(n, dtype=np.int32), "c": r.integers(0, 1000, n).astype(np.int32), "len": lens,
             "offsets": off, "tokens": r.integers(3, vocab, int(off[-1])).astype(np.int32)}
    return {"probe": probe, "build": None, "prefix": r.integers(3, vocab, max(prefix, 1)).astype(np.int32)}


def run(t, m, dm, q, **kw):
    dq = DeviceQuery(t, m, q, dmodel=dm, **kw)
    dq.run()
    torch.cuda.synchronize()
    r = dq.results()
    dq.close()
    return r


def close_to_full(last, full, what):
    """Same selection; logits within the bf16 tolerance; labels equal where
    the full computation's margin is outside it."""
    assert last["status"] == 0 and full["status"] == 0
    np.testing.assert_array_equal(last["sel_ids"], full["sel_ids"])
    assert last["n_tokens"] == full["n_tokens"]
    diff = float(np.max(np.abs(last["logits"] - full["logits"]))) if len(full["logits"]) else 0.0
    say(f"  {what}: {len(full['sel_ids'])} sequences, max |logit difference| {diff:.2e}")
    assert diff <= TOL_BF16
    lg = full["logits"]
    marg = np.abs(lg[:, 0] - lg[:, 1]) if lg.shape[1] == 2 else np.sort(lg, 1)[:, -1] - np.sort(lg, 1)[:, -2]
    firm = marg > TOL_BF16
    np.testing.assert_array_equal(last["labels"][firm], full["labels"][firm])


@pytest.mark.parametrize("mname", list(MODELS))
def test_last_rows_vs_full_last_layer(mname):
    say(f"case: last layer on last positions vs full, model {mname}")
    m, dm = model(mname)
    t = tables(2500, 5)
    q = Query(preds=(Pred("c", "lt", 700),), labels=(1, 2), decision="binary_gt", agg="count")
    close_to_full(run(t, m, dm, q), run(t, m, dm, q, full_last_layer=True), mname)


@pytest.mark.parametrize("mname", ["mha64", "gqa128_rep3"])
def test_last_rows_vs_oracle(mname):
    say(f"case: last layer on last positions vs oracle, model {mname}")
    m, dm = model(mname)
    t = tables(1500, 9)
    q = Query(preds=(Pred("c", "lt", 500),), labels=(1, 2, 3), decision="argmax", agg="count")
    r = run(t, m, dm, q)
    rows, _ = relational(t, q)
    np.testing.assert_array_equal(r["sel_ids"], rows)
    lens = t["probe"]["len"][rows]
    rng = np.random.default_rng(4)
    sample = np.unique(np.concatenate([rng.integers(0, len(rows), 20), [int(np.argmin(lens)), int(np.argmax(lens))]]))
    seqs = oracle.sequences(t["probe"], rows[sample], t["prefix"][:0])
    lg = oracle.label_logits(m, seqs, q.labels)
    labels = r["labels"].copy()
    labels[sample] = check_labels(r["logits"][sample], r["labels"][sample], lg, decide(lg, q), margin(lg, q),
                                  TOL_BF16, "sample")
    agg = aggregate(t, rows, None, labels, q)
    np.testing.assert_array_equal(r["kept_ids"], agg["kept_ids"])
    assert r["count"] == agg["count"]


def test_last_rows_chunking_bit_identical():
    """70,000 selected sequences of 1..4 tokens: one block of last positions
    in one chunk, and one per chunk over several chunks, give the same bits;
    the result stays within tolerance of the full last layer."""
    say("case: last positions over one and several chunks")
    m, dm = model("mha64")
    t = tables(72000, 13, max_len=4)
    q = Query(preds=(Pred("c", "lt", 980),), labels=(1, 2), decision="binary_gt", agg="count")
    one = run(t, m, dm, q)
    assert one["n_selected"] > 65536
    chunked = run(t, m, dm, q, chunk_tokens=40000)
    for k in ("sel_ids", "labels", "kept_ids"):
        np.testing.assert_array_equal(one[k], chunked[k])
    np.testing.assert_array_equal(one["logits"].view(np.int32), chunked["logits"].view(np.int32))
    close_to_full(one, run(t, m, dm, q, full_last_layer=True), "one block")


def test_last_rows_two_blocks_bit_identical():
    """300,000 selected sequences of 1..2 tokens: two blocks of last
    positions (262,144 per block) in one chunk give the same bits as one
    block per chunk over several chunks."""
    say("case: last positions over two blocks")
    m, dm = model("mha64")
    t = tables(306000, 19, max_len=2)
    q = Query(preds=(Pred("c", "lt", 980),), labels=(1, 2), decision="binary_gt", agg="count")
    one = run(t, m, dm, q)
    assert one["status"] == 0 and one["n_selected"] > 262144
    chunked = run(t, m, dm, q, chunk_tokens=200000)
    for k in ("sel_ids", "labels", "kept_ids"):
        np.testing.assert_array_equal(one[k], chunked[k])
    np.testing.assert_array_equal(one["logits"].view(np.int32), chunked["logits"].view(np.int32))


def test_last_rows_prefill_entry_point():
    """aiq_prefill_packed: label logits and full-vocabulary last-position
    logits within tolerance of the full last layer."""
    say("case: prefill-only entry point, last positions vs full")
    m, dm = model("gqa64_rep4")
    r = np.random.default_rng(17)
    lens = r.integers(1, 300, size=700)
    cu = np.zeros(len(lens) + 1, np.int32)
    cu[1:] = np.cumsum(lens)
    tok = torch.tensor(r.integers(3, 1000, int(cu[-1])).astype(np.int32), device="cuda")
    cu_t = torch.tensor(cu, device="cuda")
    out = {}
    for full in (False, True):
        pf = DevicePrefill(m, labels=(1, 2), max_tokens=int(cu[-1]), dmodel=dm, full_last_layer=full)
        out[full] = (pf.run(tok, cu_t).cpu().numpy(), pf.run(tok, cu_t, full_vocab=True).cpu().numpy())
        torch.cuda.synchronize()
    for a, b, what in ((out[False][0], out[True][0], "labels"), (out[False][1], out[True][1], "full vocabulary")):
        d = float(np.max(np.abs(a - b)))
        say(f"  {what}: max |logit difference| {d:.2e}")
        assert d <= TOL_BF16
