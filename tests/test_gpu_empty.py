"""Degenerate inputs through the whole device pipeline: a table with no rows
(bf16 model with the last layer on the last positions, fp32 model; binary,
argmax + GROUP BY, relational-only plans) and a selection that keeps
nothing.  Everything is launched (counts come from device memory) and every
count, token total, status and group list comes back empty."""
import numpy as np
import pytest
import torch

from paper_2608_10139_amd.device import DeviceModel, DeviceQuery
from synth.configs import ModelSpec, Pred, Query
from synth.gen import make_model

pytestmark = pytest.mark.gpu

MODELS = {
    "bf16": ModelSpec(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, d_ff=512, vocab=1000, act="swiglu",
                      dtype="bf16", weight_seed=41),
    "fp32": ModelSpec(n_layers=1, d_model=64, n_heads=2, n_kv_heads=2, d_ff=64, vocab=1000, act="gelu",
                      dtype="f32", weight_seed=42),
}
_M = {}


def say(*a):
    print(*a, flush=True)


def model(name):
    if name not in _M:
        m = make_model(MODELS[name])
        _M[name] = (m, DeviceModel(m))
    return _M[name]


def table(n, seed=0):
    r = np.random.default_rng(seed)
    lens = r.integers(1, 30, size=n).astype(np.int32)
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    return {"id": np.arange(n, dtype=np.int32), "c": r.integers(0, 1000, n).astype(np.int32),
            "g": r.integers(0, 16, n).astype(np.int32), "len": lens, "offsets": off,
            "tokens": r.integers(3, 1000, int(off[-1])).astype(np.int32)}


def run(t, m, dm, q, **kw):
    dq = DeviceQuery(t, m, q, dmodel=dm, **kw)
    dq.run()
    torch.cuda.synchronize()
    r = dq.results()
    dq.close()
    return r


def nothing(r):
    assert r["status"] == 0
    assert r["n_selected"] == 0 and r["count"] == 0 and r["n_tokens"] == 0
    assert len(r["kept_ids"]) == 0 and len(r["sel_ids"]) == 0


QUERIES = {
    "binary": Query(preds=(Pred("c", "lt", 500),), labels=(1, 2), decision="binary_gt", agg="count"),
    "argmax_group_by": Query(preds=(Pred("c", "lt", 500),), labels=(1, 2, 3), decision="argmax",
                             agg="avg_label_count_by", group_col="g", n_group_keys=16),
}


@pytest.mark.parametrize("mname", list(MODELS))
@pytest.mark.parametrize("qname", list(QUERIES))
def test_table_without_rows(mname, qname):
    say(f"case: table with no rows, model {mname}, query {qname}")
    m, dm = model(mname)
    t = {"probe": table(0), "build": None, "prefix": np.zeros(0, np.int32)}
    r = run(t, m, dm, QUERIES[qname])
    nothing(r)
    if qname == "argmax_group_by":
        assert len(r["groups"][0]) == 0
    nothing(run(t, m, dm, QUERIES["binary"], relational_only=True))


@pytest.mark.parametrize("mname", list(MODELS))
def test_selection_keeps_nothing_on_a_large_table(mname):
    """40,000 rows (five blocks of the compaction), none selected."""
    say(f"case: nothing selected, model {mname}")
    m, dm = model(mname)
    t = {"probe": table(40000, 3), "build": None, "prefix": np.zeros(0, np.int32)}
    q = Query(preds=(Pred("c", "gt", 5000),), labels=(1, 2, 3), decision="argmax", agg="avg_label_count_by",
              group_col="g", n_group_keys=16)
    r = run(t, m, dm, q)
    nothing(r)
    assert len(r["groups"][0]) == 0


def _trailing_empty_table(n_full, n_empty, seed):
    """n_full rows with tokens, then n_empty rows whose lists are empty, all
    selected by c >= 0."""
    r = np.random.default_rng(seed)
    lens = np.concatenate([r.integers(1, 40, n_full), np.zeros(n_empty, np.int64)]).astype(np.int32)
    off = np.zeros(len(lens) + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    n = len(lens)
    probe = {"id": np.arange(n, dtype=np.int32), "c": r.integers(0, 1000, n).astype(np.int32), "len": lens,
             "offsets": off, "tokens": r.integers(3, 1000, int(off[-1])).astype(np.int32)}
    return {"probe": probe, "build": None, "prefix": r.integers(3, 1000, 64).astype(np.int32)}


@pytest.mark.parametrize("npre", [0, 8])
@pytest.mark.parametrize("chunk_tokens", [0, 256])
def test_trailing_empty_rows_are_classified(npre, chunk_tokens):
    """Rows with empty lists after the last token (every row selected) belong
    to a chunk: with chunks of 256 units there are more empty rows (700) than
    one chunk's tokens, and with the default chunk the whole batch is one
    chunk whose token count equals the table's.  Each empty row's logits are
    the oracle's: the prompt prefix alone, or all zero without a prefix (the
    binary decision then rejects it)."""
    import oracle
    from oracle.query import decide, margin
    from tests._parity import TOL_BF16, check_labels
    say(f"case: trailing empty rows, prefix {npre}, chunk_tokens {chunk_tokens}")
    m, dm = model("bf16")
    t = _trailing_empty_table(300, 700, 5 + npre)
    q = Query(preds=(Pred("c", "ge", 0),), labels=(1, 2), decision="binary_gt", agg="count", n_prefix=npre)
    r = run(t, m, dm, q, chunk_tokens=chunk_tokens)
    assert r["status"] == 0, hex(r["status"])
    n = len(t["probe"]["id"])
    assert r["n_selected"] == n
    assert r["n_tokens"] == int(t["probe"]["len"].sum()) + npre * n
    rows = np.arange(n)
    sample = np.concatenate([np.arange(0, 300, 37), [299, 300, 301, 650, 998, 999]])
    seqs = oracle.sequences(t["probe"], rows[sample], t["prefix"][:npre])
    lg = oracle.label_logits(m, seqs, q.labels)
    check_labels(r["logits"][sample], r["labels"][sample], lg, decide(lg, q), margin(lg, q), TOL_BF16,
                 "trailing empty rows")
    empty = r["logits"][300:]
    assert np.all(empty == empty[0]), "every empty row carries the same logits"
    if npre == 0:
        assert np.all(empty == 0.0) and np.all(r["labels"][300:] == 0)
    one = run(t, m, dm, q)   # one chunk: bit-identical
    np.testing.assert_array_equal(r["logits"], one["logits"])
    np.testing.assert_array_equal(r["kept_ids"], one["kept_ids"])
