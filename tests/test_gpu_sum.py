"""The paper's running query shape on the device: a filter on an fp32 column
and the SUM of that column over the rows the semantic filter keeps (Table 1
SUM row, Figure 2).  Selections must equal the oracle's exactly; labels
agree outside the tie band; the SUM is compared with the oracle's exactly
rounded sum over the device's kept rows, within the bound stated in the C
header (2^-52 (n + 64) sum|v|), and must be bit-identical between runs."""
import numpy as np
import pytest
import torch

import oracle
from oracle.query import aggregate, decide, margin, relational
from paper_2608_10139_amd.device import DeviceModel, DeviceQuery
from synth import WORKLOADS
from synth.configs import ModelSpec, Pred, Query
from synth.gen import make_model, make_tables
from tests._parity import TOL_BF16, TOL_F32, check_labels

pytestmark = pytest.mark.gpu

REL = ModelSpec(n_layers=1, d_model=64, n_heads=2, n_kv_heads=2, d_ff=64, vocab=500, act="gelu",
                dtype="f32", weight_seed=5, init_std=0.1)


def say(*a):
    print(*a, flush=True)


def run(tables, model, dm, q):
    dq = DeviceQuery(tables, model, q, dmodel=dm)
    dq.run()
    torch.cuda.synchronize()
    r1 = dq.results()
    dq.run()
    torch.cuda.synchronize()
    r2 = dq.results()
    dq.close()
    return r1, r2


def check_sum(r1, r2, tables, q, rows, labels_dev):
    agg = aggregate(tables, rows, None, labels_dev, q)
    np.testing.assert_array_equal(r1["kept_ids"], agg["kept_ids"])
    assert r1["count"] == agg["count"]
    v = tables["probe"][q.group_col][agg["kept_ids"]].astype(np.float64)
    if np.isfinite(agg["sum"]):
        bound = 2.0 ** -52 * (len(v) + 64) * float(np.abs(v).sum())
        assert abs(r1["sum"] - agg["sum"]) <= bound, (r1["sum"], agg["sum"], bound)
    else:   # an infinity or NaN was kept: the IEEE result
        assert (np.isnan(agg["sum"]) and np.isnan(r1["sum"])) or agg["sum"] == r1["sum"], (r1["sum"], agg["sum"])
    assert np.float64(r1["sum"]).tobytes() == np.float64(r2["sum"]).tobytes()   # same bits every run


def test_tiny_sum_query():
    say("case: tiny_sum (full oracle)")
    w = WORKLOADS["tiny_sum"]
    t = make_tables(w)
    q = w.queries[0]
    m = make_model(w.model)
    dm = DeviceModel(m)
    rows, _ = relational(t, q)
    seqs = oracle.sequences(t["probe"], rows, t["prefix"][:0])
    lg = oracle.label_logits(m, seqs, q.labels)
    r1, r2 = run(t, m, dm, q)
    assert r1["status"] == 0
    np.testing.assert_array_equal(r1["sel_ids"], rows)
    labels = check_labels(r1["logits"], r1["labels"], lg, decide(lg, q), margin(lg, q), TOL_F32)
    check_sum(r1, r2, t, q, rows, labels)


def test_reviews_sum_query():
    say("case: reviews_sum (16,384 rows; sampled logits)")
    w = WORKLOADS["reviews_sum"]
    t = make_tables(w)
    q = w.queries[0]
    m = make_model(w.model)
    dm = DeviceModel(m)
    rows, _ = relational(t, q)
    r1, r2 = run(t, m, dm, q)
    assert r1["status"] == 0
    np.testing.assert_array_equal(r1["sel_ids"], rows)
    rng = np.random.default_rng(0)
    lens = t["probe"]["len"][rows]
    sample = np.unique(np.concatenate([rng.integers(0, len(rows), 24), [np.argmin(lens), np.argmax(lens)]]))
    seqs = oracle.sequences(t["probe"], rows[sample], t["prefix"][:0])
    lg = oracle.label_logits(m, seqs, q.labels)
    check_labels(r1["logits"][sample], r1["labels"][sample], lg, decide(lg, q), margin(lg, q), TOL_BF16)
    check_sum(r1, r2, t, q, rows, r1["labels"])


@pytest.fixture(scope="module")
def rel_model():
    m = make_model(REL)
    return m, DeviceModel(m)


def float_table(n, seed):
    r = np.random.default_rng(seed)
    lens = r.integers(1, 9, size=n).astype(np.int32)
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    v = (r.random(n) * 200 - 50).astype(np.float32)
    # edge values: the thresholds, their fp32 neighbours, signed zeros, NaN, infinities
    edges = np.float32([70.0, np.nextafter(np.float32(70), np.float32(100)), np.nextafter(np.float32(70), np.float32(0)),
                        0.0, -0.0, np.nan, np.inf, -np.inf, 12.5, -3.25])
    v[r.choice(n, size=min(n, 400), replace=False)] = np.resize(edges, min(n, 400))
    return {"id": np.arange(n, dtype=np.int32), "v": v, "a": r.integers(-100, 100, n).astype(np.int8),
            "len": lens, "offsets": off, "tokens": r.integers(0, 500, int(off[-1])).astype(np.int32)}


@pytest.mark.parametrize("op,k", [("gt", 70.0), ("ge", 70.0), ("lt", 0.0), ("le", -0.0), ("eq", 12.5), ("ne", 70.0)])
def test_float_predicates_exact(rel_model, op, k):
    say(f"case: float predicate {op} {k}")
    m, dm = rel_model
    t = {"probe": float_table(70001, 9), "build": None, "prefix": np.zeros(0, np.int32)}
    q = Query(preds=(Pred("v", op, k), Pred("a", "ne", 3)), labels=(1, 2), decision="binary_gt", agg="sum_f32",
              group_col="v")
    rows, _ = relational(t, q)
    r1, r2 = run(t, m, dm, q)
    assert r1["status"] == 0
    np.testing.assert_array_equal(r1["sel_ids"], rows)
    check_sum(r1, r2, t, q, rows, r1["labels"])
