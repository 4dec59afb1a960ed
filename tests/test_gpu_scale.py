"""Full-size workloads through the C ABI, in the launch configuration the
benchmark uses (default chunking):

* 1B-class 5-way classify + GROUP BY (131,072 rows), reviews JOIN movies with
  a shared 32-token prefix (262,144 reviews), and the 3B-class selectivity
  sweep at 1 % and 10 % (1,048,576 rows): selected rows, token counts, kept ids
  and groups exact; label logits of a sample of at least 128 selected rows
  (shortest and longest included, every decision outcome present) within the
  bf16 tolerance of the oracle; every aggregate recomputed by the oracle from
  the device's per-row labels and compared exactly.
* The sweep's 50 % and 100 % thresholds with the 3B-class model on the
  table's first 8,192 rows, to the same bar.
* All four thresholds on the whole sweep table with a one-layer fp32 model:
  the relational result (selection, tokens) exact at every selectivity,
  sampled labels against the oracle, the COUNT and kept ids exact given the
  labels.

A missing golden file fails the test (tests/golden/make_golden.py writes them).
"""
import numpy as np
import pytest
import torch

import oracle
from oracle.query import aggregate, decide, margin, relational
from paper_2608_10139_amd.device import DeviceModel, DeviceQuery
from synth import WORKLOADS
from synth.configs import ModelSpec
from synth.gen import make_model, make_tables
from tests._parity import TOL_BF16, TOL_F32, check_labels, check_query, load_golden

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


_T = {}


def tables(name):
    if name not in _T:
        _T[name] = make_tables(WORKLOADS[name])
    return _T[name]


def run(t, model, q, dm):
    dq = DeviceQuery(t, model, q, dmodel=dm)
    dq.run()
    torch.cuda.synchronize()
    r = dq.results()
    dq.close()
    return r


def golden(name):
    g = load_golden(name)
    assert g is not None, f"golden file for {name} missing: run python -m tests.golden.make_golden {name}"
    return g


def outcomes(q):
    return {0, 1} if q.decision == "binary_gt" else set(int(l) for l in q.labels)


_MODELS = {}


def device_model(w):
    key = w.model
    if key not in _MODELS:
        _MODELS.clear()   # one large model resident at a time
        m = make_model(w.model)
        _MODELS[key] = (m, DeviceModel(m))
    return _MODELS[key]


def check_against_golden(gname, t, w, qi):
    g = golden(gname)
    q = w.queries[qi]
    model, dm = device_model(w)
    say("  running on the device")
    r = run(t, model, q, dm)
    say(f"  selected {r['n_selected']} tokens {r['n_tokens']} kept {r['count']} status {r['status']:#x}")
    p = f"q{qi}_"
    sample = g[p + "sample"]
    assert len(sample) >= min(128, len(g[p + "rows"])), "golden sample smaller than 128 rows"
    assert outcomes(q) <= set(g[p + "labels"].tolist()), "golden sample misses a decision outcome"
    check_query(r, t, q, g[p + "rows"], g.get(p + "payload"), g[p + "logits"], g[p + "labels"], g[p + "margin"],
                TOL_BF16, sample=sample)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name,qi", [("groupby1b", 0), ("join1b", 0), ("sweep3b", 0), ("sweep3b", 1)])
def test_full_size_workload(name, qi):
    w = WORKLOADS[name]
    say(f"case: {name} query {qi} full size ({w.description}); generating inputs")
    check_against_golden(name, tables(name), w, qi)


def head_tables(n):
    """The first n rows of the sweep table (token lists included)."""
    t = tables("sweep3b")
    p = t["probe"]
    off = p["offsets"][: n + 1]
    probe = {k: v[:n] for k, v in p.items() if k not in ("offsets", "tokens")}
    probe["offsets"] = off
    probe["tokens"] = p["tokens"][: int(off[-1])]
    return {"probe": probe, "build": None, "prefix": t["prefix"]}


@pytest.mark.timeout(600)
@pytest.mark.parametrize("qi", [2, 3])
def test_sweep_3b_model_high_selectivity(qi):
    w = WORKLOADS["sweep3b"]
    say(f"case: sweep table first 8,192 rows, c < {w.queries[qi].preds[0].k}, 3B-class model")
    check_against_golden("sweep3b_head", head_tables(8192), w, qi)


@pytest.fixture(scope="module")
def small32k():
    spec = ModelSpec(n_layers=1, d_model=64, n_heads=2, n_kv_heads=2, d_ff=64, vocab=32000, act="gelu",
                     dtype="f32", weight_seed=6, init_std=0.1)
    m = make_model(spec)
    return m, DeviceModel(m)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("qi", [0, 1, 2, 3])
def test_sweep_relational_every_threshold(small32k, qi):
    m, dm = small32k
    w = WORKLOADS["sweep3b"]
    q = w.queries[qi]
    say(f"case: sweep table, threshold c < {q.preds[0].k}, one-layer fp32 model")
    t = tables("sweep3b")
    rows, _ = relational(t, q)
    r = run(t, m, q, dm)
    say(f"  selected {r['n_selected']} tokens {r['n_tokens']} kept {r['count']}")
    assert r["status"] == 0
    np.testing.assert_array_equal(r["sel_ids"], rows)
    assert r["n_tokens"] == int(t["probe"]["len"][rows].sum())
    rng = np.random.default_rng(qi)
    sample = np.unique(np.concatenate([rng.integers(0, len(rows), 40),
                                       [0, len(rows) - 1, int(np.argmax(t["probe"]["len"][rows]))]]))
    seqs = oracle.sequences(t["probe"], rows[sample], t["prefix"][:0])
    lg = oracle.label_logits(m, seqs, q.labels)
    check_labels(r["logits"][sample], r["labels"][sample], lg, decide(lg, q), margin(lg, q), TOL_F32)
    agg = aggregate(t, rows, None, r["labels"], q)
    np.testing.assert_array_equal(r["kept_ids"], agg["kept_ids"])
    assert r["count"] == agg["count"]
