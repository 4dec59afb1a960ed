"""Full-size workloads through the C ABI, in the launch configuration the
benchmark uses (default chunking):

* 1B-class 5-way classify + GROUP BY (131,072 rows), reviews JOIN movies with
  a shared 32-token prefix (262,144 reviews), and the 3B-class selectivity
  sweep at 1 % (1,048,576 rows): selected rows, token counts, kept ids and
  groups exact; label logits of a seeded sample of rows (shortest and longest
  included) within the bf16 tolerance of the oracle; every aggregate recomputed
  by the oracle from the device's per-row labels and compared exactly.
* All four thresholds of the sweep table with a one-layer fp32 model: the
  relational result (selection, tokens) exact at every selectivity, sampled
  labels against the oracle, the COUNT and kept ids exact given the labels.
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


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["groupby1b", "join1b", "sweep3b"])
def test_full_size_workload(name):
    g = load_golden(name)
    if g is None:
        pytest.skip(f"golden file for {name} not generated")
    w = WORKLOADS[name]
    q = w.queries[0]
    say(f"case: {name} full size ({w.description}); generating inputs")
    t = tables(name)
    model = make_model(w.model)
    dm = DeviceModel(model)
    say("  running on the device")
    r = run(t, model, q, dm)
    say(f"  selected {r['n_selected']} tokens {r['n_tokens']} kept {r['count']} status {r['status']:#x}")
    rows = g["q0_rows"]
    payload = g.get("q0_payload")
    check_query(r, t, q, rows, payload, g["q0_logits"], g["q0_labels"], g["q0_margin"], TOL_BF16,
                sample=g["q0_sample"])
    del dm


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
