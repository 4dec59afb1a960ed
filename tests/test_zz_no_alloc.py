"""The entry point that allocates nothing (aiq_run_relational_static): its
outputs must equal aiq_run's with a caller workspace for the same
relational-only plan, exactly, on two calls in a row of which the second has
a smaller input (the scratch keeps the first call's contents), with and
without a join, and both equal the oracle's selection."""
import numpy as np
import pytest
import torch

from oracle.query import relational
from paper_2608_10139_amd.device import DeviceModel, DeviceQuery
from synth.configs import Join, ModelSpec, Pred, Query
from synth.gen import make_model

pytestmark = pytest.mark.gpu

REL = ModelSpec(n_layers=1, d_model=64, n_heads=2, n_kv_heads=2, d_ff=64, vocab=500, act="gelu",
                dtype="f32", weight_seed=5, init_std=0.1)


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def rel_model():
    m = make_model(REL)
    return m, DeviceModel(m)


def table(n, seed, max_len=40):
    r = np.random.default_rng(seed)
    lens = r.integers(0, max_len + 1, size=n).astype(np.int32)
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    pool = np.concatenate([np.arange(100, 900, 7, dtype=np.int32), np.array([-5, np.iinfo(np.int32).min], np.int32)])
    return {"id": np.arange(n, dtype=np.int32), "c": r.integers(0, 1000, n).astype(np.int32),
            "movie_id": pool[r.integers(0, len(pool), n)], "len": lens, "offsets": off,
            "tokens": r.integers(0, 500, int(off[-1])).astype(np.int32)}


def movies():
    ids = np.arange(100, 900, 7, dtype=np.int32)
    r = np.random.default_rng(9)
    return {"movie_id": ids, "genre": r.integers(0, 20, len(ids)).astype(np.int8),
            "year": r.integers(1950, 2026, len(ids)).astype(np.int16)}


def both(t, m, dm, q):
    """(aiq_run with a workspace, aiq_run_relational_static) results."""
    ws = DeviceQuery(t, m, q, dmodel=dm, relational_only=True)
    st = DeviceQuery(t, m, q, dmodel=dm, relational_only=True)
    ws.run()
    st.run_static()
    torch.cuda.synchronize()
    a, b = ws.results(), st.results()
    ws.close()
    st.close()
    return a, b


def same(a, b, t, q):
    assert a["status"] == 0 and b["status"] == 0, (hex(a["status"]), hex(b["status"]))
    np.testing.assert_array_equal(a["scalars"], b["scalars"])
    np.testing.assert_array_equal(a["kept_ids"], b["kept_ids"])
    np.testing.assert_array_equal(a["sel_ids"], b["sel_ids"])
    rows, _ = relational(t, q)
    np.testing.assert_array_equal(b["sel_ids"], rows)
    assert b["n_tokens"] == int(np.diff(t["probe"]["offsets"])[rows].sum()) + q.n_prefix * len(rows)


@pytest.mark.parametrize("join", [False, True])
def test_static_scratch_equals_workspace_run(rel_model, join):
    m, dm = rel_model
    for n, seed in ((70000, 1), (3000, 2)):   # the second call has the smaller input
        say(f"case: static scratch vs workspace, join {join}, {n} rows")
        t = {"probe": table(n, seed), "build": movies() if join else None, "prefix": np.array([5, 6, 7], np.int32)}
        if join:
            q = Query(preds=(Pred("c", "lt", 600),), labels=(1, 2), decision="binary_gt", agg="count", n_prefix=3,
                      join=Join("movie_id", "movie_id", "genre", (Pred("year", "gt", 1990),)))
        else:
            q = Query(preds=(Pred("c", "lt", 300 if n > 5000 else 900),), labels=(1, 2), decision="binary_gt",
                      agg="count")
        a, b = both(t, m, dm, q)
        say(f"  selected {b['n_selected']} tokens {b['n_tokens']}")
        same(a, b, t, q)
