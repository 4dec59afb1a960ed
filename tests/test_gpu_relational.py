"""Relational steps on the device vs the oracle, exact: ragged table sizes,
every predicate operator, empty results, the PK-FK join, GROUP BY, and the
device status bits.  A one-layer fp32 model keeps the semantic step cheap."""
import numpy as np
import pytest
import torch

import oracle
from oracle.query import aggregate, decide, margin, relational
from paper_2608_10139_amd import binding as B
from paper_2608_10139_amd.device import DeviceModel, DeviceQuery
from synth.configs import Join, ModelSpec, Pred, Query
from synth.gen import make_model
from tests._parity import TOL_F32, check_query

pytestmark = pytest.mark.gpu

REL = ModelSpec(n_layers=1, d_model=64, n_heads=2, n_kv_heads=2, d_ff=64, vocab=500, act="gelu",
                dtype="f32", weight_seed=5, init_std=0.1)


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def rel_model():
    m = make_model(REL)
    return m, DeviceModel(m)


def table(n, seed, vocab=500, max_len=12):
    r = np.random.default_rng(seed)
    lens = r.integers(1, max_len + 1, size=n).astype(np.int32)
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    return {"id": np.arange(n, dtype=np.int32), "a": r.integers(-128, 128, n).astype(np.int8),
            "b": r.integers(-50, 50, n).astype(np.int16), "c": r.integers(0, 1000, n).astype(np.int32),
            "g": r.integers(0, 50, n).astype(np.int32), "len": lens, "offsets": off,
            "tokens": r.integers(0, vocab, int(off[-1])).astype(np.int32)}


def run(tables, model, dm, q, tweak=None):
    dq = DeviceQuery(tables, model, q, dmodel=dm)
    if tweak:
        tweak(dq)
    dq.run()
    torch.cuda.synchronize()
    r = dq.results()
    dq.close()
    return r


def full_check(tables, model, dm, q):
    rows, payload = relational(tables, q)
    seqs = oracle.sequences(tables["probe"], rows, tables["prefix"][:q.n_prefix])
    lg = oracle.label_logits(model, seqs, q.labels)
    r = run(tables, model, dm, q)
    check_query(r, tables, q, rows, payload, lg, decide(lg, q), margin(lg, q), TOL_F32)
    return r


@pytest.mark.parametrize("n", [1, 63, 64, 65, 2047, 2048, 2049, 5000])
def test_selection_ragged_sizes(rel_model, n):
    say(f"case: selection n={n}")
    m, dm = rel_model
    t = {"probe": table(n, n), "build": None, "prefix": np.zeros(0, np.int32)}
    q = Query(preds=(Pred("a", "ge", -60), Pred("b", "in", values=(-3, 0, 7, 11, 49, -50))), labels=(1, 2),
              decision="binary_gt", agg="count")
    full_check(t, m, dm, q)


@pytest.mark.parametrize("op,k", [("lt", 500), ("le", 0), ("gt", 998), ("ge", 999), ("eq", 17), ("ne", 17)])
def test_each_operator(rel_model, op, k):
    say(f"case: operator {op} {k}")
    m, dm = rel_model
    t = {"probe": table(3000, 7), "build": None, "prefix": np.zeros(0, np.int32)}
    q = Query(preds=(Pred("c", op, k),), labels=(3, 4), decision="binary_gt", agg="count")
    full_check(t, m, dm, q)


def test_no_survivors(rel_model):
    say("case: empty selection")
    m, dm = rel_model
    t = {"probe": table(4000, 3), "build": None, "prefix": np.zeros(0, np.int32)}
    q = Query(preds=(Pred("a", "gt", 127),), labels=(1, 2), decision="binary_gt", agg="count")
    r = run(t, m, dm, q)
    assert r["status"] == 0 and r["n_selected"] == 0 and r["count"] == 0 and r["n_tokens"] == 0


def test_prefix_and_argmax_group_by(rel_model):
    say("case: prefix + argmax + group by")
    m, dm = rel_model
    t = {"probe": table(6000, 11), "build": None, "prefix": np.array([5, 6, 7, 8, 9], np.int32)}
    q = Query(preds=(Pred("b", "lt", 20),), labels=(1, 2, 3, 4), decision="argmax", agg="avg_label_count_by",
              n_prefix=5, group_col="g", n_group_keys=50)
    full_check(t, m, dm, q)


def movies(n, seed):
    r = np.random.default_rng(seed)
    return {"movie_id": r.choice(1_000_000, size=n, replace=False).astype(np.int32),
            "genre": r.integers(0, 20, n).astype(np.int8), "year": r.integers(1950, 2026, n).astype(np.int16)}


def test_join_count_by_payload(rel_model):
    say("case: join + count by genre")
    m, dm = rel_model
    mv = movies(700, 1)
    pr = table(9000, 2)
    r = np.random.default_rng(3)
    # dangling keys too, among them the hash table's empty-slot value (INT32_MIN), which matches no movie
    pool = np.concatenate([mv["movie_id"], np.array([-5, 2_000_000, np.iinfo(np.int32).min], np.int32)])
    pr["movie_id"] = pool[r.integers(0, len(pool), 9000)]
    t = {"probe": pr, "build": mv, "prefix": np.array([11, 12], np.int32)}
    q = Query(preds=(Pred("a", "lt", 100),), labels=(1, 2), decision="binary_gt", agg="count_by_payload",
              n_prefix=2, n_group_keys=20,
              join=Join("movie_id", "movie_id", "genre", (Pred("genre", "in", values=(2, 5, 11)),
                                                          Pred("year", "gt", 2000))))
    full_check(t, m, dm, q)


def test_status_duplicate_build_key(rel_model):
    say("case: duplicate build key flagged")
    m, dm = rel_model
    mv = movies(100, 4)
    mv["movie_id"][10] = mv["movie_id"][20]
    mv["year"][10] = mv["year"][20] = 2010
    pr = table(500, 5)
    pr["movie_id"] = mv["movie_id"][np.random.default_rng(6).integers(0, 100, 500)]
    t = {"probe": pr, "build": mv, "prefix": np.zeros(0, np.int32)}
    q = Query(preds=(), labels=(1, 2), decision="binary_gt", agg="count", n_group_keys=20,
              join=Join("movie_id", "movie_id", "genre", (Pred("year", "gt", 2000),)))
    r = run(t, m, dm, q)
    assert r["status"] & B.AIQ_DEV_DUP_KEY


def test_status_token_range_and_ids_cap(rel_model):
    say("case: token range + ids capacity flagged")
    m, dm = rel_model
    pr = table(3000, 8)
    pr["tokens"][5] = 10_000
    t = {"probe": pr, "build": None, "prefix": np.zeros(0, np.int32)}
    q = Query(preds=(), labels=(1, 2), decision="binary_gt", agg="count")

    def small_cap(dq):
        dq.out.ids_cap = 3
    r = run(t, m, dm, q, tweak=small_cap)
    assert r["status"] & B.AIQ_DEV_TOKEN_RANGE
    assert r["status"] & B.AIQ_DEV_IDS_CAP


def run_relational_only(tables, model, dm, q):
    dq = DeviceQuery(tables, model, q, dmodel=dm, relational_only=True)
    dq.run()
    torch.cuda.synchronize()
    r = dq.results()
    dq.close()
    return r


def check_relational_only(r, tables, q):
    rows, _ = relational(tables, q)
    assert r["status"] == 0
    assert r["n_selected"] == r["count"] == len(rows)
    np.testing.assert_array_equal(r["kept_ids"], rows)
    np.testing.assert_array_equal(r["sel_ids"], rows)
    lens = np.diff(tables["probe"]["offsets"])
    assert r["n_tokens"] == int(lens[rows].sum()) + q.n_prefix * len(rows)


@pytest.mark.parametrize("n", [1, 64, 2049, 70000])
def test_relational_only_mode(rel_model, n):
    """The plan flag that stops after the relational part: every selected id
    kept, counts and token totals exact; the token column is never read."""
    say(f"case: relational-only n={n}")
    m, dm = rel_model
    probe = table(n, 100 + n)
    q = Query(preds=(Pred("c", "lt", 400), Pred("a", "ne", 5)), labels=(1, 2), decision="binary_gt", agg="count")
    t = {"probe": probe, "build": None, "prefix": np.zeros(0, np.int32)}
    check_relational_only(run_relational_only(t, m, dm, q), t, q)
    # without a token column at all
    t2 = {"probe": {k: v for k, v in probe.items() if k != "tokens"}, "build": None,
          "prefix": np.zeros(0, np.int32)}
    check_relational_only(run_relational_only(t2, m, dm, q), t2, q)


def test_relational_only_join_with_prefix(rel_model):
    say("case: relational-only join")
    m, dm = rel_model
    r = np.random.default_rng(11)
    nb = 300
    build = {"key": r.choice(1 << 30, nb, replace=False).astype(np.int32),
             "genre": r.integers(0, 7, nb).astype(np.int8), "year": r.integers(1950, 2020, nb).astype(np.int16)}
    probe = table(4000, 12)
    probe["fk"] = build["key"][r.integers(0, nb, 4000)]
    t = {"probe": probe, "build": build, "prefix": np.arange(3, 8, dtype=np.int32)}
    q = Query(preds=(Pred("a", "gt", -100),), labels=(1, 2), decision="binary_gt", agg="count",
              join=Join(probe_key="fk", build_key="key", payload="genre",
                        build_preds=(Pred("year", "gt", 1990),)), n_prefix=5)
    check_relational_only(run_relational_only(t, m, dm, q), t, q)


# ---- GROUP BY over any int32 key (hash table, groups sorted by key) and the
# join probed from the LDS-staged build table or, when more build rows pass
# than LDS holds, from the global one

def sparse_keys(n, seed):
    """Hot keys (negative, zero, the int32 extremes) mixed with thousands of
    distinct random keys, so a workgroup's private table fills and merges."""
    r = np.random.default_rng(seed)
    hot = np.array([np.iinfo(np.int32).min, -7, -1, 0, 3, 1 << 30, np.iinfo(np.int32).max], np.int64)
    cold = r.integers(np.iinfo(np.int32).min, np.iinfo(np.int32).max, 6000, dtype=np.int64, endpoint=True)
    pick = np.where(r.random(n) < 0.5, hot[r.integers(0, len(hot), n)], cold[r.integers(0, len(cold), n)])
    return pick.astype(np.int32)


@pytest.mark.parametrize("n", [1, 3000, 40000])
def test_hash_group_by_any_int32_key(rel_model, n):
    say(f"case: hash group by over sparse int32 keys, {n} rows")
    m, dm = rel_model
    pr = table(n, 20 + n)
    pr["g"] = sparse_keys(n, n)
    t = {"probe": pr, "build": None, "prefix": np.zeros(0, np.int32)}
    q = Query(preds=(Pred("b", "lt", 40),), labels=(1, 2, 3, 4), decision="argmax", agg="avg_label_count_by",
              group_col="g", n_group_keys=0)
    r = full_check(t, m, dm, q)
    assert len(r["groups"][0]) == len(np.unique(pr["g"][relational(t, q)[0]]))


@pytest.mark.parametrize("col", ["a", "b"])
def test_hash_group_by_narrow_columns(rel_model, col):
    say(f"case: hash group by over the {col} column (negative int8 / int16 keys)")
    m, dm = rel_model
    t = {"probe": table(9000, 31), "build": None, "prefix": np.zeros(0, np.int32)}
    q = Query(preds=(Pred("c", "lt", 700),), labels=(1, 2), decision="binary_gt", agg="avg_label_count_by",
              group_col=col, n_group_keys=0)
    full_check(t, m, dm, q)


@pytest.mark.parametrize("n_movies,payload", [(700, "genre"), (700, "movie_id"), (5000, "movie_id")])
def test_join_hash_groups_and_staging(rel_model, n_movies, payload):
    say(f"case: join with {n_movies} movies, count by {payload} (hash groups)")
    m, dm = rel_model
    mv = movies(n_movies, 40)
    pr = table(12000, 41)
    r = np.random.default_rng(42)
    pool = np.concatenate([mv["movie_id"], np.array([-5, np.iinfo(np.int32).min], np.int32)])
    pr["movie_id"] = pool[r.integers(0, len(pool), 12000)]
    t = {"probe": pr, "build": mv, "prefix": np.zeros(0, np.int32)}
    # 5000 movies with every one passing: more than the LDS table holds
    bpred = (Pred("year", "gt", 1900),) if n_movies > 1024 else (Pred("genre", "in", values=(2, 5, 11)),)
    q = Query(preds=(Pred("a", "lt", 90),), labels=(1, 2), decision="binary_gt", agg="count_by_payload",
              n_group_keys=0, join=Join("movie_id", "movie_id", payload, bpred))
    full_check(t, m, dm, q)


def test_hash_group_by_group_cap_and_empty(rel_model):
    say("case: hash group by with more groups than grp_cap, and with no survivors")
    m, dm = rel_model
    pr = table(3000, 77)
    pr["g"] = sparse_keys(3000, 7)
    t = {"probe": pr, "build": None, "prefix": np.zeros(0, np.int32)}
    q = Query(preds=(Pred("b", "lt", 40),), labels=(1, 2), decision="binary_gt", agg="avg_label_count_by",
              group_col="g", n_group_keys=0)
    full = full_check(t, m, dm, q)
    assert full["status"] == 0 and len(full["groups"][0]) > 5

    def cap5(dq):
        dq.out.grp_cap = 5

    capped = run(t, m, dm, q, tweak=cap5)
    # the groups past the cap are dropped and flagged; the first five (the
    # smallest keys) are the full run's
    assert capped["status"] == B.AIQ_DEV_GROUP_CAP
    assert len(capped["groups"][0]) == 5
    for a, b in zip(capped["groups"], full["groups"]):
        np.testing.assert_array_equal(a, b[:5])
    # nothing passes: no groups, no flag
    q0 = Query(preds=(Pred("b", "lt", -1000),), labels=(1, 2), decision="binary_gt", agg="avg_label_count_by",
               group_col="g", n_group_keys=0)
    r0 = run(t, m, dm, q0)
    assert r0["status"] == 0 and r0["n_selected"] == 0 and len(r0["groups"][0]) == 0
