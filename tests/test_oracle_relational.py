"""Pins of the oracle's relational steps against brute-force pure-Python loops
on tiny tables, and of the join against its foreign-key invariant."""
import numpy as np
import pytest

import oracle
from oracle.query import aggregate, decide, margin, relational
from oracle.relational import eval_pred, sum_f32
from synth.configs import Join, Pred, Query

OPS = {"lt": lambda a, b: a < b, "le": lambda a, b: a <= b, "gt": lambda a, b: a > b,
       "ge": lambda a, b: a >= b, "eq": lambda a, b: a == b, "ne": lambda a, b: a != b}


def tiny_table(seed, n=300):
    r = np.random.default_rng(seed)
    lens = r.integers(0, 9, size=n).astype(np.int32)
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    return {
        "id": np.arange(n, dtype=np.int32),
        "a": r.integers(-128, 128, size=n).astype(np.int8),
        "b": r.integers(-300, 300, size=n).astype(np.int16),
        "c": r.integers(-2**31, 2**31 - 1, size=n, dtype=np.int64).astype(np.int32),
        "len": lens, "offsets": off,
        "tokens": r.integers(0, 50, size=int(off[-1])).astype(np.int32),
    }


def brute_select(t, preds):
    out = []
    for r in range(len(t["id"])):
        ok = True
        for p in preds:
            v = int(t[p.col][r])
            if p.op == "in":
                ok = ok and any(v == x for x in p.values)
            else:
                ok = ok and OPS[p.op](v, p.k)
        if ok:
            out.append(r)
    return out


@pytest.mark.parametrize("seed", range(6))
def test_select_matches_brute_force(seed):
    t = tiny_table(seed)
    r = np.random.default_rng(100 + seed)
    preds = []
    for col in ("a", "b", "c"):
        op = ["lt", "le", "gt", "ge", "eq", "ne", "in"][int(r.integers(0, 7))]
        pick = int(t[col][int(r.integers(0, len(t["id"])))])
        if op == "in":
            preds.append(Pred(col, "in", values=(pick, pick + 1, -5)))
        else:
            preds.append(Pred(col, op, pick))
        got = oracle.select(t, tuple(preds), len(t["id"]))
        assert got.tolist() == brute_select(t, preds)


def test_select_empty_conjunction_and_empty_result():
    t = tiny_table(9)
    assert oracle.select(t, (), 300).tolist() == list(range(300))
    assert oracle.select(t, (Pred("a", "gt", 127),), 300).tolist() == []


def test_int_widening_is_exact():
    # int8 column against constants outside its range, and int32 extremes
    t = {"a": np.array([-128, 0, 127], dtype=np.int8), "c": np.array([-2**31, 0, 2**31 - 1], dtype=np.int32)}
    assert oracle.select(t, (Pred("a", "lt", 128),), 3).tolist() == [0, 1, 2]
    assert oracle.select(t, (Pred("a", "ge", -129),), 3).tolist() == [0, 1, 2]
    assert oracle.select(t, (Pred("c", "gt", 2**31 - 2),), 3).tolist() == [2]
    assert oracle.select(t, (Pred("c", "le", -2**31),), 3).tolist() == [0]


def movies_and_reviews(seed, n_movies=40, n_reviews=500):
    r = np.random.default_rng(seed)
    ids = r.choice(10_000, size=n_movies, replace=False).astype(np.int32)
    movies = {"movie_id": ids, "genre": r.integers(0, 20, n_movies).astype(np.int8),
              "year": r.integers(1950, 2026, n_movies).astype(np.int16)}
    pool = np.concatenate([ids, np.array([10_001, 10_002], dtype=np.int32)])  # some dangling keys
    reviews = tiny_table(seed, n_reviews)
    reviews["movie_id"] = pool[r.integers(0, len(pool), n_reviews)]
    return movies, reviews


@pytest.mark.parametrize("seed", range(4))
def test_join_matches_nested_loops(seed):
    movies, reviews = movies_and_reviews(seed)
    j = Join("movie_id", "movie_id", "genre", (Pred("genre", "in", values=(2, 5, 11)), Pred("year", "gt", 2000)))
    probe_rows = oracle.select(reviews, (Pred("a", "ge", -50),), len(reviews["id"]))
    rows, pay = oracle.hash_join(reviews, movies, j, probe_rows)
    exp_r, exp_p = [], []
    for r in probe_rows:
        for m in range(len(movies["movie_id"])):
            if (movies["movie_id"][m] == reviews["movie_id"][r] and movies["genre"][m] in (2, 5, 11)
                    and movies["year"][m] > 2000):
                exp_r.append(int(r)); exp_p.append(int(movies["genre"][m]))
    assert rows.tolist() == exp_r and pay.tolist() == exp_p


def test_join_fk_invariant_and_duplicate_key():
    movies, reviews = movies_and_reviews(7)
    reviews["movie_id"] = movies["movie_id"][np.random.default_rng(1).integers(0, 40, 500)]
    j = Join("movie_id", "movie_id", "genre", ())
    rows, pay = oracle.hash_join(reviews, movies, j, np.arange(500))
    assert len(rows) == 500   # every review matches exactly one movie
    bad = dict(movies, movie_id=movies["movie_id"].copy())
    bad["movie_id"][3] = bad["movie_id"][4]
    with pytest.raises(ValueError):
        oracle.hash_join(reviews, bad, j, np.arange(500))


def test_sequences_and_pack_identities():
    t = tiny_table(3)
    rows = np.array([0, 5, 7, 299])
    pre = np.array([91, 92, 93])
    seqs = oracle.sequences(t, rows, pre)
    for s, r in zip(seqs, rows):
        exp = [91, 92, 93] + [int(t["tokens"][i]) for i in range(t["offsets"][r], t["offsets"][r + 1])]
        assert s.tolist() == exp
    cu, flat = oracle.pack(seqs)
    assert cu[0] == 0 and cu[-1] == len(flat) == sum(len(s) for s in seqs)
    assert np.all(np.diff(cu) == [len(s) for s in seqs])
    for i, s in enumerate(seqs):
        assert flat[cu[i]:cu[i + 1]].tolist() == s.tolist()


def test_group_avg_count_matches_dict():
    r = np.random.default_rng(5)
    keys = r.integers(0, 30, 1000); vals = r.integers(1, 6, 1000)
    k, c, s, a = oracle.group_avg_count(keys, vals)
    d = {}
    for kk, vv in zip(keys.tolist(), vals.tolist()):
        cc, ss = d.get(kk, (0, 0)); d[kk] = (cc + 1, ss + vv)
    assert k.tolist() == sorted(d)
    assert c.tolist() == [d[x][0] for x in sorted(d)]
    assert s.tolist() == [d[x][1] for x in sorted(d)]
    assert a.tolist() == [d[x][1] / d[x][0] for x in sorted(d)]
    assert oracle.group_avg_count(np.zeros(0), np.zeros(0))[0].size == 0


def test_group_avg_count_any_int32_key():
    # negative keys, both int32 extremes and sparse keys order like plain integers
    keys = np.array([2**31 - 1, -2**31, -7, 5, -7, 0, -2**31, 123456789, 5, -1], dtype=np.int32)
    vals = np.array([3, 1, 2, 4, 5, 1, 2, 3, 3, 2])
    k, c, s, a = oracle.group_avg_count(keys, vals)
    assert k.tolist() == [-2**31, -7, -1, 0, 5, 123456789, 2**31 - 1]
    assert c.tolist() == [2, 2, 1, 1, 2, 1, 1]
    assert s.tolist() == [3, 7, 2, 1, 7, 3, 3]
    assert a.tolist() == [1.5, 3.5, 2.0, 1.0, 3.5, 3.0, 3.0]
    kk, cc = oracle.count_by(keys)
    assert kk.tolist() == k.tolist() and cc.tolist() == c.tolist()


def test_decision_strict_and_argmax_ties():
    qb = Query(preds=(), labels=(1, 2), decision="binary_gt", agg="count")
    lg = np.array([[1.0, 0.5], [0.5, 0.5], [0.1, 0.2]])
    assert decide(lg, qb).tolist() == [1, 0, 0]          # equal logits reject
    qa = Query(preds=(), labels=(1, 2, 3, 4, 5), decision="argmax", agg="count")
    lg = np.array([[0, 3, 3, 1, 0], [5, 0, 0, 0, 5], [0, 0, 0, 0, 1.0]])
    assert decide(lg, qa).tolist() == [2, 1, 5]           # ties go to the lowest index
    np.testing.assert_allclose(margin(lg, qa), [0, 0, 1])


def test_aggregate_binary_count_and_groups():
    t = tiny_table(11, 50)
    t["movie_id"] = (np.arange(50) % 7).astype(np.int32)
    rows = np.array([1, 4, 9, 20, 33])
    labels = np.array([1, 0, 1, 1, 0])
    q = Query(preds=(), labels=(1, 2), decision="binary_gt", agg="count")
    out = aggregate({"probe": t}, rows, None, labels, q)
    assert out["kept_ids"].tolist() == [1, 9, 20] and out["count"] == 3
    qg = Query(preds=(), labels=(1, 2, 3), decision="argmax", agg="avg_label_count_by",
               group_col="movie_id", n_group_keys=7)
    out = aggregate({"probe": t}, rows, None, np.array([3, 1, 2, 3, 1]), qg)
    # keys: 1, 4, 2, 6, 5 -> one row each
    assert out["groups"][0].tolist() == [1, 2, 4, 5, 6]
    assert out["groups"][2].tolist() == [3, 2, 1, 1, 3]
    qp = Query(preds=(), labels=(1, 2), decision="binary_gt", agg="count_by_payload", n_group_keys=20)
    out = aggregate({"probe": t}, rows, np.array([5, 5, 2, 5, 9]), labels, qp)
    assert out["groups"][0].tolist() == [2, 5] and out["groups"][1].tolist() == [1, 2]


def test_relational_with_join_end_to_end():
    movies, reviews = movies_and_reviews(2)
    j = Join("movie_id", "movie_id", "genre", (Pred("year", "gt", 1990),))
    q = Query(preds=(Pred("b", "lt", 100),), labels=(1, 2), decision="binary_gt", agg="count_by_payload",
              join=j, n_group_keys=20)
    rows, pay = relational({"probe": reviews, "build": movies}, q)
    exp = [r for r in brute_select(reviews, q.preds)
           if any(movies["movie_id"][m] == reviews["movie_id"][r] and movies["year"][m] > 1990
                  for m in range(40))]
    assert rows.tolist() == exp


# ---------------------------------------------------------------- float columns and SUM

def test_float_predicate_matches_python_comparisons():
    """fp32 columns compare exactly against the fp64 constant, IEEE semantics:
    values at, just below and just above the threshold, signed zeros, NaN."""
    k = 70.0
    up = float(np.nextafter(np.float32(k), np.float32(np.inf)))
    dn = float(np.nextafter(np.float32(k), np.float32(-np.inf)))
    vals = np.array([k, up, dn, 0.0, -0.0, np.nan, np.inf, -np.inf, 69.99999, 70.00001, 1e30, -1e-30],
                    dtype=np.float32)
    cols = {"v": vals}
    import operator
    ops = {"lt": operator.lt, "le": operator.le, "gt": operator.gt, "ge": operator.ge,
           "eq": operator.eq, "ne": operator.ne}
    for name, f in ops.items():
        for kk in (k, 0.0, -0.0, 70.00001, float(np.float32(0.1)), 0.1):
            got = eval_pred(cols, Pred("v", name, kk))
            want = np.array([f(float(x), kk) for x in vals])
            np.testing.assert_array_equal(got, want, err_msg=f"{name} {kk}")
    # the fp64 constant is not rounded to fp32 first: 0.1 (fp64) > 0.1f32 is False
    assert not eval_pred({"v": np.float32([0.1])}, Pred("v", "lt", 0.1))[0]
    with pytest.raises(ValueError):
        eval_pred(cols, Pred("v", "in", values=(1,)))


def test_sum_f32_is_the_exactly_rounded_sum():
    """SUM equals the rational sum of the fp32 values rounded once to fp64:
    checked with exact Fraction arithmetic on random values of mixed scale,
    on cancelling pairs (exactly 0) and on a closed form."""
    from fractions import Fraction
    r = np.random.default_rng(3)
    for n in (1, 2, 17, 500):
        v = (r.standard_normal(n) * 10.0 ** r.integers(-20, 20, n)).astype(np.float32)
        exact = sum((Fraction(float(x)) for x in v), Fraction(0))
        assert sum_f32(v) == float(exact)
    v = r.standard_normal(999).astype(np.float32)
    assert sum_f32(np.concatenate([v, -v[::-1]])) == 0.0
    # closed form: n copies of x sum to n * x exactly while below 2^53 ulps
    x = np.float32(0.1)
    assert sum_f32(np.full(1000, x, dtype=np.float32)) == float(Fraction(float(x)) * 1000)
    assert sum_f32(np.zeros(0, dtype=np.float32)) == 0.0


def test_sum_f32_non_finite_follows_ieee():
    inf, nan = np.float32(np.inf), np.float32(np.nan)
    assert sum_f32(np.float32([1, inf, 2])) == np.inf
    assert sum_f32(np.float32([-inf, 5])) == -np.inf
    assert np.isnan(sum_f32(np.float32([inf, -inf])))
    assert np.isnan(sum_f32(np.float32([1, nan])))
    # the same as IEEE left-to-right addition in any order
    for v in ([1, inf, -3], [inf, -inf, 2], [nan, 1], [-inf, -inf]):
        a = np.float32(v).astype(np.float64)
        for order in (a, a[::-1]):
            acc = 0.0
            for x in order:
                acc += x
            got = sum_f32(np.float32(v))
            assert (np.isnan(acc) and np.isnan(got)) or acc == got


def test_aggregate_sum_over_kept_rows():
    probe = {"v": np.float32([1.5, 2.25, -4.0, 8.0, 0.125]), "id": np.arange(5, dtype=np.int32)}
    q = Query(preds=(), labels=(1, 2), decision="binary_gt", agg="sum_f32", group_col="v")
    rows = np.array([0, 1, 3, 4])
    labels = np.array([1, 0, 1, 1])
    out = aggregate({"probe": probe}, rows, None, labels, q)
    assert out["count"] == 3
    np.testing.assert_array_equal(out["kept_ids"], [0, 3, 4])
    assert out["sum"] == 1.5 + 8.0 + 0.125
