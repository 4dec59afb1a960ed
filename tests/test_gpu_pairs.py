"""Pairs of rows classified together (Section 4, Q4: the self-join on the
movie id with AI_IF over [A.text, B.text]) on the device vs the oracle.

Exact: the candidate pairs (their number, rows and order), token totals,
kept pairs and COUNT given the labels, the cap and the key-range flag.  Label
logits within the fp32 / bf16 tolerance (all candidates on small tables, a
sample on the larger one)."""
import numpy as np
import pytest
import torch

from oracle.pairs import candidate_pairs, pair_sequences
from oracle.query import decide, margin, relational
from oracle.transformer import label_logits
from paper_2608_10139_amd import binding as B
from paper_2608_10139_amd.device import DeviceModel, DeviceQuery
from synth.configs import ModelSpec, Pred, Query
from synth.gen import make_model
from tests._parity import TOL_BF16, TOL_F32, check_labels

pytestmark = pytest.mark.gpu

F32 = ModelSpec(n_layers=1, d_model=64, n_heads=2, n_kv_heads=2, d_ff=64, vocab=500, act="gelu", dtype="f32",
                weight_seed=61, init_std=0.1)
BF16 = ModelSpec(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, d_ff=512, vocab=512, act="swiglu", dtype="bf16",
                 weight_seed=62, init_std=0.05)
_M = {}


def say(*a):
    print(*a, flush=True)


def model(spec):
    if spec not in _M:
        m = make_model(spec)
        _M[spec] = (m, DeviceModel(m))
    return _M[spec]


def tables(n, n_keys, seed, max_len=24, vocab=500, hot=0):
    r = np.random.default_rng(seed)
    lens = r.integers(0, max_len + 1, size=n).astype(np.int32)
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    keys = r.integers(0, n_keys, n).astype(np.int32)
    if hot:
        keys[r.choice(n, hot, replace=False)] = 7   # one key with many rows
    probe = {"id": np.arange(n, dtype=np.int32), "c": r.integers(0, 1000, n).astype(np.int32),
             "movie_id": keys, "len": lens, "offsets": off,
             "tokens": r.integers(3, vocab, int(off[-1])).astype(np.int32)}
    return {"probe": probe, "build": None, "prefix": r.integers(3, vocab, 16).astype(np.int32)}


def query(n_keys, max_pairs, npre=0):
    return Query(preds=(Pred("c", "lt", 500),), labels=(1, 2), decision="binary_gt", agg="count", n_prefix=npre,
                 pair_key="movie_id", n_group_keys=n_keys, max_pairs=max_pairs)


def run(t, m, dm, q, **kw):
    dq = DeviceQuery(t, m, q, dmodel=dm, **kw)
    dq.run()
    torch.cuda.synchronize()
    r = dq.results()
    dq.close()
    return r


def oracle_pairs(t, q, n_keys):
    rows, _ = relational(t, q)
    keys = t["probe"]["movie_id"][rows]
    rows = rows[(keys >= 0) & (keys < n_keys)]   # keys outside the domain are left out (and flagged)
    return candidate_pairs(t["probe"], rows, "movie_id")


def check(t, m, q, r, a, b, tol, sample=None):
    assert r["n_pairs"] == len(a)
    np.testing.assert_array_equal(r["cand_a"], a)
    np.testing.assert_array_equal(r["cand_b"], b)
    lens = t["probe"]["len"]
    assert r["n_tokens"] == int(lens[a].sum() + lens[b].sum()) + q.n_prefix * len(a)
    idx = np.arange(len(a)) if sample is None else sample
    seqs = pair_sequences(t["probe"], a[idx], b[idx], t["prefix"][:q.n_prefix])
    lg = label_logits(m, seqs, q.labels)
    labels = r["labels"].copy()
    labels[idx] = check_labels(r["logits"][idx], r["labels"][idx], lg, decide(lg, q), margin(lg, q), tol, "pairs")
    keep = labels == 1
    np.testing.assert_array_equal(r["kept_pairs"], np.flatnonzero(keep))
    np.testing.assert_array_equal(r["pair_a"], a[keep])
    np.testing.assert_array_equal(r["pair_b"], b[keep])
    assert r["count"] == int(keep.sum())


@pytest.mark.parametrize("n,n_keys", [(1, 4), (40, 3), (300, 20)])
def test_pairs_small_tables_fp32(n, n_keys):
    say(f"case: pairs, fp32 model, {n} rows, {n_keys} keys")
    m, dm = model(F32)
    t = tables(n, n_keys, n + n_keys)
    q = query(n_keys, 100_000)
    r = run(t, m, dm, q)
    assert r["status"] == 0, hex(r["status"])
    a, b = oracle_pairs(t, q, n_keys)
    say(f"  {r['n_selected']} selected rows, {r['n_pairs']} pairs, {r['count']} kept")
    check(t, m, q, r, a, b, TOL_F32)


def test_pairs_many_rows_hot_key_fp32():
    """More than one 1024-row round of the key sort, a key with ~170
    selected rows (more partners than a wave has lanes)."""
    say("case: pairs, 2,500 rows, a hot key")
    m, dm = model(F32)
    t = tables(2500, 400, 5, hot=340)
    q = query(400, 200_000)
    r = run(t, m, dm, q)
    assert r["status"] == 0, hex(r["status"])
    a, b = oracle_pairs(t, q, 400)
    say(f"  {r['n_selected']} selected rows, {r['n_pairs']} pairs, {r['count']} kept")
    assert r["n_selected"] > 1024 and len(a) > 10_000
    rng = np.random.default_rng(2)
    check(t, m, q, r, a, b, TOL_F32, sample=np.unique(rng.integers(0, len(a), 60)))


def test_pairs_cap_and_key_range():
    say("case: pairs cap and keys outside the domain")
    m, dm = model(F32)
    t = tables(300, 10, 9)
    t["probe"]["movie_id"][::17] = 10          # outside [0, 10)
    q = query(10, 100_000)
    full = run(t, m, dm, q)
    assert full["status"] == B.AIQ_DEV_GROUP_RANGE, hex(full["status"])
    a, b = oracle_pairs(t, q, 10)
    assert full["n_pairs"] == len(a)
    np.testing.assert_array_equal(full["cand_a"], a)
    cap = len(a) // 3
    r = run(t, m, dm, query(10, cap))
    assert r["status"] == B.AIQ_DEV_GROUP_RANGE | B.AIQ_DEV_PAIR_CAP, hex(r["status"])
    assert r["n_pairs"] == cap
    np.testing.assert_array_equal(r["cand_a"], a[:cap])
    np.testing.assert_array_equal(r["cand_b"], b[:cap])
    np.testing.assert_array_equal(r["logits"], full["logits"][:cap])   # a pair's result does not depend on the others


@pytest.mark.parametrize("share", [True, False])
def test_pairs_bf16_with_prefix(share):
    say(f"case: pairs, bf16 model, 16-token prefix, shared={share}")
    m, dm = model(BF16)
    t = tables(200, 12, 13, vocab=512)
    q = query(12, 100_000, npre=16)
    r = run(t, m, dm, q, share_prefix=share)
    assert r["status"] == 0, hex(r["status"])
    a, b = oracle_pairs(t, q, 12)
    check(t, m, q, r, a, b, TOL_BF16)
