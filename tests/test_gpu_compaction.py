"""The one-launch compaction (masks, stable compaction and token offsets with
a look-back across blocks of 8192 rows) against the oracle and against the
separate mask / scan / scatter launches: tables spanning one to several
hundred blocks, ragged tails, a join, a prompt prefix, empty and full
selections.  Ids, counts and token totals are exact; the full pipeline's
label logits (which depend on every token offset through the packing) are
bit-identical between the two compaction forms."""
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


def table(n, seed, vocab=500, max_len=12, tokens=True):
    r = np.random.default_rng(seed)
    lens = r.integers(0, max_len + 1, size=n).astype(np.int32)
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    ids = np.arange(n, dtype=np.int32)
    t = {"id": ids, "a": r.integers(-128, 128, n).astype(np.int8),
         "c": r.integers(0, 1000, n).astype(np.int32),
         # runs of 64 (63) consecutive rows alike: 64 (65 or 66) runs of survivors per block of 8192
         "g64": ((ids // 64) % 2).astype(np.int32), "g63": ((ids // 63) % 2).astype(np.int32),
         "len": lens, "offsets": off}
    if tokens:
        t["tokens"] = r.integers(0, vocab, int(off[-1])).astype(np.int32)
    return t


def run(tables, model, dm, q, **kw):
    dq = DeviceQuery(tables, model, q, dmodel=dm, **kw)
    dq.run()
    torch.cuda.synchronize()
    r = dq.results()
    dq.close()
    return r


def same(r1, r2):
    for k in ("status", "n_selected", "count", "n_tokens"):
        assert r1[k] == r2[k], k
    for k in ("kept_ids", "sel_ids", "labels"):
        np.testing.assert_array_equal(r1[k], r2[k], err_msg=k)
    np.testing.assert_array_equal(r1["logits"].view(np.int32), r2["logits"].view(np.int32))


# Survivor patterns: "mixed" about 30 % at random (thousands of runs of
# consecutive survivors per block of 8192 rows); "all" one run per block;
# "sparse" about 0.5 % (some 40 runs); "runs64" exactly 64 runs of 64 rows
# per block, aligned to the 64-row mask words; "runs63" 65 or 66 runs of 63
# rows, crossing word and block boundaries.
PATTERNS = {"mixed": (Pred("c", "lt", 300), Pred("a", "ne", 5)), "all": (Pred("c", "lt", 1000),),
            "sparse": (Pred("c", "lt", 5),), "runs64": (Pred("g64", "eq", 0),), "runs63": (Pred("g63", "eq", 0),)}
CASES = [(n, "mixed") for n in (8191, 8192, 8193, 3 * 8192 + 5, 70001)] + \
    [(n, p) for n in (8193, 70001) for p in ("all", "sparse", "runs64", "runs63")]


@pytest.mark.parametrize("n,pattern", CASES)
def test_one_launch_vs_multipass_full_pipeline(rel_model, n, pattern):
    say(f"case: one-launch vs multipass compaction, full pipeline, n={n}, {pattern}")
    m, dm = rel_model
    t = {"probe": table(n, 1000 + n), "build": None, "prefix": np.array([7, 8, 9], np.int32)}
    q = Query(preds=PATTERNS[pattern], labels=(1, 2), decision="binary_gt", agg="count", n_prefix=3)
    r1 = run(t, m, dm, q)
    r2 = run(t, m, dm, q, multipass_compact=True)
    rows, _ = relational(t, q)
    assert r1["status"] == 0 and r1["n_selected"] == len(rows)
    np.testing.assert_array_equal(r1["sel_ids"], rows)
    lens = np.diff(t["probe"]["offsets"])
    assert r1["n_tokens"] == int(lens[rows].sum()) + 3 * len(rows)
    same(r1, r2)


def test_one_launch_join_several_blocks(rel_model):
    say("case: one-launch compaction with a join over 5 blocks")
    m, dm = rel_model
    r = np.random.default_rng(21)
    nb = 900
    build = {"key": r.choice(1 << 30, nb, replace=False).astype(np.int32),
             "genre": r.integers(0, 20, nb).astype(np.int8), "year": r.integers(1950, 2026, nb).astype(np.int16)}
    n = 4 * 8192 + 333
    probe = table(n, 22)
    pool = np.concatenate([build["key"], np.array([-7, 1 << 30], np.int32)])   # dangling keys too
    probe["fk"] = pool[r.integers(0, len(pool), n)]
    t = {"probe": probe, "build": build, "prefix": np.array([3, 4], np.int32)}
    q = Query(preds=(Pred("a", "lt", 90),), labels=(1, 2), decision="binary_gt", agg="count_by_payload",
              n_prefix=2, n_group_keys=20,
              join=Join("fk", "key", "genre", (Pred("genre", "in", values=(2, 5, 11)), Pred("year", "gt", 1990))))
    r1 = run(t, m, dm, q)
    r2 = run(t, m, dm, q, multipass_compact=True)
    rows, _ = relational(t, q)
    assert r1["status"] == 0 and r1["n_selected"] == len(rows) > 0
    np.testing.assert_array_equal(r1["sel_ids"], rows)
    same(r1, r2)
    for a, b in zip(r1["groups"], r2["groups"]):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("k", [0, 5, 10, 1000])
def test_one_launch_many_blocks_relational_only(rel_model, k):
    """513 blocks (more than one 64-block look-back window, more blocks than
    fit on the chip at once): selected ids and the token total exact at
    0 %, 0.5 %, 1 % and 100 % selectivity, and equal to the multipass form."""
    n = 512 * 8192 + 4321
    say(f"case: one-launch compaction, relational only, n={n}, c < {k}")
    m, dm = rel_model
    probe = table(n, 77, max_len=1024, tokens=False)
    t = {"probe": probe, "build": None, "prefix": np.zeros(0, np.int32)}
    q = Query(preds=(Pred("c", "lt", k),), labels=(1, 2), decision="binary_gt", agg="count")
    r1 = run(t, m, dm, q, relational_only=True)
    r2 = run(t, m, dm, q, relational_only=True, multipass_compact=True)
    rows = np.flatnonzero(probe["c"] < k)
    assert r1["status"] == 0 and r1["n_selected"] == r1["count"] == len(rows)
    np.testing.assert_array_equal(r1["sel_ids"], rows)
    np.testing.assert_array_equal(r1["kept_ids"], rows)
    assert r1["n_tokens"] == int(probe["len"][rows].astype(np.int64).sum())
    for key in ("status", "n_selected", "count", "n_tokens"):
        assert r1[key] == r2[key]
    np.testing.assert_array_equal(r1["sel_ids"], r2["sel_ids"])
