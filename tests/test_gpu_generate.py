"""AI_TRANSFORM on the device: greedy generation after the prefill and the
LIKE filter over the generated tokens (Table 1; Section 4, Q3 and Q5).

Several generations are correct where two logits are within rounding of each
other, so the device's tokens are checked for validity rather than equality:
with the oracle's fp64 logits over prompt + the device's own earlier tokens
(one forward, teacher forcing), every generated token must be within the bf16
tolerance of that position's maximum.  Everything else is exact: the pad
after the end token, the LIKE flags recomputed by the oracle from the
device's tokens, kept ids and COUNT, and bit-identical tokens across runs,
chunkings and the shared / per-row prompt prefix.
"""
import numpy as np
import pytest
import torch

from oracle.generate import generated_length, like_tokens, position_logits
from oracle.query import relational
from paper_2608_10139_amd.device import DeviceModel, DeviceQuery
from synth.configs import ModelSpec, Pred, Query
from synth.gen import make_model
from tests._parity import TOL_BF16

pytestmark = pytest.mark.gpu

MODELS = {
    "hd64": ModelSpec(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, d_ff=512, vocab=1024, act="swiglu",
                      dtype="bf16", weight_seed=31, init_std=0.05),
    "hd128": ModelSpec(n_layers=2, d_model=512, n_heads=8, n_kv_heads=2, d_ff=512, vocab=1024, act="swiglu",
                       dtype="bf16", weight_seed=32, init_std=0.05),
}
_M = {}


def say(*a):
    print(*a, flush=True)


def model(name):
    if name not in _M:
        m = make_model(MODELS[name])
        _M[name] = (m, DeviceModel(m))
    return _M[name]


def tables(n, seed, max_len=40, vocab=1024):
    r = np.random.default_rng(seed)
    lens = r.integers(1, max_len + 1, size=n).astype(np.int32)
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    probe = {"id": np.arange(n, dtype=np.int32), "c": r.integers(0, 1000, n).astype(np.int32), "len": lens,
             "offsets": off, "tokens": r.integers(0, vocab, int(off[-1])).astype(np.int32)}
    return {"probe": probe, "build": None, "prefix": r.integers(0, vocab, 64).astype(np.int32)}


def query(G, npre=0, eos=-1, pad=0, like=()):
    return Query(preds=(Pred("c", "lt", 500),), labels=(), decision="binary_gt", agg="count", n_prefix=npre,
                 gen_tokens=G, eos_id=eos, pad_id=pad, like=tuple(like))


def run(t, m, dm, q, **kw):
    dq = DeviceQuery(t, m, q, dmodel=dm, **kw)
    dq.run()
    torch.cuda.synchronize()
    r = dq.results()
    dq.close()
    return r


def check_valid_tokens(m, t, q, r, sample):
    """Teacher forcing: each generated token is within tol of that step's
    maximal oracle logit (given the device's earlier tokens)."""
    rows, _ = relational(t, q)
    pre = t["prefix"][:q.n_prefix].astype(np.int64)
    off, tok = t["probe"]["offsets"], t["probe"]["tokens"]
    exact = total = 0
    for i in sample:
        row = int(rows[i])
        prompt = np.concatenate([pre, tok[off[row]:off[row + 1]].astype(np.int64)])
        gen = r["gen"][i]
        n = generated_length(gen, q.eos_id)
        assert np.all(gen[n:] == q.pad_id), f"row {row}: slots after the end are not pad"
        lg = position_logits(m, np.concatenate([prompt, gen[:n - 1]]))[len(prompt) - 1:]
        assert lg.shape[0] == n
        top = lg.max(axis=1)
        got = lg[np.arange(n), gen[:n]]
        gap = top - got
        assert gap.max() <= TOL_BF16, f"row {row}: token {int(gap.argmax())} is {gap.max():.3e} below the maximum"
        exact += int(np.sum(lg.argmax(axis=1) == gen[:n]))
        total += n
    return exact, total


@pytest.mark.parametrize("mname", ["hd64", "hd128"])
def test_generation_tokens_are_greedy(mname):
    say(f"case: generation validity, model {mname}")
    m, dm = model(mname)
    t = tables(300, 41)
    q = query(12)
    r = run(t, m, dm, q)
    assert r["status"] == 0
    rows, _ = relational(t, q)
    np.testing.assert_array_equal(r["sel_ids"], rows)
    assert r["gen"].shape == (len(rows), 12)
    assert r["count"] == len(rows)          # no LIKE: every selected row kept
    np.testing.assert_array_equal(r["kept_ids"], rows)
    rng = np.random.default_rng(1)
    lens = t["probe"]["len"][rows]
    sample = np.unique(np.concatenate([rng.integers(0, len(rows), 20), [int(np.argmin(lens)), int(np.argmax(lens))]]))
    exact, total = check_valid_tokens(m, t, q, r, sample)
    say(f"  {exact}/{total} sampled tokens equal the oracle's own argmax")
    assert exact >= 0.9 * total


def test_generation_end_token_and_like():
    say("case: end token, pad, LIKE flags and COUNT")
    m, dm = model("hd64")
    t = tables(400, 43)
    free = run(t, m, dm, query(10))
    # an end token the rows actually produce, and a pattern some rows contain
    vals, cnts = np.unique(free["gen"][:, 1:], return_counts=True)
    eos = int(vals[np.argmax(cnts)])
    g = free["gen"]
    i0 = next(i for i in range(len(g)) if generated_length(g[i], eos) >= 4)
    pat = (int(g[i0, 2]), int(g[i0, 3]))
    q = query(10, eos=eos, pad=1023, like=pat)
    r = run(t, m, dm, q)
    assert r["status"] == 0
    rows, _ = relational(t, q)
    for i in range(len(rows)):
        n = generated_length(free["gen"][i], eos)
        np.testing.assert_array_equal(r["gen"][i, :n], free["gen"][i, :n])   # same greedy path up to the end
        assert np.all(r["gen"][i, n:] == 1023)
    flags = np.array([like_tokens(r["gen"][i], pat, eos) for i in range(len(rows))])
    assert 0 < flags.sum() < len(rows)
    np.testing.assert_array_equal(r["labels"], flags.astype(np.int64))
    np.testing.assert_array_equal(r["kept_ids"], rows[flags])
    assert r["count"] == int(flags.sum())
    check_valid_tokens(m, t, q, r, np.arange(0, len(rows), 17))


@pytest.mark.parametrize("npre", [32, 33])
def test_generation_shared_prefix_bitwise_equals_per_row(npre):
    say(f"case: generation with a {npre}-token prefix, shared vs per row")
    m, dm = model("hd128")
    t = tables(300, 47)
    q = query(8, npre=npre)
    a = run(t, m, dm, q)
    b = run(t, m, dm, q, share_prefix=False)
    assert a["status"] == 0 and b["status"] == 0
    np.testing.assert_array_equal(a["gen"], b["gen"])
    check_valid_tokens(m, t, q, a, np.arange(0, a["n_selected"], 11))


def test_generation_chunking_and_repeat_bitwise():
    say("case: generation over several chunks vs one, and a repeated run")
    m, dm = model("hd64")
    t = tables(600, 53)
    q = query(6)
    one = run(t, m, dm, q)
    many = run(t, m, dm, q, chunk_tokens=2048)
    again = run(t, m, dm, q)
    np.testing.assert_array_equal(one["gen"], many["gen"])
    np.testing.assert_array_equal(one["gen"], again["gen"])
    np.testing.assert_array_equal(one["kept_ids"], many["kept_ids"])


def test_first_token_is_the_argmax_of_the_full_vocabulary_logits():
    """The generation head keeps only per-64-column maxima; its first token
    must equal the argmax (lowest id on ties) of the full fp32 logits that
    the prefill-only entry point writes for the same prompts."""
    from paper_2608_10139_amd.device import DevicePrefill
    say("case: first generated token vs full-vocabulary logits")
    m, dm = model("hd64")
    t = tables(200, 59)
    q = query(3)
    r = run(t, m, dm, q)
    rows, _ = relational(t, q)
    off, tok = t["probe"]["offsets"], t["probe"]["tokens"]
    seqs = [tok[off[x]:off[x + 1]] for x in rows]
    cu = np.zeros(len(seqs) + 1, dtype=np.int32)
    cu[1:] = np.cumsum([len(s) for s in seqs])
    pf = DevicePrefill(m, max_tokens=int(cu[-1]), dmodel=dm)
    lg = pf.run(torch.from_numpy(np.concatenate(seqs).astype(np.int32)).cuda(), torch.from_numpy(cu).cuda(),
                full_vocab=True)
    torch.cuda.synchronize()
    lg = lg.cpu().numpy()
    pf.close()
    np.testing.assert_array_equal(r["gen"][:, 0], lg.argmax(axis=1))


# ---------------------------------------------------------------- the benchmarked shapes
_W = {}


def reviews_workload(name):
    """The reviews table (16,384 rows) and its 4-layer d512 model with the
    32,000-token vocabulary."""
    from synth import WORKLOADS
    from synth.gen import make_tables
    if name not in _W:
        w = WORKLOADS[name]
        m = make_model(w.model)
        _W.clear()
        _W[name] = (w, make_tables(w), m, DeviceModel(m))
    return _W[name]


def spread_sample(n, k, seed):
    """k indices over [0, n): the first and last rows, both sides of every
    4,096-row block edge of the generation head, and seeded picks."""
    edges = [0, n - 1] + [e + d for e in range(4096, n, 4096) for d in (-1, 0)]
    rng = np.random.default_rng(seed)
    pick = set(i for i in edges if 0 <= i < n)
    while len(pick) < min(k, n):
        pick.add(int(rng.integers(0, n)))
    return np.array(sorted(pick))


@pytest.mark.timeout(300)
def test_q3_generation_at_vocab_32000_over_several_head_blocks():
    """Q3 at values_a < 50: 8,187 selected rows (two 4,096-row blocks of the
    full-vocabulary head), 32 new tokens after an 8-token shared prompt."""
    say("case: Q3 generation, reviews table, values_a < 50, vocab 32,000")
    w, t, m, dm = reviews_workload("reviews_transform")
    q = w.queries[2]
    r = run(t, m, dm, q)
    assert r["status"] == 0, hex(r["status"])
    rows, _ = relational(t, q)
    np.testing.assert_array_equal(r["sel_ids"], rows)
    assert len(rows) > 4096 and r["gen"].shape == (len(rows), 32)
    assert r["count"] == len(rows)
    np.testing.assert_array_equal(r["kept_ids"], rows)
    sample = spread_sample(len(rows), 128, 7)
    exact, total = check_valid_tokens(m, t, q, r, sample)
    say(f"  {exact}/{total} sampled tokens equal the oracle's own argmax")
    assert exact >= 0.9 * total


@pytest.mark.timeout(300)
def test_q5_long_generation_with_end_token_and_like():
    """Q5: every row (16,384; four head blocks), 128 new tokens, end token 2,
    LIKE over the generated tokens; flags, kept ids and COUNT recomputed by the
    oracle from the device's tokens, and sampled tokens valid."""
    say("case: Q5 generation + LIKE, reviews table, 128 tokens, vocab 32,000")
    w, t, m, dm = reviews_workload("reviews_like")
    q = w.queries[0]
    r = run(t, m, dm, q)
    assert r["status"] == 0, hex(r["status"])
    rows, _ = relational(t, q)
    np.testing.assert_array_equal(r["sel_ids"], rows)
    flags = np.array([like_tokens(r["gen"][i], q.like, q.eos_id) for i in range(len(rows))])
    np.testing.assert_array_equal(r["labels"], flags.astype(np.int64))
    np.testing.assert_array_equal(r["kept_ids"], rows[flags])
    assert r["count"] == int(flags.sum())
    sample = spread_sample(len(rows), 128, 9)
    exact, total = check_valid_tokens(m, t, q, r, sample)
    say(f"  {exact}/{total} sampled tokens equal the oracle's own argmax; {int(flags.sum())} rows kept")
    assert exact >= 0.9 * total
