"""Device pipeline vs the oracle on the tiny (fp32) and reviews (bf16)
workloads, through the C ABI: selection, label logits, decision, kept ids,
COUNT.  Plus determinism, packing and chunking invariance, and the
layer-by-layer prefill entry point."""
import numpy as np
import pytest
import torch

import oracle
from oracle.query import relational
from paper_2608_10139_amd.device import DeviceModel, DevicePrefill, DeviceQuery
from synth import WORKLOADS
from synth.gen import make_model, make_tables
from tests._parity import TOL_BF16, TOL_F32, check_labels, check_query, load_golden

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


_CACHE = {}


def workload(name):
    if name not in _CACHE:
        w = WORKLOADS[name]
        t = make_tables(w)
        t["model"] = make_model(w.model)
        t["workload"] = w
        _CACHE[name] = t
    return _CACHE[name]


def run_query(w, q, **kw):
    dq = DeviceQuery(w, w["model"], q, **kw)
    dq.run()
    torch.cuda.synchronize()
    r = dq.results()
    dq.close()
    return r


# ---------------------------------------------------------------- tiny, fp32

def test_tiny_end_to_end():
    say("case: tiny end-to-end (256 rows, fp32 2-layer)")
    w = workload("tiny")
    q = w["workload"].queries[0]
    g = load_golden("tiny")
    r = run_query(w, q)
    check_query(r, w, q, g["q0_rows"], None, g["q0_logits"], g["q0_labels"], g["q0_margin"], TOL_F32)


def test_tiny_run_to_run_bit_identical():
    say("case: tiny determinism")
    w = workload("tiny")
    q = w["workload"].queries[0]
    a, b = run_query(w, q), run_query(w, q)
    assert a["logits"].tobytes() == b["logits"].tobytes()
    np.testing.assert_array_equal(a["kept_ids"], b["kept_ids"])


def test_tiny_chunking_does_not_change_results():
    say("case: tiny chunked (chunk_tokens=300) vs one chunk")
    w = workload("tiny")
    q = w["workload"].queries[0]
    a = run_query(w, q)
    b = run_query(w, q, chunk_tokens=300)
    assert a["logits"].tobytes() == b["logits"].tobytes()
    np.testing.assert_array_equal(a["kept_ids"], b["kept_ids"])


# ---------------------------------------------------------------- reviews model, bf16, prefill entry

@pytest.fixture(scope="module", params=["f16", "bf16"])
def reviews_prefill(request):
    w = workload("reviews")
    dm = DeviceModel(w["model"], compute=request.param)
    return w, dm


def _seqs(w, rows):
    p = w["probe"]
    return [p["tokens"][p["offsets"][r]:p["offsets"][r + 1]].astype(np.int64) for r in rows]


def _packed(seqs):
    cu = np.zeros(len(seqs) + 1, dtype=np.int32)
    cu[1:] = np.cumsum([len(s) for s in seqs])
    tok = np.concatenate(seqs).astype(np.int32)
    return torch.from_numpy(tok).cuda(), torch.from_numpy(cu).cuda()


@pytest.mark.parametrize("n_layers", [0, 1, 4])
def test_reviews_prefill_layer_stack(reviews_prefill, n_layers):
    say(f"case: reviews prefill, {n_layers} layers")
    w, dm = reviews_prefill
    rows = [0, 1, 2, 3, 5, 8, 13, 21, 34, 55, 89, 144]
    seqs = _seqs(w, rows)
    tok, cu = _packed(seqs)
    pf = DevicePrefill(w["model"], labels=(1, 2), max_tokens=int(cu[-1].item()), n_layers=n_layers, dmodel=dm)
    got = pf.run(tok, cu).cpu().numpy()
    torch.cuda.synchronize()
    pf.close()
    ref = oracle.label_logits(w["model"], seqs, (1, 2), n_layers=n_layers)
    err = np.abs(got - ref).max()
    say(f"  max |dlogit| = {err:.3e}")
    assert err <= TOL_BF16


def test_reviews_packing_invariance_bitwise(reviews_prefill):
    say("case: reviews packing invariance")
    w, dm = reviews_prefill
    a, b, c = _seqs(w, [7, 11, 19])
    pf = DevicePrefill(w["model"], labels=(1, 2), max_tokens=len(a) + len(b) + len(c), dmodel=dm)
    alone = pf.run(*_packed([b])).cpu().numpy()
    mixed = pf.run(*_packed([a, b, c])).cpu().numpy()
    torch.cuda.synchronize()
    pf.close()
    assert alone[0].tobytes() == mixed[1].tobytes()


def test_reviews_full_vocab_head(reviews_prefill):
    say("case: reviews full-vocab head")
    w, dm = reviews_prefill
    seqs = _seqs(w, [3, 4, 5, 6])
    tok, cu = _packed(seqs)
    pf = DevicePrefill(w["model"], labels=(1, 2), max_tokens=int(cu[-1].item()), dmodel=dm)
    full = pf.run(tok, cu, full_vocab=True).cpu().numpy()
    lab = pf.run(tok, cu).cpu().numpy()
    torch.cuda.synchronize()
    pf.close()
    ref = oracle.full_logits(w["model"], seqs)
    assert np.abs(full - ref).max() <= TOL_BF16
    assert np.abs(full[:, [1, 2]] - lab).max() <= TOL_BF16


# ---------------------------------------------------------------- reviews end to end

@pytest.mark.parametrize("compute", ["f16", "bf16"])
def test_reviews_end_to_end(compute):
    say(f"case: reviews end-to-end (16,384 rows, 4-layer d512, {compute} projections)")
    g = load_golden("reviews")
    assert g is not None, "golden file for the reviews workload missing: run python -m tests.golden.make_golden reviews"
    w = workload("reviews")
    q = w["workload"].queries[0]
    r = run_query(w, q, dmodel=DeviceModel(w["model"], compute=compute))
    check_query(r, w, q, g["q0_rows"], None, g["q0_logits"], g["q0_labels"], g["q0_margin"], TOL_BF16)
    say(f"  selected {r['n_selected']} kept {r['count']} tokens {r['n_tokens']}")
