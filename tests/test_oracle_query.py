"""End-to-end oracle on the tiny workload, pinned against brute-force selection
and the independent torch-fp64 forward."""
import numpy as np

import oracle
from synth import make_workload
from tests._torch_ref import forward_last_logits


def test_tiny_workload_end_to_end():
    w = make_workload("tiny")
    q = w["workload"].queries[0]
    res = oracle.run_query(w, w["model"], q)
    probe = w["probe"]
    exp_rows = [r for r in range(256) if int(probe["rating"][r]) >= 3]
    assert res["rows"].tolist() == exp_rows
    for i in range(0, len(exp_rows), 7):
        r = exp_rows[i]
        seq = probe["tokens"][probe["offsets"][r]:probe["offsets"][r + 1]]
        ref = forward_last_logits(w["model"], seq, q.labels).numpy()
        np.testing.assert_allclose(res["logits"][i], ref, rtol=1e-10, atol=1e-12)
    kept = [exp_rows[i] for i in range(len(exp_rows)) if res["logits"][i, 0] > res["logits"][i, 1]]
    assert res["kept_ids"].tolist() == kept and res["count"] == len(kept)
    assert res["n_tokens"] == int(sum(probe["len"][exp_rows]))
