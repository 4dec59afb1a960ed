"""Comparison of device results with the oracle (shared by the GPU tests)."""
import os

import numpy as np

from oracle.query import aggregate

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

TOL_F32 = 1e-4   # |logit difference| bound for fp32 models
TOL_BF16 = 2e-2  # ... and for bf16 models


def load_golden(name):
    path = os.path.join(GOLDEN, f"{name}_oracle.npz")
    if not os.path.exists(path):
        return None
    with np.load(path, allow_pickle=False) as z:
        return {k: z[k] for k in z.files}


def check_labels(gpu_logits, gpu_labels, ref_logits, ref_labels, ref_margin, tol, what=""):
    """Logits within tol; labels equal except where the oracle's margin is inside tol.
    Returns the oracle labels with the device's choice adopted inside the band."""
    gpu_logits = np.asarray(gpu_logits, dtype=np.float64)
    err = np.abs(gpu_logits - ref_logits)
    assert np.all(np.isfinite(gpu_logits)), f"{what}: non-finite logits"
    assert err.max(initial=0.0) <= tol, f"{what}: max |dlogit| {err.max():.3e} > {tol} at row {int(err.max(1).argmax())}"
    band = ref_margin < tol
    diff = gpu_labels != ref_labels
    assert not np.any(diff & ~band), f"{what}: {int((diff & ~band).sum())} label mismatches outside the tie band"
    return np.where(band, gpu_labels, ref_labels)


def check_query(res, tables, query, rows, payload, ref_logits, ref_labels, ref_margin, tol, sample=None):
    """Full comparison of one aiq_run against the oracle.

    rows: oracle's selected rows (exact match required).  With ``sample`` the
    oracle logits cover only those indices; the aggregate is then recomputed
    from the device's labels and compared exactly."""
    assert res["status"] == 0, f"device status {res['status']:#x}"
    np.testing.assert_array_equal(res["sel_ids"], rows)
    assert res["n_selected"] == len(rows)
    n_tok = int(tables["probe"]["len"][rows].sum()) + len(rows) * query.n_prefix
    assert res["n_tokens"] == n_tok
    labels = res["labels"].copy()
    if sample is None:
        labels = check_labels(res["logits"], res["labels"], ref_logits, ref_labels, ref_margin, tol, "all rows")
    else:
        adopted = check_labels(res["logits"][sample], res["labels"][sample], ref_logits, ref_labels,
                               ref_margin, tol, "sample")
        labels[sample] = adopted
    agg = aggregate(tables, rows, payload, labels, query)
    np.testing.assert_array_equal(res["kept_ids"], agg["kept_ids"])
    assert res["count"] == agg["count"]
    if "groups" in agg:
        for a, b in zip(res["groups"], agg["groups"]):
            np.testing.assert_array_equal(np.asarray(a), np.asarray(b).astype(np.asarray(a).dtype))
    return labels
