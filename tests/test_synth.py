"""The seeded generators: determinism and the stated distributions."""
import numpy as np

from synth import WORKLOADS
from synth.configs import ModelSpec
from synth.gen import (as_f32, bf16_round, make_model, make_movies, make_probe, make_tables,
                       zipf_cdf)


def test_tables_are_deterministic():
    a = make_tables(WORKLOADS["tiny"])["probe"]
    b = make_tables(WORKLOADS["tiny"])["probe"]
    for k in a:
        assert a[k].tobytes() == b[k].tobytes()


def test_tiny_table_shape():
    t = make_tables(WORKLOADS["tiny"])["probe"]
    assert t["id"].tolist() == list(range(256))
    assert t["len"].min() >= 8 and t["len"].max() <= 64
    assert t["rating"].min() >= 1 and t["rating"].max() <= 5
    assert t["tokens"].max() < 1024 and t["tokens"].min() >= 0
    assert np.array_equal(np.diff(t["offsets"]), t["len"])


def test_reviews_distributions():
    t = make_probe(WORKLOADS["reviews"].table)
    L = t["len"]
    assert L.min() >= 16 and L.max() <= 512
    assert abs(np.median(L) - 120) <= 3
    # rating probabilities .1 .1 .2 .3 .3 (16384 draws: 4-sigma band)
    p = np.bincount(t["rating"], minlength=6)[1:] / len(L)
    for got, exp in zip(p, (0.1, 0.1, 0.2, 0.3, 0.3)):
        assert abs(got - exp) < 4 * np.sqrt(exp * (1 - exp) / len(L))
    # bounded Zipf(1.1) over 32000: mass of token 0 is 1 / H(32000, 1.1)
    p1 = 1.0 / np.sum(np.arange(1, 32001, dtype=np.float64) ** -1.1)
    assert abs(p1 - 0.142) < 0.001
    f = np.mean(t["tokens"] == 0)
    assert abs(f - p1) < 4 * np.sqrt(p1 * (1 - p1) / len(t["tokens"]))


def test_zipf_keys_top_mass():
    p1 = 1.0 / np.sum(np.arange(1, 4097, dtype=np.float64) ** -1.2)
    assert abs(p1 - 0.2153) < 1e-3
    cdf = zipf_cdf(1.2, 4096)
    assert cdf[-1] == 1.0 and np.all(np.diff(cdf) > 0)


def test_movies_and_fk():
    w = WORKLOADS["join1b"]
    m = make_movies(w.movies)
    assert len(np.unique(m["movie_id"])) == 8192
    assert m["movie_id"].min() >= 0
    assert m["genre"].min() >= 0 and m["genre"].max() <= 19
    assert m["year"].min() >= 1950 and m["year"].max() <= 2025


def test_bf16_round_nearest_even():
    x = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-8, 1.0 + 2**-9, -2.5], dtype=np.float32)
    got = as_f32(bf16_round(x))
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7 -> even (1.0); 1 + 3*2^-8 ties up to 1 + 2^-6
    assert got.tolist() == [1.0, 1.0, 1.0 + 2**-6, 1.0, -2.5]


def test_model_streams_independent_of_depth():
    spec = ModelSpec(n_layers=3, d_model=32, n_heads=2, n_kv_heads=1, d_ff=40, vocab=50,
                     act="swiglu", dtype="bf16", weight_seed=9)
    full = make_model(spec)
    short = make_model(spec, n_layers=2)
    assert full["layers"][1]["wq"].tobytes() == short["layers"][1]["wq"].tobytes()
    assert full["emb"].dtype == np.uint16
    s = as_f32(full["layers"][0]["w_gate"]).std()
    assert 0.015 < s < 0.025
