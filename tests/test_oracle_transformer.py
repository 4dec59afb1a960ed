"""Pins of the oracle's transformer against closed forms, invariants and an
independent torch-fp64 formulation (no test here compares the oracle with
itself)."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle.transformer import forward_hidden
from synth.configs import ModelSpec
from synth.gen import make_model, as_f32
from tests._torch_ref import forward_last_logits, rope_complex

RNG = np.random.default_rng(1234)

GQA = ModelSpec(n_layers=2, d_model=64, n_heads=8, n_kv_heads=2, d_ff=96, vocab=97,
                act="swiglu", dtype="bf16", weight_seed=77, init_std=0.08)
GELU = ModelSpec(n_layers=2, d_model=32, n_heads=4, n_kv_heads=4, d_ff=48, vocab=61,
                 act="gelu", dtype="f32", weight_seed=78, init_std=0.1)


@pytest.fixture(scope="module", params=[GQA, GELU], ids=["swiglu-gqa-bf16", "gelu-mha-f32"])
def model(request):
    return make_model(request.param)


# ---------------------------------------------------------------- RMSNorm

def test_rmsnorm_constant_vector_closed_form():
    c, eps = 3.0, 1e-5
    x = np.full((1, 16), c)
    g = np.arange(1, 17, dtype=np.float64)
    y = oracle.rmsnorm(x, g, eps)
    np.testing.assert_allclose(y[0], c / math.sqrt(c * c + eps) * g, rtol=1e-15)


def test_rmsnorm_unit_gain_mean_square():
    x = RNG.standard_normal((5, 64))
    y = oracle.rmsnorm(x, np.ones(64), 1e-5)
    ms = (x * x).mean(-1)
    np.testing.assert_allclose((y * y).mean(-1), ms / (ms + 1e-5), rtol=1e-13)


def test_rmsnorm_matches_torch():
    x = RNG.standard_normal((7, 48))
    g = RNG.standard_normal(48)
    ref = F.rms_norm(torch.from_numpy(x), (48,), weight=torch.from_numpy(g), eps=1e-5).numpy()
    np.testing.assert_allclose(oracle.rmsnorm(x, g, 1e-5), ref, rtol=1e-13, atol=1e-14)


# ---------------------------------------------------------------- RoPE

def test_rope_position_zero_is_identity():
    x = RNG.standard_normal((3, 1, 16))
    np.testing.assert_array_equal(oracle.rope(x, np.array([0]), 10000.0), x)


def test_rope_hd2_is_plane_rotation():
    # hd = 2: theta_0 = 1, so position m rotates (a, b) by m radians
    x = np.array([[[1.0, 0.0], [0.0, 1.0], [0.6, 0.8]]])
    pos = np.array([1, 2, 5])
    y = oracle.rope(x, pos, 10000.0)
    exp = np.array([[math.cos(1), math.sin(1)],
                    [-math.sin(2), math.cos(2)],
                    [0.6 * math.cos(5) - 0.8 * math.sin(5), 0.8 * math.cos(5) + 0.6 * math.sin(5)]])
    np.testing.assert_allclose(y[0], exp, rtol=1e-14, atol=1e-15)


@pytest.mark.parametrize("hd", [8, 32, 64, 128])
def test_rope_matches_complex_definition(hd):
    x = RNG.standard_normal((2, 40, hd))
    pos = np.arange(40) * 7 + 3
    ref = rope_complex(torch.from_numpy(x), torch.from_numpy(pos), 10000.0).numpy()
    np.testing.assert_allclose(oracle.rope(x, pos, 10000.0), ref, rtol=1e-12, atol=1e-13)


def test_rope_preserves_norm_and_is_relative():
    hd = 64
    q, k = RNG.standard_normal(hd), RNG.standard_normal(hd)
    def r(v, m):
        return oracle.rope(v[None, None, :], np.array([m]), 10000.0)[0, 0]
    np.testing.assert_allclose(np.linalg.norm(r(q, 37)), np.linalg.norm(q), rtol=1e-13)
    d1 = r(q, 50) @ r(k, 20)
    d2 = r(q, 130) @ r(k, 100)
    np.testing.assert_allclose(d1, d2, rtol=1e-11)


# ---------------------------------------------------------------- attention

def test_attention_single_token_returns_value():
    q = RNG.standard_normal((2, 1, 8)); k = RNG.standard_normal((2, 1, 8)); v = RNG.standard_normal((2, 1, 8))
    np.testing.assert_allclose(oracle.causal_attention(q, k, v), v, rtol=1e-15)


def test_attention_uniform_keys_give_prefix_mean():
    T, hd = 9, 16
    q = RNG.standard_normal((3, T, hd))
    k = np.tile(RNG.standard_normal(hd), (1, T, 1))
    v = RNG.standard_normal((1, T, hd))
    out = oracle.causal_attention(q, k, v)
    exp = np.cumsum(v[0], axis=0) / np.arange(1, T + 1)[:, None]
    for j in range(3):
        np.testing.assert_allclose(out[j], exp, rtol=1e-12, atol=1e-14)


def test_attention_constant_values_are_reproduced():
    q = RNG.standard_normal((2, 12, 8)); k = RNG.standard_normal((2, 12, 8))
    v = np.ones((2, 12, 8)) * 2.5
    np.testing.assert_allclose(oracle.causal_attention(q, k, v), v, rtol=1e-14)


def test_gqa_equals_mha_with_repeated_kv():
    q = RNG.standard_normal((8, 10, 16)); k = RNG.standard_normal((2, 10, 16)); v = RNG.standard_normal((2, 10, 16))
    a = oracle.causal_attention(q, k, v)
    b = oracle.causal_attention(q, np.repeat(k, 4, axis=0), np.repeat(v, 4, axis=0))
    np.testing.assert_allclose(a, b, rtol=1e-14)


def test_attention_matches_torch_sdpa_fp64():
    q = RNG.standard_normal((6, 33, 32)); k = RNG.standard_normal((3, 33, 32)); v = RNG.standard_normal((3, 33, 32))
    ref = F.scaled_dot_product_attention(torch.from_numpy(q), torch.from_numpy(np.repeat(k, 2, 0)),
                                         torch.from_numpy(np.repeat(v, 2, 0)), is_causal=True).numpy()
    np.testing.assert_allclose(oracle.causal_attention(q, k, v), ref, rtol=1e-11, atol=1e-13)


# ---------------------------------------------------------------- activations

def test_gelu_values():
    assert oracle.gelu_erf(np.array([0.0]))[0] == 0.0
    # Phi(1) and Phi(-2) are standard normal CDF values
    np.testing.assert_allclose(oracle.gelu_erf(np.array([1.0, -2.0])),
                               [0.8413447460685429, -2.0 * 0.022750131948179195], rtol=1e-14)
    x = RNG.standard_normal(100) * 3
    ref = F.gelu(torch.from_numpy(x), approximate="none").numpy()
    np.testing.assert_allclose(oracle.gelu_erf(x), ref, rtol=1e-13, atol=1e-15)


def test_silu_values():
    x = RNG.standard_normal(100) * 4
    np.testing.assert_allclose(oracle.silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-13, atol=1e-15)
    assert oracle.silu(np.array([0.0]))[0] == 0.0


# ---------------------------------------------------------------- whole model

def _seqs(spec, n, lo=1, hi=20):
    r = np.random.default_rng(spec.weight_seed)
    return [r.integers(0, spec.vocab, size=int(r.integers(lo, hi + 1))) for _ in range(n)]


def test_forward_matches_torch_formulation(model):
    spec = model["spec"]
    seqs = _seqs(spec, 5)
    got = oracle.label_logits(model, seqs, (1, 2, 5))
    for i, s in enumerate(seqs):
        ref = forward_last_logits(model, s, (1, 2, 5)).numpy()
        np.testing.assert_allclose(got[i], ref, rtol=1e-10, atol=1e-12)


def test_causal_prefix_invariance(model):
    s = _seqs(model["spec"], 1, 25, 25)[0]
    full = forward_hidden(model, [s])[0]
    for m in (1, 7, 24):
        part = forward_hidden(model, [s[:m]])[0]
        np.testing.assert_allclose(part, full[:m], rtol=1e-12, atol=1e-13)


def test_batch_independence(model):
    a, b, c = _seqs(model["spec"], 3)
    together = oracle.label_logits(model, [a, b, c], (1, 2))
    for i, s in enumerate((a, b, c)):
        # equal up to the BLAS's own rounding of a stacked vs single-row product
        np.testing.assert_allclose(together[i], oracle.label_logits(model, [s], (1, 2))[0],
                                   rtol=1e-13, atol=1e-15)


def test_label_slice_equals_full_vocab(model):
    seqs = _seqs(model["spec"], 4)
    full = oracle.full_logits(model, seqs)
    sl = oracle.label_logits(model, seqs, (3, 1, 2))
    np.testing.assert_allclose(sl, full[:, [3, 1, 2]], rtol=1e-13, atol=1e-15)


def test_zero_output_projections_make_layers_identity(model):
    # With W_o = 0 and W_down = 0 every block adds nothing to the residual, so the
    # logits are the final norm of the last token's embedding times the head rows.
    spec = model["spec"]
    m = dict(model)
    m["layers"] = [dict(L, wo=np.zeros_like(L["wo"]), w_down=np.zeros_like(L["w_down"]))
                   for L in model["layers"]]
    s = _seqs(spec, 1)[0]
    e = as_f32(model["emb"][s[-1]]).astype(np.float64)
    hf = e / math.sqrt(float(np.mean(e * e)) + spec.norm_eps)
    exp = as_f32(model["lm_head"][[1, 2]]).astype(np.float64) @ hf
    np.testing.assert_allclose(oracle.label_logits(m, [s], (1, 2))[0], exp, rtol=1e-12)


def test_empty_sequence_has_zero_logits(model):
    lg = oracle.label_logits(model, [np.zeros(0, dtype=np.int64)], (1, 2))
    assert lg.shape == (1, 2) and np.all(lg == 0.0)


def test_truncated_stack_matches_zero_layers_closed_form(model):
    spec = model["spec"]
    s = _seqs(spec, 1)[0]
    e = as_f32(model["emb"][s[-1]]).astype(np.float64)
    hf = e / math.sqrt(float(np.mean(e * e)) + spec.norm_eps)
    exp = as_f32(model["lm_head"][[1, 2]]).astype(np.float64) @ hf
    np.testing.assert_allclose(oracle.label_logits(model, [s], (1, 2), n_layers=0)[0], exp, rtol=1e-12)
