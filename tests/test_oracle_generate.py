"""Pins of the oracle's generation and token LIKE (oracle/generate.py):
an independent torch-fp64 greedy loop, the teacher-forcing identity of a
single forward over prompt + generation, end-of-sequence handling, the empty
prompt, and brute-force string containment for LIKE."""
import numpy as np
import pytest
import torch

from oracle.generate import generated_length, greedy_generate, like_tokens, position_logits
from oracle.transformer import full_logits
from synth.configs import ModelSpec
from synth.gen import make_model
from tests._torch_ref import forward_last_logits

SMALL = [
    ModelSpec(n_layers=2, d_model=64, n_heads=8, n_kv_heads=2, d_ff=96, vocab=97, act="swiglu", dtype="bf16",
              weight_seed=81, init_std=0.3),
    ModelSpec(n_layers=2, d_model=32, n_heads=4, n_kv_heads=4, d_ff=48, vocab=61, act="gelu", dtype="f32",
              weight_seed=82, init_std=0.3),
]


@pytest.fixture(scope="module", params=SMALL, ids=["swiglu-gqa-bf16", "gelu-mha-f32"])
def model(request):
    return make_model(request.param)


def prompts(vocab, n=4, seed=5):
    r = np.random.default_rng(seed)
    return [r.integers(0, vocab, int(r.integers(1, 9))) for _ in range(n)]


def torch_greedy(model, seq, n_new):
    """Greedy loop over the independent torch formulation (torch.argmax takes
    the first maximal index)."""
    cur = [int(t) for t in seq]
    out = []
    for _ in range(n_new):
        t = int(torch.argmax(forward_last_logits(model, cur)))
        out.append(t)
        cur.append(t)
    return np.array(out)


def test_greedy_equals_independent_torch_loop(model):
    for seq in prompts(model["spec"].vocab):
        np.testing.assert_array_equal(greedy_generate(model, seq, 6), torch_greedy(model, seq, 6))


def test_one_forward_reproduces_every_step(model):
    """Position t's logits over prompt + generation are the step logits that
    chose token t + 1, so one forward's argmax per position is the generation."""
    for seq in prompts(model["spec"].vocab, seed=6):
        gen = greedy_generate(model, seq, 7)
        lg = position_logits(model, np.concatenate([seq, gen[:-1]]))
        np.testing.assert_array_equal(lg[len(seq) - 1:].argmax(axis=1), gen)


def test_position_logits_last_row_is_the_last_position_logits(model):
    seq = prompts(model["spec"].vocab, n=1, seed=7)[0]
    np.testing.assert_allclose(position_logits(model, seq)[-1], full_logits(model, [seq])[0], rtol=0, atol=1e-12)


def test_end_of_sequence_stops_and_pads(model):
    seq = prompts(model["spec"].vocab, n=1, seed=8)[0]
    free = greedy_generate(model, seq, 8)
    eos = int(free[2])
    k = int(np.flatnonzero(free == eos)[0])       # first occurrence ends the generation
    got = greedy_generate(model, seq, 8, eos=eos, pad=-7)
    np.testing.assert_array_equal(got[:k + 1], free[:k + 1])
    assert np.all(got[k + 1:] == -7)
    assert generated_length(got, eos) == k + 1


def test_empty_prompt_starts_at_token_zero(model):
    g = greedy_generate(model, [], 4)
    assert g[0] == 0
    np.testing.assert_array_equal(g[1:], greedy_generate(model, [0], 3))


def _as_text(tokens):
    return "".join(f"<{int(t)}>" for t in tokens)


def test_like_equals_string_containment():
    r = np.random.default_rng(11)
    for _ in range(400):
        G = int(r.integers(1, 14))
        gen = r.integers(0, 5, G)
        eos = int(r.integers(-1, 5))
        pat = r.integers(0, 5, int(r.integers(1, 4)))
        n = generated_length(gen, eos)
        assert like_tokens(gen, pat, eos) == (_as_text(pat) in _as_text(gen[:n]))


def test_like_edges():
    gen = np.array([4, 9, 9, 2, 7, 3])
    assert like_tokens(gen, [4])                 # at the start
    assert like_tokens(gen, [7, 3])              # at the end
    assert not like_tokens(gen, [9, 2, 8])
    assert not like_tokens(gen, [7, 3], eos=2)   # after the end of generation
    assert like_tokens(gen, [9, 2], eos=2)       # the end token itself belongs to the output
    assert not like_tokens(gen, [4, 9, 9, 2, 7, 3, 1])
    assert like_tokens(gen, [])


def test_ties_go_to_the_lowest_token_id(model):
    """With an all-zero LM head every logit is exactly 0 at each step: the
    first token id wins every time."""
    m = dict(model)
    m["lm_head"] = np.zeros_like(np.asarray(model["lm_head"]))
    seq = prompts(model["spec"].vocab, n=1, seed=9)[0]
    np.testing.assert_array_equal(greedy_generate(m, seq, 4), np.zeros(4, dtype=np.int64))
