"""AI_TRANSFORM (generation) and the LIKE filter over generated tokens, in
fp64, per sequence.  Test infrastructure only (see the package docstring).

Table 1 maps AI_TRANSFORM to a causal-LM forward pass with generative
decoding whose output is masked with a pad id; Section 4 (Q3, Q5) filters and
counts rows by a LIKE pattern over the generated text.  The paper names no
decoding rule; the readings taken here:

* greedy decoding: each new token is the argmax of the last position's
  logits over the whole vocabulary, ties to the lowest token id;
* generation stops after the end-of-sequence token (it is kept as the last
  generated token); every later slot holds the pad id;
* an empty prompt has all-zero logits, so its first token is 0;
* ``col LIKE '%p%'`` holds when the pattern's tokens occur contiguously in
  the generated tokens up to the end of generation (token-level matching:
  there is no tokenizer here, patterns are token ids).
"""
from __future__ import annotations

import numpy as np

from .transformer import Weights64, forward_hidden, rmsnorm


def position_logits(model: dict, seq) -> np.ndarray:
    """Logits over the vocabulary at every position of one sequence, [len, V]."""
    spec = model["spec"]
    x = forward_hidden(model, [np.asarray(seq, dtype=np.int64)])[0]
    if len(x) == 0:
        return np.zeros((0, spec.vocab))
    hf = rmsnorm(x, Weights64.w(model["final_norm"]), spec.norm_eps)
    return hf @ Weights64.w(model["lm_head"]).T


def greedy_generate(model: dict, seq, n_new: int, eos: int = -1, pad: int = 0) -> np.ndarray:
    """n_new generated tokens after ``seq`` (see the module readings)."""
    out = np.full(n_new, pad, dtype=np.int64)
    cur = [int(t) for t in np.asarray(seq, dtype=np.int64)]
    for k in range(n_new):
        if cur:
            lg = position_logits(model, cur)[-1]
        else:
            lg = np.zeros(model["spec"].vocab)
        t = int(np.argmax(lg))          # first index of the maximum
        out[k] = t
        cur.append(t)
        if t == eos:
            break
    return out


def generated_length(gen, eos: int) -> int:
    """Tokens up to and including the first end-of-sequence token."""
    g = np.asarray(gen)
    hit = np.flatnonzero(g == eos) if eos >= 0 else np.zeros(0, dtype=np.int64)
    return int(hit[0]) + 1 if len(hit) else len(g)


def like_tokens(gen, pattern, eos: int = -1) -> bool:
    """``gen LIKE '%pattern%'`` over token ids, within the generated length."""
    g = [int(t) for t in np.asarray(gen)[:generated_length(gen, eos)]]
    p = [int(t) for t in pattern]
    if not p:
        return True
    return any(g[i:i + len(p)] == p for i in range(len(g) - len(p) + 1))
