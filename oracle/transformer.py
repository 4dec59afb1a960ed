"""Decoder-only transformer forward of the oracle, per sequence, in fp64.
Test infrastructure only (see the package docstring).

The paper's semantic operator runs a causal LM over each row's text and reads
the logits at the last position (Figure 2, Section 3.1).  The architecture is
the random-init Llama-style decoder of the workloads (the paper's Gemma-2B is
not available): pre-norm RMSNorm, rotary position embedding on q and k
(rotate-half pairing of dimension i with i + hd/2), causal softmax attention
with grouped K/V heads, an SwiGLU (or exact-erf GELU) feed-forward block, a
final RMSNorm and an untied LM head.  Each sequence is processed alone: no
packing, no padding, positions start at 0.

Weights arrive exactly as stored (fp32, or bf16 bit patterns) and are widened
to fp64; all arithmetic is fp64.
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf

from synth.gen import as_f32


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x**2) + eps) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotary embedding of head vectors x[..., t, hd] at positions pos[t].

    Dimension i is paired with i + hd/2 and the pair is rotated by the angle
    pos * theta**(-2i/hd)."""
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=np.float64) / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """softmax(q k^T / sqrt(hd)) v with key s visible to query t iff s <= t.

    q: [n_q, T, hd]; k, v: [n_kv, T, hd]; query head j reads kv head
    j // (n_q / n_kv)."""
    n_q, T, hd = q.shape
    n_kv = k.shape[0]
    rep = n_q // n_kv
    out = np.empty_like(q)
    mask = np.tril(np.ones((T, T), dtype=bool))
    for j in range(n_q):
        kv = j // rep
        s = (q[j] @ k[kv].T) / np.sqrt(hd)
        s = np.where(mask, s, -np.inf)
        s = s - s.max(axis=-1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=-1, keepdims=True)
        out[j] = p @ v[kv]
    return out


def gelu_erf(x: np.ndarray) -> np.ndarray:
    """Exact GELU: x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2))."""
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


class Weights64:
    """fp64 views of one model's weights, widened one layer at a time."""

    def __init__(self, model: dict):
        self.model = model
        self.spec = model["spec"]

    @staticmethod
    def w(t: np.ndarray) -> np.ndarray:
        return as_f32(t).astype(np.float64)

    def layer(self, l: int) -> dict:
        return {k: self.w(v) for k, v in self.model["layers"][l].items()}


def _layer(x: np.ndarray, W: dict, spec) -> np.ndarray:
    T = x.shape[0]
    hd, nq, nkv = spec.head_dim, spec.n_heads, spec.n_kv_heads
    pos = np.arange(T)
    h = rmsnorm(x, W["attn_norm"], spec.norm_eps)
    q = (h @ W["wq"].T).reshape(T, nq, hd).transpose(1, 0, 2)
    k = (h @ W["wk"].T).reshape(T, nkv, hd).transpose(1, 0, 2)
    v = (h @ W["wv"].T).reshape(T, nkv, hd).transpose(1, 0, 2)
    q = rope(q, pos, spec.rope_theta)
    k = rope(k, pos, spec.rope_theta)
    a = causal_attention(q, k, v).transpose(1, 0, 2).reshape(T, nq * hd)
    x = x + a @ W["wo"].T
    h2 = rmsnorm(x, W["ffn_norm"], spec.norm_eps)
    if spec.act == "swiglu":
        f = silu(h2 @ W["w_gate"].T) * (h2 @ W["w_up"].T)
    else:
        f = gelu_erf(h2 @ W["w_gate"].T)
    return x + f @ W["w_down"].T


def forward_hidden(model: dict, seqs: list, n_layers: int | None = None) -> list:
    """Residual stream after the last layer, [len, d] per sequence (before the
    final norm).  The layer loop is outermost so each layer's weights are
    widened once; every sequence is still computed on its own."""
    spec = model["spec"]
    W = Weights64(model)
    emb = model["emb"]
    xs = [as_f32(emb[np.asarray(s, dtype=np.int64)]).astype(np.float64) for s in seqs]
    L = len(model["layers"]) if n_layers is None else n_layers
    for l in range(L):
        Wl = W.layer(l)
        xs = [_layer(x, Wl, spec) if len(x) else x for x in xs]
    return xs


def _last_normed(model: dict, xs: list) -> np.ndarray:
    spec = model["spec"]
    g = Weights64.w(model["final_norm"])
    if not xs:
        return np.zeros((0, spec.d_model))
    return np.stack([rmsnorm(x[-1], g, spec.norm_eps) if len(x) else np.zeros(spec.d_model) for x in xs])


def label_logits(model: dict, seqs: list, labels, n_layers: int | None = None) -> np.ndarray:
    """Last-position logits of the label tokens only, [n_seq, K] (Figure 2:
    logits[:, -1, :] then the Yes / No columns).  ``n_layers`` truncates the
    layer stack (diagnostics).  An empty sequence has all-zero logits."""
    hf = _last_normed(model, forward_hidden(model, seqs, n_layers))
    rows = Weights64.w(model["lm_head"][np.asarray(labels, dtype=np.int64)])
    return hf @ rows.T


def full_logits(model: dict, seqs: list, n_layers: int | None = None) -> np.ndarray:
    """Last-position logits over the whole vocabulary, [n_seq, V]."""
    hf = _last_normed(model, forward_hidden(model, seqs, n_layers))
    return hf @ Weights64.w(model["lm_head"]).T
