"""A second, independent formulation of the decoder forward in torch-CPU fp64
library ops, used only to pin the oracle (never the device path).

It differs from the oracle's own arithmetic on purpose: torch's
``F.rms_norm``, ``F.linear``, ``F.scaled_dot_product_attention`` (causal, K/V
heads repeated for grouped attention), complex multiplication for the rotary
embedding, and ``F.silu`` / ``F.gelu(approximate="none")``.
"""
import numpy as np
import torch
import torch.nn.functional as F

from synth.gen import as_f32


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(as_f32(a)).astype(np.float64))


def rope_complex(x: torch.Tensor, pos: torch.Tensor, theta: float) -> torch.Tensor:
    """Rotary embedding as multiplication of z_i = x_i + i x_{i+hd/2} by exp(i pos theta_i)."""
    hd = x.shape[-1]
    half = hd // 2
    freqs = theta ** (-torch.arange(0, hd, 2, dtype=torch.float64) / hd)
    ang = pos.to(torch.float64)[:, None] * freqs[None, :]
    z = torch.complex(x[..., :half], x[..., half:]) * torch.polar(torch.ones_like(ang), ang)
    return torch.cat([z.real, z.imag], dim=-1)


def forward_last_logits(model: dict, seq, labels=None) -> torch.Tensor:
    spec = model["spec"]
    d, hd, nq, nkv = spec.d_model, spec.head_dim, spec.n_heads, spec.n_kv_heads
    tok = torch.as_tensor(np.asarray(seq, dtype=np.int64))
    x = _t(model["emb"])[tok]
    T = x.shape[0]
    pos = torch.arange(T)
    for L in model["layers"]:
        h = F.rms_norm(x, (d,), weight=_t(L["attn_norm"]), eps=spec.norm_eps)
        q = F.linear(h, _t(L["wq"])).view(T, nq, hd).transpose(0, 1)
        k = F.linear(h, _t(L["wk"])).view(T, nkv, hd).transpose(0, 1)
        v = F.linear(h, _t(L["wv"])).view(T, nkv, hd).transpose(0, 1)
        q = rope_complex(q, pos, spec.rope_theta)
        k = rope_complex(k, pos, spec.rope_theta)
        k = k.repeat_interleave(nq // nkv, dim=0)
        v = v.repeat_interleave(nq // nkv, dim=0)
        a = F.scaled_dot_product_attention(q, k, v, is_causal=True)
        x = x + F.linear(a.transpose(0, 1).reshape(T, nq * hd), _t(L["wo"]))
        h2 = F.rms_norm(x, (d,), weight=_t(L["ffn_norm"]), eps=spec.norm_eps)
        if spec.act == "swiglu":
            f = F.silu(F.linear(h2, _t(L["w_gate"]))) * F.linear(h2, _t(L["w_up"]))
        else:
            f = F.gelu(F.linear(h2, _t(L["w_gate"])), approximate="none")
        x = x + F.linear(f, _t(L["w_down"]))
    hf = F.rms_norm(x[-1], (d,), weight=_t(model["final_norm"]), eps=spec.norm_eps)
    W = _t(model["lm_head"])
    if labels is not None:
        W = W[torch.as_tensor(list(labels))]
    return F.linear(hf, W)
