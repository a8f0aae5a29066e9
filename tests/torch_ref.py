"""A float64 decoder built from PyTorch library primitives, used only to pin the oracle.

It is a different formulation from the oracle's: the whole sequence at once
with F.scaled_dot_product_attention(is_causal=True) instead of an incremental
KV cache, F.rms_norm, F.silu, and the rotary embedding as a complex
multiplication by exp(i * pos * theta) (torch.polar) instead of the
rotate-half formula.

Rows [0, n_full) run the full model; rows [n_full, T) run with the skip mask
z, which is how a draft sees a cache whose prefix the full model wrote (the
suffix attends to the prefix and, in non-skipped attention sublayers, to
earlier suffix rows).
"""

from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as F


def forward(cfg, w64, tokens, skip=None, n_full=None, start_pos=0, hide_key=None, kv_out=None):
    """Logits [T, vocab] (float64) of a causal forward over tokens.  hide_key
    (a row index) removes that key from every other row's attention, a planted
    mistake for measuring how far logits move when attention loses a key.
    kv_out (a list): receives one (k, v) pair per layer, float64 arrays
    [T, n_kv_heads, head_dim], k rotated, both rounded to bf16 values for a
    bf16 model (what a KV cache holds)."""
    tok = torch.as_tensor(np.asarray(tokens, dtype=np.int64))
    T = tok.numel()
    n_full = T if (skip is None or n_full is None) else n_full
    W = {k: torch.as_tensor(v) for k, v in w64.items()}
    d, H, KVH, dh, Fd = cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.ffn_dim
    half = dh // 2
    grp = H // KVH

    pos = torch.arange(start_pos, start_pos + T, dtype=torch.float64)
    inv_freq = cfg.rope_base ** (-(torch.arange(0, dh, 2, dtype=torch.float64) / dh))
    ang = pos[:, None] * inv_freq[None, :]
    rot = torch.polar(torch.ones_like(ang), ang)  # [T, dh/2] complex128

    def rope(x):  # [T, nh, dh]; element i pairs with i + dh/2 as a complex number
        xc = torch.complex(x[..., :half], x[..., half:]) * rot[:, None, :]
        return torch.cat([xc.real, xc.imag], dim=-1)

    row_full = torch.zeros(T, dtype=torch.bool)
    row_full[:n_full] = True

    def applies(sub):  # which rows run sublayer `sub`
        if skip is None or not skip[sub]:
            return torch.ones(T, dtype=torch.bool)
        return row_full

    h = F.embedding(tok, W["tok_emb"])
    for l in range(cfg.n_layers):
        a = applies(2 * l)
        if a.any():
            u = F.rms_norm(h, (d,), W[f"layers.{l}.attn_norm"], eps=cfg.rms_eps)
            qkv = F.linear(u, W[f"layers.{l}.w_qkv"])
            q = rope(qkv[:, : H * dh].reshape(T, H, dh))
            k = rope(qkv[:, H * dh: (H + KVH) * dh].reshape(T, KVH, dh))
            v = qkv[:, (H + KVH) * dh:].reshape(T, KVH, dh)
            if cfg.dtype == "bf16":  # the KV cache of a bf16 model holds bf16 values
                k = k.to(torch.bfloat16).to(torch.float64)
                v = v.to(torch.bfloat16).to(torch.float64)
            if kv_out is not None:
                kv_out.append((k.numpy().copy(), v.numpy().copy()))
            k = k.repeat_interleave(grp, dim=1)
            v = v.repeat_interleave(grp, dim=1)
            if hide_key is None:
                o = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                                   is_causal=True)
            else:
                allow = torch.ones(T, T, dtype=torch.bool).tril()
                allow[:, hide_key] = False
                allow[hide_key, hide_key] = True
                o = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                                   attn_mask=allow)
            o = o.transpose(0, 1).reshape(T, H * dh)
            h = h + a[:, None] * F.linear(o, W[f"layers.{l}.w_o"])
        m = applies(2 * l + 1)
        if m.any():
            u = F.rms_norm(h, (d,), W[f"layers.{l}.mlp_norm"], eps=cfg.rms_eps)
            gu = F.linear(u, W[f"layers.{l}.w_gate_up"])
            y = F.linear(F.silu(gu[:, :Fd]) * gu[:, Fd:], W[f"layers.{l}.w_down"])
            h = h + m[:, None] * y
    u = F.rms_norm(h, (d,), W["final_norm"], eps=cfg.rms_eps)
    return F.linear(u, W["lm_head"]).numpy()
