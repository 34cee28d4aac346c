"""Brute-force pin for the oracle's decoder: torch CPU float64 library
routines (F.rms_norm, F.linear, F.scaled_dot_product_attention, F.silu) with
no KV cache -- every step recomputes the whole prefix.  RoPE is written as a
complex rotation (torch.polar / complex multiply), a different formulation
from the oracle's real 2x2 rotation.  bf16 rounding uses torch.frexp /
torch.round (half-to-even) / torch.ldexp.

This is test code; it shares nothing with the oracle or the GPU path.
"""
import numpy as np
import torch
import torch.nn.functional as F

import lede_inputs as li


def _to64(a, dtype):
    if dtype == "bf16":
        return torch.from_numpy(li.bf16_to_f32(a).astype(np.float64))
    return torch.from_numpy(a.astype(np.float64))


def round_bf16(x: torch.Tensor) -> torch.Tensor:
    m, e = torch.frexp(x)
    return torch.ldexp(torch.round(m * 256.0), e - 8)


def rope_complex(x: torch.Tensor, pos: torch.Tensor, base: float) -> torch.Tensor:
    """x [..., T, hd]; pos [T].  Pair (i, i + hd/2) is the complex number
    x_i + j x_{i+hd/2}, multiplied by exp(j * pos * base^(-2i/hd))."""
    hd = x.shape[-1]
    half = hd // 2
    i = torch.arange(half, dtype=torch.float64)
    ang = pos[:, None].to(torch.float64) * torch.pow(torch.tensor(base, dtype=torch.float64), -2.0 * i / hd)
    rot = torch.polar(torch.ones_like(ang), ang)
    z = torch.complex(x[..., :half], x[..., half:]) * rot
    return torch.cat([z.real, z.imag], dim=-1)


class TorchReference:
    def __init__(self, model, weights):
        self.m = model
        dt = model.dtype
        self.rnd = round_bf16 if dt == "bf16" else (lambda t: t)
        self.embed = _to64(weights["embed"], dt)
        self.head = _to64(weights["head"], dt)
        self.fnorm = _to64(weights["final_norm"], dt)
        self.layers = [{k: _to64(v, dt) for k, v in lw.items()} for lw in weights["layers"]]

    def hidden(self, tokens, l_end):
        m = self.m
        toks = torch.tensor(np.asarray(tokens), dtype=torch.long)
        T = len(toks)
        pos = torch.arange(T)
        x = self.embed[toks]
        nq, nkv, hd = m.n_heads, m.n_kv_heads, m.head_dim
        for lw in self.layers[:l_end]:
            u = self.rnd(F.rms_norm(x, (m.d_model,), lw["attn_norm"], eps=m.rms_eps))
            q = F.linear(u, lw["wq"]).view(T, nq, hd).transpose(0, 1)
            k = F.linear(u, lw["wk"]).view(T, nkv, hd).transpose(0, 1)
            v = F.linear(u, lw["wv"]).view(T, nkv, hd).transpose(0, 1)
            q = rope_complex(q, pos, m.rope_base)
            k = self.rnd(rope_complex(k, pos, m.rope_base))
            v = self.rnd(v)
            o = F.scaled_dot_product_attention(q[None], k[None], v[None], is_causal=True,
                                               enable_gqa=(nq != nkv))[0]
            o = self.rnd(o.transpose(0, 1).reshape(T, nq * hd))
            x = x + F.linear(o, lw["wo"])
            n = self.rnd(F.rms_norm(x, (m.d_model,), lw["ffn_norm"], eps=m.rms_eps))
            a = self.rnd(F.silu(F.linear(n, lw["wg"])) * F.linear(n, lw["wu"]))
            x = x + F.linear(a, lw["wd"])
        return x

    def logits(self, tokens, l_end=None):
        l_end = self.m.n_layers if l_end is None else l_end
        x = self.hidden(tokens, l_end)
        u = self.rnd(F.rms_norm(x, (self.m.d_model,), self.fnorm, eps=self.m.rms_eps))
        return F.linear(u, self.head)

    def greedy(self, prompt, n_gen):
        seq = list(int(t) for t in prompt)
        out, rows = [], []
        for _ in range(n_gen):
            z = self.logits(seq)[-1]
            t = int(torch.argmax(z))
            out.append(t)
            rows.append(z.numpy())
            seq.append(t)
        return out, rows
