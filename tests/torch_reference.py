"""A second, structurally different formulation of the decoder, built from
torch library routines in float64 on the CPU, used only to pin the oracle.

The oracle loops one token row at a time; this module processes a chunk of T
tokens at once in matrix form: ``torch.matmul`` for every projection,
``torch.nn.functional.rms_norm``, ``scaled_dot_product_attention`` with an
explicit causal mask over [cached prefix | chunk], ``torch.nn.functional.silu``
and ``torch.softmax`` / ``torch.topk`` for routing.  The model's storage
points are applied with torch's own bf16 / fp32 casts.  A dropped term, a
transposed operand, a wrong rotation sign or a missing rounding point in the
oracle would make the two disagree far beyond fp64 rounding noise.
"""
from __future__ import annotations

import torch
import torch.nn.functional as F

f64 = torch.float64


def _bf(t: torch.Tensor) -> torch.Tensor:
    """float64 -> nearest bf16 (ties to even), returned as float64.

    torch casts float64 to bfloat16 through float32, which double-rounds:
    about one value in 2^16 lands on a bf16 tie after the first rounding.
    Rounding to float32 with round-to-odd first (truncate, then set the last
    bit if inexact) keeps the second rounding correct, because float32 has
    more than two extra significand bits over bf16."""
    f = t.to(torch.float32)
    inexact = f.to(f64) != t
    away = f.to(f64).abs() > t.abs()
    f = torch.where(inexact & away, torch.nextafter(f, torch.zeros_like(f)), f)
    b = f.view(torch.int32)
    b = torch.where(inexact, b | 1, b)
    return b.view(torch.float32).to(torch.bfloat16).to(f64)


def _w(t: torch.Tensor) -> torch.Tensor:
    return t.to(f64)


def _rope(x: torch.Tensor, pos: torch.Tensor, theta: float) -> torch.Tensor:
    """x [T, n, d] rotated by angle pos * theta^(-2i/d) on the pair (i, i+d/2)."""
    d = x.shape[-1]
    half = d // 2
    i = torch.arange(half, dtype=f64)
    inv = torch.pow(torch.tensor(theta, dtype=f64), -2.0 * i / d)
    ang = pos.to(f64)[:, None] * inv[None, :]
    c, s = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return torch.cat([x1 * c - x2 * s, x2 * c + x1 * s], dim=-1)


def _swiglu(h, wgu, wd, Fd):
    gu = h @ _w(wgu).T
    g, u = _bf(gu[:, :Fd]), _bf(gu[:, Fd:])
    a = _bf(F.silu(g) * u)
    return a @ _w(wd).T


def forward_chunk(cfg: dict, W, tokens, start: int, k_prefix, v_prefix, force=None, routing=None):
    """Run tokens [T] at positions start..start+T-1 of one request.

    W: workload.Weights (bf16 tensors).  k_prefix, v_prefix: per layer bf16
    [nkv, start, d] cache of the positions before the chunk.
    Mixture of experts: force ([L][T][k], optional) replaces each row's top-k
    expert set (weights: the softmax renormalised over the given set);
    routing (a list, optional) receives per layer (router logits [T, E],
    torch.topk ids [T, k]).
    Returns (logits [T, V] float64, k_new, v_new: per layer bf16 [nkv, T, d]).
    """
    H, d = cfg["hidden"], cfg["head_dim"]
    nq, nkv = cfg["n_heads"], cfg["n_kv_heads"]
    eps, theta = cfg["rms_eps"], cfg["rope_theta"]
    T = len(tokens)
    pos = torch.arange(start, start + T)
    x = W.embed[torch.as_tensor(tokens, dtype=torch.long)].to(torch.float32)
    ks, vs = [], []
    # mask[i, j]: query at start+i may see key j (prefix keys 0..start-1, then chunk keys)
    allowed = torch.arange(start + T)[None, :] <= pos[:, None]
    for l in range(cfg["n_layers"]):
        h = _bf(F.rms_norm(x.to(f64), (H,), weight=_w(W.attn_norm[l]), eps=eps))
        qkv = _bf(h @ _w(W.w_qkv[l]).T)
        q = qkv[:, : nq * d].reshape(T, nq, d)
        k = qkv[:, nq * d:(nq + nkv) * d].reshape(T, nkv, d)
        v = qkv[:, (nq + nkv) * d:].reshape(T, nkv, d)
        q, k = _bf(_rope(q, pos, theta)), _bf(_rope(k, pos, theta))
        ks.append(k.transpose(0, 1).to(torch.bfloat16))
        vs.append(v.transpose(0, 1).to(torch.bfloat16))
        K = torch.cat([k_prefix[l].to(f64), k.transpose(0, 1)], dim=1)   # [nkv, S, d]
        V = torch.cat([v_prefix[l].to(f64), v.transpose(0, 1)], dim=1)
        K = K.repeat_interleave(nq // nkv, dim=0)
        V = V.repeat_interleave(nq // nkv, dim=0)
        o = F.scaled_dot_product_attention(q.transpose(0, 1), K, V, attn_mask=allowed)
        o = _bf(o.transpose(0, 1).reshape(T, nq * d))
        x = (x.to(f64) + o @ _w(W.w_o[l]).T).to(torch.float32)
        h = _bf(F.rms_norm(x.to(f64), (H,), weight=_w(W.mlp_norm[l]), eps=eps))
        if cfg["n_experts"] == 0:
            y = _swiglu(h, W.w_gate_up[l], W.w_down[l], cfg["ffn"])
        else:
            E, K_, Fe = cfg["n_experts"], cfg["top_k"], cfg["expert_ffn"]
            rl = h @ _w(W.w_router[l]).T
            p = torch.softmax(rl, dim=-1)
            top_p, top_e = torch.topk(p, K_, dim=-1)
            if routing is not None:
                routing.append((rl, top_e))
            if force is not None:
                top_e = torch.as_tensor(force[l], dtype=torch.long).reshape(T, K_)
                top_p = torch.gather(p, 1, top_e)
            wts = top_p / top_p.sum(-1, keepdim=True)
            y = torch.zeros(T, H, dtype=f64)
            for t in range(T):
                for r in range(K_):
                    e = int(top_e[t, r])
                    y[t] += wts[t, r] * _swiglu(h[t:t + 1], W.w_exp_gate_up[l][e],
                                                W.w_exp_down[l][e], Fe)[0]
        x = (x.to(f64) + y).to(torch.float32)
    h = _bf(F.rms_norm(x.to(f64), (H,), weight=_w(W.final_norm), eps=eps))
    return h @ _w(W.lm_head).T, ks, vs
