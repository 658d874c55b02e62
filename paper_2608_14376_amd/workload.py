"""Seeded synthetic workloads: model shapes, random-init weights, KV contents
and padded decode batches.

This module produces inputs only.  It holds none of the decode step's
arithmetic, so both the HIP path and the CPU oracle may consume what it makes.

The paper evaluates on trained models and on the BurstGPT / Blazedit traces
(Sec. V, "Experimental Setup"); neither is available here, so seeded random
tensors of the evaluated model families' shapes and seeded length
distributions stand in for them.

Every tensor is drawn from its own generator, seeded from (model seed, tensor
index), so a subset of layers can be regenerated bit-identically without the
rest.  Matrices are N(0, 0.02) drawn in fp32 and rounded to bf16 (round to
nearest even); RMSNorm gains are 1 + N(0, 0.02); MoE router rows are
N(0, 1/H) so that router logits are about N(0, 1) at unit-RMS input.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np
import torch

# --------------------------------------------------------------------------
# Model shapes
# --------------------------------------------------------------------------

CONFIGS = {
    # two-layer GQA decoder used for exhaustive invariance and oracle parity
    "tiny": dict(n_layers=2, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64, ffn=688,
                 vocab=1024, n_experts=0, top_k=0, expert_ffn=0, rms_eps=1e-6, rope_theta=10000.0),
    # 8B-class dense decoder (Qwen3-8B family shape)
    "8b": dict(n_layers=36, hidden=4096, n_heads=32, n_kv_heads=8, head_dim=128, ffn=12288,
               vocab=151936, n_experts=0, top_k=0, expert_ffn=0, rms_eps=1e-6, rope_theta=1e6),
    # 32B-class dense decoder (Qwen3-32B family shape); nq*d = 8192 != hidden
    "32b": dict(n_layers=64, hidden=5120, n_heads=64, n_kv_heads=8, head_dim=128, ffn=27648,
                vocab=152064, n_experts=0, top_k=0, expert_ffn=0, rms_eps=1e-6, rope_theta=1e6),
    # mixture-of-experts decoder (Qwen3-30B-A3B family shape)
    "moe": dict(n_layers=48, hidden=2048, n_heads=32, n_kv_heads=4, head_dim=128, ffn=0,
                vocab=151936, n_experts=128, top_k=8, expert_ffn=768, rms_eps=1e-6, rope_theta=1e6),
    # two-layer decoder with the 8B family's head geometry (d = 128, 4 query
    # heads per KV head), for oracle parity of the d = 128 kernels
    "small128": dict(n_layers=2, hidden=512, n_heads=8, n_kv_heads=2, head_dim=128, ffn=1024,
                     vocab=2048, n_experts=0, top_k=0, expert_ffn=0, rms_eps=1e-6, rope_theta=1e6),
    # small mixture-of-experts decoder for oracle parity
    "tiny_moe": dict(n_layers=2, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64, ffn=0,
                     vocab=1024, n_experts=16, top_k=4, expert_ffn=96, rms_eps=1e-6,
                     rope_theta=10000.0),
    # small mixture-of-experts decoder whose expert width is a multiple of 64
    # (the packed expert copies with the fused SwiGLU, as at full size)
    "small_moe": dict(n_layers=2, hidden=512, n_heads=8, n_kv_heads=2, head_dim=128, ffn=0,
                      vocab=1024, n_experts=16, top_k=4, expert_ffn=128, rms_eps=1e-6,
                      rope_theta=1e6),
}


def config(name: str, **over) -> dict:
    c = dict(CONFIGS[name])
    c.update(over)
    return c


def qkv_rows(c: dict) -> int:
    return (c["n_heads"] + 2 * c["n_kv_heads"]) * c["head_dim"]


def streamed_weight_params(c: dict) -> int:
    """Parameters read from HBM by one decode step at full expert coverage:
    every layer matrix plus lm_head (the embedding is gathered, not streamed)."""
    H, d, nq = c["hidden"], c["head_dim"], c["n_heads"]
    per = H * qkv_rows(c) + H * nq * d + 2 * H
    if c["n_experts"]:
        per += c["n_experts"] * H + c["n_experts"] * 3 * H * c["expert_ffn"]
    else:
        per += 3 * H * c["ffn"]
    return c["n_layers"] * per + c["vocab"] * H + H


def kv_bytes_per_token(c: dict) -> int:
    """K and V bytes of one token over all layers (bf16)."""
    return c["n_layers"] * 2 * c["n_kv_heads"] * c["head_dim"] * 2


# --------------------------------------------------------------------------
# Weights
# --------------------------------------------------------------------------

def _gen(seed: int, idx: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1_000_003 + idx * 7919 + 17) % (2**63 - 1))
    return g


def _normal_bf16(shape, std, seed, idx, device, mean=0.0):
    g = _gen(seed, idx, device)
    t = torch.randn(shape, generator=g, dtype=torch.float32, device=device)
    t.mul_(std)
    if mean:
        t.add_(mean)
    return t.to(torch.bfloat16)


@dataclass
class Weights:
    """bf16 torch tensors in PyTorch Linear layout [out, in]."""
    cfg: dict
    embed: torch.Tensor
    final_norm: torch.Tensor
    lm_head: torch.Tensor
    attn_norm: list
    w_qkv: list
    w_o: list
    mlp_norm: list
    w_gate_up: list
    w_down: list
    w_router: list
    w_exp_gate_up: list
    w_exp_down: list

    def layer_tensors(self):
        for lst in (self.attn_norm, self.w_qkv, self.w_o, self.mlp_norm, self.w_gate_up,
                    self.w_down, self.w_router, self.w_exp_gate_up, self.w_exp_down):
            yield from lst


def make_weights(c: dict, seed: int = 0, device="cpu", layers=None, std: float = 0.02) -> Weights:
    """Random-init weights.  Tensor index order: embed 0, final_norm 1,
    lm_head 2, then per layer l at 16 + 16 l: attn_norm, w_qkv, w_o, mlp_norm,
    w_gate_up (gate rows first), w_down, w_router, w_exp_gate_up, w_exp_down.
    `layers` (an iterable of layer ids) limits which layers are drawn; the
    drawn ones are bit-identical to a full draw."""
    H, d, nq, F = c["hidden"], c["head_dim"], c["n_heads"], c["ffn"]
    E, Fe, V = c["n_experts"], c["expert_ffn"], c["vocab"]
    L = c["n_layers"]
    layers = range(L) if layers is None else list(layers)
    w = Weights(c, _normal_bf16((V, H), std, seed, 0, device),
                _normal_bf16((H,), std, seed, 1, device, mean=1.0),
                _normal_bf16((V, H), std, seed, 2, device), [], [], [], [], [], [], [], [], [])
    for l in layers:
        b = 16 + 16 * l
        w.attn_norm.append(_normal_bf16((H,), std, seed, b + 0, device, mean=1.0))
        w.w_qkv.append(_normal_bf16((qkv_rows(c), H), std, seed, b + 1, device))
        w.w_o.append(_normal_bf16((H, nq * d), std, seed, b + 2, device))
        w.mlp_norm.append(_normal_bf16((H,), std, seed, b + 3, device, mean=1.0))
        if E:
            w.w_router.append(_normal_bf16((E, H), 1.0 / math.sqrt(H), seed, b + 6, device))
            w.w_exp_gate_up.append(_normal_bf16((E, 2 * Fe, H), std, seed, b + 7, device))
            w.w_exp_down.append(_normal_bf16((E, H, Fe), std, seed, b + 8, device))
        else:
            w.w_gate_up.append(_normal_bf16((2 * F, H), std, seed, b + 4, device))
            w.w_down.append(_normal_bf16((H, F), std, seed, b + 5, device))
    return w


def bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> numpy uint16 bit patterns (host copy)."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def from_bits(a: np.ndarray, device="cpu") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)


# --------------------------------------------------------------------------
# Decode batches and KV caches
# --------------------------------------------------------------------------

@dataclass
class Batch:
    tokens: np.ndarray      # int32 [B]
    valid: np.ndarray       # uint8 [B]
    seq_lens: np.ndarray    # int32 [B]: tokens already cached = new token's position


def make_batch(B: int, vocab: int, seed: int, len_lo: int, len_hi: int,
               live_frac=(0.25, 1.0), n_live: int | None = None,
               log_uniform: bool = False) -> Batch:
    """A padded decode batch: n_live = clamp(round(f B), 1, B) with f uniform
    in live_frac, live slots a seeded random subset, lengths uniform integers
    in [len_lo, len_hi] (or log-uniform).  Padding rows carry arbitrary
    (seeded) garbage tokens and lengths, which the step must ignore."""
    r = np.random.default_rng(seed)
    if n_live is None:
        f = r.uniform(*live_frac)
        n_live = int(min(max(round(f * B), 1), B))
    live = r.permutation(B)[:n_live]
    valid = np.zeros(B, np.uint8)
    valid[live] = 1
    if log_uniform:
        lens = np.exp(r.uniform(math.log(len_lo), math.log(len_hi), B)).astype(np.int64)
        lens = np.clip(lens, len_lo, len_hi)
    else:
        lens = r.integers(len_lo, len_hi + 1, B)
    toks = r.integers(0, vocab, B)
    garbage_toks = r.integers(-(2**31), 2**31 - 1, B)
    garbage_lens = r.integers(-(2**31), 2**31 - 1, B)
    tokens = np.where(valid == 1, toks, garbage_toks).astype(np.int32)
    seq_lens = np.where(valid == 1, lens, garbage_lens).astype(np.int32)
    return Batch(tokens, valid, seq_lens)


def make_kv_contiguous(c: dict, n_slots: int, max_seq_len: int, seed: int, device="cpu",
                       layers=None, std: float = 1.0):
    """Contiguous per-slot cache, bf16 N(0, std): per layer K and V of shape
    [n_slots, n_kv_heads, max_seq_len, head_dim]."""
    L = c["n_layers"]
    layers = range(L) if layers is None else list(layers)
    kshape = (n_slots, c["n_kv_heads"], max_seq_len, c["head_dim"])
    vshape = kshape
    K = [_normal_bf16(kshape, std, seed, 2 * l, device) for l in layers]
    V = [_normal_bf16(vshape, std, seed, 2 * l + 1, device) for l in layers]
    return K, V


def make_page_table(n_slots: int, max_pages_per_seq: int, num_pages: int, seed: int) -> np.ndarray:
    """A seeded random permutation of page ids, max_pages_per_seq per slot."""
    assert num_pages >= n_slots * max_pages_per_seq
    r = np.random.default_rng(seed)
    perm = r.permutation(num_pages)[: n_slots * max_pages_per_seq]
    return perm.reshape(n_slots, max_pages_per_seq).astype(np.int32)


def make_kv_paged(c: dict, num_pages: int, page_size: int, seed: int, device="cpu",
                  layers=None, std: float = 1.0):
    """Paged cache, bf16 N(0, std): per layer K and V of shape [num_pages,
    n_kv_heads, page_size, head_dim]."""
    L = c["n_layers"]
    layers = range(L) if layers is None else list(layers)
    kshape = (num_pages, c["n_kv_heads"], page_size, c["head_dim"])
    vshape = kshape
    K = [_normal_bf16(kshape, std, seed, 2 * l, device) for l in layers]
    V = [_normal_bf16(vshape, std, seed, 2 * l + 1, device) for l in layers]
    return K, V


def make_prompt(vocab: int, length: int, seed: int) -> np.ndarray:
    return np.random.default_rng(seed).integers(0, vocab, length).astype(np.int32)
