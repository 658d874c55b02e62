"""Shared helpers for the GPU tests: device copies of seeded inputs, the
oracle's host view of the same inputs, and the parity metrics."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2608_14376_amd import workload as wl

DEV = "cuda"


def to_device(W: wl.Weights) -> wl.Weights:
    mv = lambda lst: [t.to(DEV) for t in lst]
    return wl.Weights(W.cfg, W.embed.to(DEV), W.final_norm.to(DEV), W.lm_head.to(DEV), mv(W.attn_norm),
                      mv(W.w_qkv), mv(W.w_o), mv(W.mlp_norm), mv(W.w_gate_up), mv(W.w_down), mv(W.w_router),
                      mv(W.w_exp_gate_up), mv(W.w_exp_down))


def host_model(W: wl.Weights) -> oracle.Model:
    b = wl.bits
    return oracle.Model(W.cfg, b(W.embed), b(W.final_norm), b(W.lm_head), [b(t) for t in W.attn_norm],
                        [b(t) for t in W.w_qkv], [b(t) for t in W.w_o], [b(t) for t in W.mlp_norm],
                        [b(t) for t in W.w_gate_up], [b(t) for t in W.w_down], [b(t) for t in W.w_router],
                        [b(t) for t in W.w_exp_gate_up], [b(t) for t in W.w_exp_down])


def oracle_kv(K, V, layout=oracle.KV_CONTIGUOUS, page_size=16, page_table=None) -> oracle.KVCache:
    k = [wl.bits(t) for t in K]
    v = [wl.bits(t) for t in V]
    if layout == oracle.KV_PAGED:
        n_slots, mpp = page_table.shape
        return oracle.KVCache(k, v, layout, n_slots, 0, page_size, k[0].shape[0], mpp,
                              np.ascontiguousarray(page_table, np.int32))
    return oracle.KVCache(k, v, layout, k[0].shape[0], k[0].shape[2])


def row_rel_err(gpu: np.ndarray, ref: np.ndarray) -> float:
    """max_v |g - o| / max_v |o| for one row."""
    return float(np.abs(gpu.astype(np.float64) - ref).max() / np.abs(ref).max())


def top2_gap(ref: np.ndarray) -> float:
    r = np.sort(ref.astype(np.float32).astype(np.float64))
    return float(r[-1] - r[-2])


def check_tokens(gpu_next, ref_logits, gpu_logits, valid, near_ties: list):
    """Greedy tokens must agree wherever the oracle's top-1/top-2 gap exceeds
    four times the row's measured logit error; closer calls are logged as
    near-ties."""
    for b in range(len(valid)):
        if not valid[b]:
            assert gpu_next[b] == -1
            continue
        ref = ref_logits[b]
        err = float(np.abs(gpu_logits[b].astype(np.float64) - ref).max())
        exp = int(np.argmax(ref.astype(np.float32)))
        if top2_gap(ref) > 4 * err:
            assert gpu_next[b] == exp, (b, gpu_next[b], exp, top2_gap(ref), err)
        elif gpu_next[b] != exp:
            near_ties.append((b, top2_gap(ref), err))
