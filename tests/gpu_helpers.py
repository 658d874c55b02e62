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


def check_routing(gsel, glog, rl, own, where, tol=2e-2):
    """The GPU's mixture-of-experts routing of one row against the oracle's
    records of the same trajectory (the oracle run with force = gsel).

    gsel [L, k], glog [L, E]: the GPU's choice and the fp32 router logits it
    was made from; rl [L, E], own [L, k]: the oracle's fp64 router logits and
    its own top-k on that trajectory.  Per layer:
      * exact: gsel is the top-k of glog, ties to the lower expert id;
      * the router logits agree within tol of the layer's largest |logit|;
      * where the two expert sets differ, the oracle's logits admit the GPU's
        set as a top-k under the measured error eps = max |glog - rl|: every
        chosen expert's logit is at least every other's minus 2 eps (each of
        the two logits can be off by eps).  Such a layer is a routing
        near-tie: both choices are correct results.
    Returns the near-ties as (where, layer, gap, eps)."""
    near = []
    L, k = gsel.shape
    for l in range(L):
        g = glog[l].astype(np.float64)
        top = np.lexsort((np.arange(g.size), -g))[:k]
        assert list(gsel[l]) == list(top), (where, l, list(gsel[l]), list(top))
        eps = float(np.abs(g - rl[l]).max())
        assert eps <= tol * np.abs(rl[l]).max(), (where, l, eps)
        if set(gsel[l].tolist()) != set(own[l].tolist()):
            chosen = rl[l][list(gsel[l])].min()
            other = np.delete(rl[l], list(gsel[l])).max()
            assert chosen >= other - 2 * eps, (where, l, float(chosen), float(other), eps)
            near.append((where, l, float(other - chosen), eps))
    return near


def routed_decode_row(m, okv, slot, token, pos, gsel, glog, where):
    """Oracle logits of one decode row following the GPU's expert sets
    (checked by check_routing); returns (logits, routing near-ties)."""
    ref, rl, own = oracle.decode_row_routed(m, okv, slot, token, pos, force=gsel)
    return ref, check_routing(gsel, glog, rl, own, where)
