"""Batch-invariant mode (`batch_invariant` option), the baseline CoRun is
measured against (Sec. III, "Batch-Dependent GPU Reductions", Fig. 3b, and
Definition 1): no split-K and one MFMA instruction chain per output element
for every batch size (the tile follows B: 32-, 64-, 128- and 256-row tiles
across the batch sizes below), split-KV off in decode attention.

* A request's logits, greedy token and appended k/v are bit-identical across
  engines of different B (1, 5, 72, 130) and slots, among other co-runners:
  Definition 1.  The default plans change their reduction partition with B
  and only promise Definition 2 (position invariance at one B).
* Batch-invariant decode and prefill agree with the oracle to the same
  tolerance as the default path (relative 2e-2 on logits).

Two configurations: small128 (every K a multiple of 64: the pipelined
kernel) and tiny (down K = 688: the LDS-tiled kernel with a K tail)."""
import ctypes as C

import numpy as np
import pytest
import torch

import oracle
from paper_2608_14376_amd import corun
from paper_2608_14376_amd import workload as wl
from tests.gpu_helpers import DEV, check_tokens, host_model, oracle_kv, row_rel_err, to_device

pytestmark = pytest.mark.gpu
TOL = 2e-2
CAP = 400
BS = (1, 5, 72, 130)
BI = corun.options(batch_invariant=True)


@pytest.fixture(scope="module", params=["small128", "tiny"])
def model(request):
    cfg = wl.config(request.param)
    Wc = wl.make_weights(cfg, seed=31)
    return cfg, to_device(Wc), host_model(Wc)


def target(cfg):
    """One request: its own cache (one slot), token and position."""
    K, V = wl.make_kv_contiguous(cfg, 1, CAP, seed=900)
    rng = np.random.default_rng(901)
    return K, V, int(rng.integers(0, cfg["vocab"])), 250


def run_at(cfg, Wg, B, slot, tgt, opt, seed):
    """The target request at `slot` of a B-row step among seeded co-runners;
    returns its logits bits, greedy token and appended k/v bits."""
    Kt, Vt, tok, pos = tgt
    K, V = wl.make_kv_contiguous(cfg, B, CAP, seed)
    for l in range(cfg["n_layers"]):
        K[l][slot] = Kt[l][0]
        V[l][slot] = Vt[l][0]
    K = [k.to(DEV) for k in K]
    V = [v.to(DEV) for v in V]
    eng = corun.Engine(cfg, Wg, B, K, V, opt=opt)
    b = wl.make_batch(B, cfg["vocab"], seed=seed + 1, len_lo=16, len_hi=CAP - 8)
    tokens, valid, seq = b.tokens.copy(), b.valid.copy(), b.seq_lens.copy()
    tokens[slot], valid[slot], seq[slot] = tok, 1, pos
    logits = torch.empty(B, cfg["vocab"], dtype=torch.float32, device=DEV)
    nxt = eng.decode_step(tokens, valid, seq, logits)
    row = logits[slot].cpu().numpy()
    kv_bits = [(K[l][slot, :, pos].cpu(), V[l][slot, :, pos].cpu()) for l in range(cfg["n_layers"])]
    eng.close()
    return row, int(nxt[slot]), kv_bits


def shape_only_kv(n_slots):
    """A contiguous cache description with null pointers (describe_plan reads shapes only)."""
    null = (C.c_void_p * 1)(None)
    kv = corun.KV(corun.KV_CONTIGUOUS, n_slots, CAP, 0, 0, 0, C.cast(null, corun._PP), C.cast(null, corun._PP), None)
    kv._keep = null
    return kv


def same_kv(a, b):
    return all(torch.equal(x[0].view(torch.int16), y[0].view(torch.int16)) and
               torch.equal(x[1].view(torch.int16), y[1].view(torch.int16)) for x, y in zip(a, b))


def test_request_is_bit_identical_across_batch_sizes(model):
    cfg, Wg, m = model
    tgt = target(cfg)
    runs = [run_at(cfg, Wg, B, (7 * i + B - 1) % B, tgt, BI, seed=910 + 10 * i) for i, B in enumerate(BS)]
    row0, tok0, kv0 = runs[0]
    for (row, tok, kv), B in zip(runs[1:], BS[1:]):
        assert np.array_equal(row.view(np.int32), row0.view(np.int32)), B
        assert tok == tok0 and same_kv(kv, kv0), B
    # the oracle: the request alone
    Kt, Vt, t, pos = tgt
    ref = oracle.decode_row(m, oracle_kv(Kt, Vt), 0, t, pos)
    assert row_rel_err(row0, ref) <= TOL
    check_tokens([tok0], ref[None], row0[None], [1], [])


def test_default_plans_are_position_invariant_at_each_B(model):
    """The default plan changes with B (tiles, and split-K factors where K
    is large enough to split), so it promises Definition 2 only: at one B
    the request is bit-identical at another slot among other co-runners.
    Whether a change reaches the logits depends on whether it changes a
    reduction partition and that flips a bf16 rounding on the way; at these
    small shapes it rarely does, at the 8B shapes it does (the benchmark
    compares B = 32 with B = 256)."""
    cfg, Wg, m = model
    plans = [corun.describe_plan(cfg, shape_only_kv(B), B) for B in (1, 130)]
    assert any(plans[0][n] != plans[1][n] for n in ("qkv", "o", "gate_up", "down", "lm_head"))
    tgt = target(cfg)
    large = run_at(cfg, Wg, 130, 77, tgt, None, seed=960)
    moved = run_at(cfg, Wg, 130, 3, tgt, None, seed=970)          # same B, other slot and co-runners
    assert np.array_equal(moved[0].view(np.int32), large[0].view(np.int32))
    assert moved[1] == large[1] and same_kv(moved[2], large[2])


@pytest.mark.parametrize("Lp", [1, 200, 333])
def test_batch_invariant_prefill_parity(model, Lp):
    cfg, Wg, m = model
    K, V = wl.make_kv_contiguous(cfg, 4, CAP, 980)
    K = [k.to(DEV) for k in K]
    V = [v.to(DEV) for v in V]
    okv = oracle_kv(K, V)
    eng = corun.Engine(cfg, Wg, 4, K, V, opt=corun.options(max_prefill_len=CAP, batch_invariant=True))
    prompt = wl.make_prompt(cfg["vocab"], Lp, seed=981)
    last = torch.empty(cfg["vocab"], dtype=torch.float32, device=DEV)
    tok = eng.prefill(prompt, 2, last)
    ref, _ = oracle.prefill(m, okv, 2, prompt)
    assert row_rel_err(last.cpu().numpy(), ref) <= TOL
    check_tokens([tok], ref[None], last.cpu().numpy()[None], [1], [])
    for l in range(cfg["n_layers"]):
        g = (wl.bits(V[l])[2, :, :Lp].astype(np.uint32) << 16).view(np.float32)
        o = (okv.v[l][2, :, :Lp].astype(np.uint32) << 16).view(np.float32)
        assert np.abs(g - o).max() <= TOL * np.abs(o).max()
    eng.close()
