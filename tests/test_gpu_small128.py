"""GPU tests with the 8B family's head geometry (head_dim 128, four query
heads per KV head) on a two-layer model: decode at B = 24, 48 and 72 (the
pipelined projection kernel with 32-, 64- and 128-row tiles, each M ragged)
and the causal prefill attention at ragged prompt lengths, against the
oracle; invariance under slot moves."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_14376_amd import corun
from paper_2608_14376_amd import workload as wl
from tests.gpu_helpers import DEV, check_tokens, host_model, oracle_kv, row_rel_err, to_device

pytestmark = pytest.mark.gpu
TOL = 2e-2
S_CAP = 400


@pytest.fixture(scope="module")
def small():
    cfg = wl.config("small128")
    Wc = wl.make_weights(cfg, seed=21)
    return cfg, Wc, to_device(Wc), host_model(Wc)


def cache(cfg, B, seed):
    K, V = wl.make_kv_contiguous(cfg, B, S_CAP, seed)
    return [k.to(DEV) for k in K], [v.to(DEV) for v in V]


@pytest.mark.parametrize("B,m_tile", [(24, 32), (48, 64), (72, 128)])
def test_decode_parity_and_slot_moves(small, B, m_tile):
    """The pipelined projection kernel with a 32-, 64- and 128-row tile (a
    ragged M tile each time), decode against the oracle row by row, then
    every live request moved to another slot: bit-identical."""
    cfg, Wc, Wg, m = small
    K, V = cache(cfg, B, 500)
    K0 = [k.clone() for k in K]
    V0 = [v.clone() for v in V]
    okv = oracle_kv(K, V)
    eng = corun.Engine(cfg, Wg, B, K, V)
    plan = eng.plan()
    for name in ("qkv", "o", "gate_up", "down", "lm_head"):
        assert plan[name]["m_tile"] == m_tile and plan[name]["n_tile"] > 0, name
    b = wl.make_batch(B, cfg["vocab"], seed=501, len_lo=16, len_hi=300)
    logits = torch.empty(B, cfg["vocab"], dtype=torch.float32, device=DEV)
    nxt = eng.decode_step(b.tokens, b.valid, b.seq_lens, logits)
    live = np.nonzero(b.valid)[0]
    sample = live[:: max(1, len(live) // 12)]          # oracle rows, one by one
    for r in sample:
        kv1 = oracle.KVCache([wl.bits(k[r:r + 1]) for k in K0], [wl.bits(v[r:r + 1]) for v in V0],
                             oracle.KV_CONTIGUOUS, 1, S_CAP)
        ref = oracle.decode_row(m, kv1, 0, int(b.tokens[r]), int(b.seq_lens[r]))
        assert row_rel_err(logits[r].cpu().numpy(), ref) <= TOL, r
    ref_logits = logits.clone()
    # move every live request to a new slot (a random permutation) with its cache
    perm = np.random.default_rng(502).permutation(B)
    for l in range(cfg["n_layers"]):
        K[l][perm] = K0[l]
        V[l][perm] = V0[l]
    t2, v2, s2 = (np.empty_like(x) for x in (b.tokens, b.valid, b.seq_lens))
    t2[perm], v2[perm], s2[perm] = b.tokens, b.valid, b.seq_lens
    nxt2 = eng.decode_step(t2, v2, s2, logits)
    for r in live:
        assert nxt2[perm[r]] == nxt[r]
        assert torch.equal(logits[perm[r]].view(torch.int32), ref_logits[r].view(torch.int32)), r


@pytest.mark.parametrize("Lp", [1, 33, 200, 333])
def test_prefill_parity_d128(small, Lp):
    cfg, Wc, Wg, m = small
    K, V = cache(cfg, 4, 510)
    okv = oracle_kv(K, V)
    eng = corun.Engine(cfg, Wg, 4, K, V, opt=corun.options(max_prefill_len=S_CAP))
    prompt = wl.make_prompt(cfg["vocab"], Lp, seed=511)
    last = torch.empty(cfg["vocab"], dtype=torch.float32, device=DEV)
    tok = eng.prefill(prompt, 3, last)
    ref, _ = oracle.prefill(m, okv, 3, prompt)
    assert row_rel_err(last.cpu().numpy(), ref) <= TOL
    check_tokens([tok], ref[None], last.cpu().numpy()[None], [1], [])
    for l in range(cfg["n_layers"]):
        g = (wl.bits(V[l])[3, :, :Lp].astype(np.uint32) << 16).view(np.float32)
        o = (okv.v[l][3, :, :Lp].astype(np.uint32) << 16).view(np.float32)
        assert np.abs(g - o).max() <= 2e-2 * np.abs(o).max()


def test_prefill_slot_independent_bitwise(small):
    cfg, Wc, Wg, m = small
    prompt = wl.make_prompt(cfg["vocab"], 257, seed=520)
    K, V = cache(cfg, 4, 521)
    eng = corun.Engine(cfg, Wg, 4, K, V, opt=corun.options(max_prefill_len=S_CAP))
    la = torch.empty(cfg["vocab"], dtype=torch.float32, device=DEV)
    lb = torch.empty_like(la)
    ta = eng.prefill(prompt, 0, la)
    tb = eng.prefill(prompt, 3, lb)
    assert ta == tb and torch.equal(la.view(torch.int32), lb.view(torch.int32))
    for l in range(cfg["n_layers"]):
        assert torch.equal(K[l][0, :, :257].view(torch.int16), K[l][3, :, :257].view(torch.int16))
