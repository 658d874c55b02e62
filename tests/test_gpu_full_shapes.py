"""GPU parity at the 8B workload's real per-layer shapes (hidden 4096, 32/8
heads of 128, FFN 12288, vocabulary 151936) on a two-layer slice: the plan
-- kernel, tile, split-K, attention chunk -- depends on B, the per-layer
shapes and the cache capacity only, so these launches are the ones the
decode and prefill benchmarks time, layer count aside.

* decode at B = 256 with the benchmark's context lengths and cache
  capacity: sampled live rows against the oracle row by row, and a
  two-slot swap bitwise;
* prefill of 600 tokens (past the 512 where the 256 x 256 projection tiles
  start): sampled positions t are recomputed by the oracle's decode row on
  the GPU-written cache prefix (teacher forcing), which checks the
  position's whole computation -- its logits at the last position, its
  cached key and value everywhere -- without an oracle prefill of 600
  positions;
* prefill of 32768 tokens (the longest benchmarked prompt), sampled
  positions checked the same way."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_14376_amd import corun
from paper_2608_14376_amd import workload as wl
from tests.gpu_helpers import DEV, check_tokens, host_model, row_rel_err

pytestmark = pytest.mark.gpu
TOL = 2e-2
B = 256
CAP = 4144          # the decode benchmark's capacity: contexts up to 4096 plus its steps, rounded to 16
LP = 600


@pytest.fixture(scope="module")
def full():
    cfg = dict(wl.config("8b"), n_layers=2)
    Wg = wl.make_weights(cfg, seed=41, device=DEV)
    return cfg, Wg, host_model(Wg)


def row_cache(K, V, r, cap):
    return oracle.KVCache([wl.bits(k[r:r + 1]) for k in K], [wl.bits(v[r:r + 1]) for v in V],
                          oracle.KV_CONTIGUOUS, 1, cap)


def test_decode_B256_full_shapes(full):
    cfg, Wg, m = full
    K, V = wl.make_kv_contiguous(cfg, B, CAP, seed=42, device=DEV)
    eng = corun.Engine(cfg, Wg, B, K, V)
    plan = eng.plan()
    # the benchmark's configurations: 256 x 256 tiles for gate/up, 256 x 128
    # for the lm_head (with its argmax epilogue), 128 x 128 (two M tiles) elsewhere
    assert (plan["gate_up"]["m_tile"], plan["gate_up"]["n_tile"]) == (256, 256)
    assert (plan["lm_head"]["m_tile"], plan["lm_head"]["n_tile"], plan["lm_head"]["split_k"]) == (256, 128, 1)
    for name in ("qkv", "o", "down"):
        assert (plan[name]["m_tile"], plan[name]["n_tile"]) == (128, 128), name
    b = wl.make_batch(B, cfg["vocab"], seed=43, len_lo=512, len_hi=4096)
    live = np.nonzero(b.valid)[0]
    sample = live[:: max(1, len(live) // 5)][:6]
    K0 = {int(r): [k[r:r + 1].clone() for k in K] for r in sample}
    V0 = {int(r): [v[r:r + 1].clone() for v in V] for r in sample}
    logits = torch.empty(B, cfg["vocab"], dtype=torch.float32, device=DEV)
    nxt = eng.decode_step(b.tokens, b.valid, b.seq_lens, logits)
    gl = logits.cpu().numpy()
    for r in sample:
        r = int(r)
        ref = oracle.decode_row(m, row_cache(K0[r], V0[r], 0, CAP), 0, int(b.tokens[r]), int(b.seq_lens[r]))
        assert row_rel_err(gl[r], ref) <= TOL, (r, row_rel_err(gl[r], ref))
    # swap two live requests' slots (tokens, lengths, caches): their rows swap bitwise
    a, c = int(live[0]), int(live[-1])
    for l in range(cfg["n_layers"]):
        ka, va = K[l][a].clone(), V[l][a].clone()
        K[l][a].copy_(K[l][c]); V[l][a].copy_(V[l][c])
        K[l][c].copy_(ka); V[l][c].copy_(va)
    t2, s2 = b.tokens.copy(), b.seq_lens.copy()
    t2[[a, c]], s2[[a, c]] = t2[[c, a]], s2[[c, a]]
    ref_logits = logits.clone()
    # the first step appended each row's new key and value at its own length;
    # the second step appends the same values there again, so the caches agree
    nxt2 = eng.decode_step(t2, b.valid, s2, logits)
    assert nxt2[a] == nxt[c] and nxt2[c] == nxt[a]
    assert torch.equal(logits[a].view(torch.int32), ref_logits[c].view(torch.int32))
    assert torch.equal(logits[c].view(torch.int32), ref_logits[a].view(torch.int32))


# The small-B plans the decode benchmark times (8B shapes, capacity 4144):
# at B = 1 the small-batch layer (every layer projection on 16-column
# fragment-packed tiles over the whole of K, norm / RoPE + KV append /
# SwiGLU / residual in the projections); at B = 8, 16 and 64 packed 32- or
# 64-row weight tiles with split-K 5 (qkv) and 8 (o, down), gate/up without
# split-K (its epilogue applies SwiGLU; at B = 8 attention applies the QKV
# epilogue); the lm_head on the packed 32- or 64-row tiles; the attention
# chunk that gives up to 33 splits at B = 1, 17 at B = 8, 9 at B = 16, 5 at B = 64.
SMALL_B = {1: (32, 128, 33), 8: (32, 256, 17), 16: (32, 512, 9), 64: (64, 1024, 5)}


@pytest.mark.parametrize("Bs", sorted(SMALL_B))
def test_decode_small_B_full_shapes(full, Bs):
    cfg, Wg, m = full
    K, V = wl.make_kv_contiguous(cfg, Bs, CAP, seed=60 + Bs, device=DEV)
    eng = corun.Engine(cfg, Wg, Bs, K, V)
    plan = eng.plan()
    mt, chunk, splits = SMALL_B[Bs]
    if Bs == 1:
        for name in ("qkv", "o", "gate_up", "down"):
            assert (plan[name]["split_k"], plan[name]["m_tile"], plan[name]["n_tile"]) == (1, 16, 16), name
    else:
        for name, S in (("qkv", 5), ("o", 8), ("gate_up", 1), ("down", 8)):
            assert (plan[name]["split_k"], plan[name]["m_tile"], plan[name]["n_tile"]) == (S, mt, 128), name
    assert (plan["lm_head"]["split_k"], plan["lm_head"]["m_tile"], plan["lm_head"]["n_tile"]) == (1, mt, 128)
    assert (plan["attn_chunk"], plan["attn_max_splits"]) == (chunk, splits)
    b = wl.make_batch(Bs, cfg["vocab"], seed=70 + Bs, len_lo=512, len_hi=4096)
    live = np.nonzero(b.valid)[0]
    sample = [int(r) for r in (live if Bs <= 16 else live[:: max(1, len(live) // 6)][:6])]
    okv = {r: row_cache(K, V, r, CAP) for r in sample}
    tokens, lens = b.tokens.copy(), b.seq_lens.copy()
    logits = torch.empty(Bs, cfg["vocab"], dtype=torch.float32, device=DEV)
    worst, near = 0.0, []
    for step in range(2):
        nxt = eng.decode_step(tokens, b.valid, lens, logits)
        gl = logits.cpu().numpy()
        for r in sample:
            ref = oracle.decode_row(m, okv[r], 0, int(tokens[r]), int(lens[r]))
            err = row_rel_err(gl[r], ref)
            worst = max(worst, err)
            assert err <= TOL, (step, r, err)
            check_tokens([nxt[r]], ref[None], gl[r][None], [1], near)
        tokens = np.where(b.valid == 1, nxt, tokens).astype(np.int32)
        lens = np.where(b.valid == 1, lens + 1, lens).astype(np.int32)
    eng.close()
    assert len(near) <= 1, near
    print(f"B={Bs}: {len(sample)} rows x 2 steps, max row-relative logit error {worst:.2e}")


def test_prefill_600_full_shapes_teacher_forced(full):
    cfg, Wg, m = full
    cap = 608
    K, V = wl.make_kv_contiguous(cfg, 2, cap, seed=44, device=DEV)
    eng = corun.Engine(cfg, Wg, 2, K, V, opt=corun.options(max_prefill_len=LP))
    prompt = wl.make_prompt(cfg["vocab"], LP, seed=45)
    last = torch.empty(cfg["vocab"], dtype=torch.float32, device=DEV)
    eng.prefill(prompt, 1, last)
    gk = [wl.bits(k[1]) for k in K]          # [nkv, cap, d] per layer
    gv = [wl.bits(v[1]) for v in V]          # [nkv, cap, d]
    f32 = lambda a: (a.astype(np.uint32) << 16).view(np.float32)
    for t in (0, 1, 255, 256, 511, 512, LP - 1):
        kv1 = row_cache(K, V, 1, cap)        # the GPU-written prefix; position t is recomputed
        ref = oracle.decode_row(m, kv1, 0, int(prompt[t]), t)
        for l in range(cfg["n_layers"]):
            ok, ov = f32(kv1.k[l][0, :, t, :]), f32(kv1.v[l][0, :, t, :])
            assert np.abs(f32(gk[l][:, t, :]) - ok).max() <= TOL * np.abs(ok).max(), (t, l)
            assert np.abs(f32(gv[l][:, t, :]) - ov).max() <= TOL * np.abs(ov).max(), (t, l)
        if t == LP - 1:
            assert row_rel_err(last.cpu().numpy(), ref) <= TOL


def test_prefill_32768_full_shapes_teacher_forced(full):
    """The longest benchmarked prompt: its projections take the largest-M
    tiles and split-K of the prefill plan, and its causal attention spans
    32768 keys; sampled positions are recomputed as above."""
    cfg, Wg, m = full
    lp, cap = 32768, 32784
    K, V = wl.make_kv_contiguous(cfg, 2, cap, seed=46, device=DEV)
    eng = corun.Engine(cfg, Wg, 2, K, V, opt=corun.options(max_prefill_len=lp))
    prompt = wl.make_prompt(cfg["vocab"], lp, seed=47)
    last = torch.empty(cfg["vocab"], dtype=torch.float32, device=DEV)
    eng.prefill(prompt, 1, last)
    eng.close()
    gk = [wl.bits(k[1]) for k in K]
    gv = [wl.bits(v[1]) for v in V]
    f32 = lambda a: (a.astype(np.uint32) << 16).view(np.float32)
    for t in (0, 4095, 16384, lp - 1):
        kv1 = row_cache(K, V, 1, cap)
        ref = oracle.decode_row(m, kv1, 0, int(prompt[t]), t)
        for l in range(cfg["n_layers"]):
            ok, ov = f32(kv1.k[l][0, :, t, :]), f32(kv1.v[l][0, :, t, :])
            assert np.abs(f32(gk[l][:, t, :]) - ok).max() <= TOL * np.abs(ok).max(), (t, l)
            assert np.abs(f32(gv[l][:, t, :]) - ov).max() <= TOL * np.abs(ov).max(), (t, l)
        if t == lp - 1:
            err = row_rel_err(last.cpu().numpy(), ref)
            print(f"prefill of {lp}: last-position relative logit error {err:.2e}")
            assert err <= TOL


def test_prefill_bits_do_not_depend_on_the_workspace(full):
    """The same 300-token prompt on two engines whose prefill workspaces
    differ (300 and 4096 tokens) gives identical k, v and logits bits: the
    plan -- here with split-K on the narrow projections -- is a function of
    the prompt length alone (Sec. IV, "Isolated Prefill")."""
    cfg, Wg, m = full
    lp, cap = 300, 320
    plan = corun.describe_prefill_plan(cfg, lp)
    assert max(plan[n]["split_k"] for n in ("qkv", "o", "gate_up", "down")) > 1, plan
    prompt = wl.make_prompt(cfg["vocab"], lp, seed=48)
    outs = []
    for pf in (lp, 4096):
        K, V = wl.make_kv_contiguous(cfg, 2, cap, seed=49, device=DEV)
        eng = corun.Engine(cfg, Wg, 2, K, V, opt=corun.options(max_prefill_len=pf))
        last = torch.empty(cfg["vocab"], dtype=torch.float32, device=DEV)
        tok = eng.prefill(prompt, 1, last)
        torch.cuda.synchronize()
        outs.append((tok, last.view(torch.int32).cpu(), [k[1, :, :lp].clone() for k in K],
                     [v[1, :, :lp].clone() for v in V]))
        eng.close()
    a, b = outs
    assert a[0] == b[0] and torch.equal(a[1], b[1])
    for l in range(cfg["n_layers"]):
        assert torch.equal(a[2][l].view(torch.int16), b[2][l].view(torch.int16)), l
        assert torch.equal(a[3][l].view(torch.int16), b[3][l].view(torch.int16)), l
