"""Edge cases of the decode step on the GPU, against the oracle and the
invariance contract (Sec. III, Definition 2):

* positions at both ends of the cache in one batch: a row at position 0
  (no cached key: it attends to its own new key only), a row at the last
  position of its capacity, rows in between; head_dim 64 and 128,
  contiguous and paged (pages ending exactly at the capacity);
* the largest fixed batch the ABI accepts (B_fixed = 1024) on the tiny
  model: sampled rows against the oracle, and a live row moved to another
  slot among other co-runners gives the same bits;
* the prefill workspace used to its last token (a prompt of exactly
  max_prefill_len tokens);
* the host copy of the page table (corun_engine_set_page_table_host) used
  by the checks in place of the device table."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_14376_amd import corun
from paper_2608_14376_amd import workload as wl
from tests.gpu_helpers import DEV, check_tokens, host_model, oracle_kv, row_rel_err, to_device

pytestmark = pytest.mark.gpu
TOL = 2e-2
CAP = 320
PS = 16


@pytest.fixture(scope="module", params=["tiny", "small128"])
def model(request):
    cfg = wl.config(request.param)
    Wc = wl.make_weights(cfg, seed=81)
    return cfg, to_device(Wc), host_model(Wc)


@pytest.mark.parametrize("paged", [False, True])
def test_first_and_last_positions(model, paged):
    cfg, Wg, m = model
    B = 6
    lens = np.array([0, CAP - 1, 1, 127, 128, CAP - 2], np.int32)
    valid = np.ones(B, np.uint8)
    tokens = np.random.default_rng(82).integers(0, cfg["vocab"], B).astype(np.int32)
    if paged:
        mpp = CAP // PS
        num_pages = B * mpp + 2
        pt = wl.make_page_table(B, mpp, num_pages, seed=83)
        K, V = wl.make_kv_paged(cfg, num_pages, PS, seed=84)
        K = [k.to(DEV) for k in K]
        V = [v.to(DEV) for v in V]
        okv = oracle_kv(K, V, layout=oracle.KV_PAGED, page_size=PS, page_table=pt)
        eng = corun.Engine(cfg, Wg, B, K, V, layout=corun.KV_PAGED, page_size=PS,
                           page_table=torch.from_numpy(pt).to(DEV))
    else:
        K, V = wl.make_kv_contiguous(cfg, B, CAP, seed=85)
        K = [k.to(DEV) for k in K]
        V = [v.to(DEV) for v in V]
        okv = oracle_kv(K, V)
        eng = corun.Engine(cfg, Wg, B, K, V)
    logits = torch.empty(B, cfg["vocab"], dtype=torch.float32, device=DEV)
    nxt = eng.decode_step(tokens, valid, lens, logits)
    ref, _ = oracle.decode_batch(m, okv, tokens, valid, lens)
    gl = logits.cpu().numpy()
    for r in range(B):
        assert row_rel_err(gl[r], ref[r]) <= TOL, (r, int(lens[r]))
    check_tokens(nxt, ref, gl, valid, [])
    # a row at the capacity limit cannot take another step
    with pytest.raises(corun.CorunError):
        eng.decode_step(tokens, valid, np.where(lens == CAP - 1, CAP, lens).astype(np.int32))
    eng.close()


def test_largest_fixed_batch():
    cfg = wl.config("tiny")
    Wc = wl.make_weights(cfg, seed=86)
    Wg, m = to_device(Wc), host_model(Wc)
    B, S = 1024, 160
    K, V = wl.make_kv_contiguous(cfg, B, S, seed=87)
    K = [k.to(DEV) for k in K]
    V = [v.to(DEV) for v in V]
    K0 = [k.clone() for k in K]
    V0 = [v.clone() for v in V]
    eng = corun.Engine(cfg, Wg, B, K, V)
    b = wl.make_batch(B, cfg["vocab"], seed=88, len_lo=16, len_hi=S - 8, live_frac=(0.3, 0.3))
    logits = torch.empty(B, cfg["vocab"], dtype=torch.float32, device=DEV)
    nxt = eng.decode_step(b.tokens, b.valid, b.seq_lens, logits)
    live = np.nonzero(b.valid)[0]
    for r in live[:: max(1, len(live) // 16)]:
        kv1 = oracle.KVCache([wl.bits(k[r:r + 1]) for k in K0], [wl.bits(v[r:r + 1]) for v in V0],
                             oracle.KV_CONTIGUOUS, 1, S)
        ref = oracle.decode_row(m, kv1, 0, int(b.tokens[r]), int(b.seq_lens[r]))
        assert row_rel_err(logits[r].cpu().numpy(), ref) <= TOL, r
    # move one live request into a padding slot, with its cache; other rows stay
    src = int(live[len(live) // 2])
    dst = int(np.nonzero(b.valid == 0)[0][-1])
    ref_bits = logits[src].clone().view(torch.int32)
    for l in range(cfg["n_layers"]):
        K[l][dst] = K0[l][src]
        V[l][dst] = V0[l][src]
        K[l][src] = K0[l][src]
        V[l][src] = V0[l][src]
    t, v, s = b.tokens.copy(), b.valid.copy(), b.seq_lens.copy()
    t[dst], v[dst], s[dst] = t[src], 1, s[src]
    v[src] = 0
    nxt2 = eng.decode_step(t, v, s, logits)
    assert nxt2[dst] == nxt[src]
    assert torch.equal(logits[dst].view(torch.int32), ref_bits)
    eng.close()


def test_prefill_fills_the_workspace(model):
    cfg, Wg, m = model
    L = 96
    K, V = wl.make_kv_contiguous(cfg, 2, CAP, seed=89)
    K = [k.to(DEV) for k in K]
    V = [v.to(DEV) for v in V]
    okv = oracle_kv(K, V)
    eng = corun.Engine(cfg, Wg, 2, K, V, opt=corun.options(max_prefill_len=L))
    prompt = wl.make_prompt(cfg["vocab"], L, seed=90)
    last = torch.empty(cfg["vocab"], dtype=torch.float32, device=DEV)
    tok = eng.prefill(prompt, 1, last)
    ref, _ = oracle.prefill(m, okv, 1, prompt)
    assert row_rel_err(last.cpu().numpy(), ref) <= TOL
    check_tokens([tok], ref[None], last.cpu().numpy()[None], [1], [])
    with pytest.raises(corun.CorunError):
        eng.prefill(wl.make_prompt(cfg["vocab"], L + 1, seed=91), 0)
    eng.close()


@pytest.mark.parametrize("poison", [False, True])
def test_time_kernel_needs_a_step_and_keeps_results(poison):
    """corun_time_kernel launches nothing before the engine's first decode
    step (CORUN_E_STATE: no validated inputs exist yet).  After a step whose
    rows sit at the last cache position (so the step's feedback moves them
    to the capacity), timing the kernels that append to and read the cache
    runs them at the step's own positions, and the next step still matches
    a fresh engine's bit for bit, caches included."""
    cfg = wl.config("tiny")
    Wg = to_device(wl.make_weights(cfg, seed=71))
    B, cap = 4, 160
    K, V = wl.make_kv_contiguous(cfg, B, cap, seed=72, device=DEV)
    b = wl.make_batch(B, cfg["vocab"], seed=73, len_lo=16, len_hi=128)
    last = b.seq_lens.copy()
    last[b.valid == 1] = cap - 1
    outs = []
    for timed in (True, False):
        Kc, Vc = [k.clone() for k in K], [v.clone() for v in V]
        eng = corun.Engine(cfg, Wg, B, Kc, Vc, opt=corun.options(poison_workspace=poison, qkv_epilogue=1))
        if timed:
            with pytest.raises(corun.CorunError) as ei:
                eng.time_kernel(corun.K_ATTN_SPLIT, 0, 3)
            assert ei.value.status == corun.E_STATE
        logits = torch.empty(B, cfg["vocab"], dtype=torch.float32, device=DEV)
        eng.decode_step(b.tokens, b.valid, last, logits)
        if timed:
            for kern in (corun.K_QKV_POST, corun.K_ATTN_SPLIT, corun.K_ATTN_MERGE):
                assert eng.time_kernel(kern, 0, 3) > 0
        eng.decode_step(b.tokens, b.valid, last, logits)
        torch.cuda.synchronize()
        outs.append((logits.cpu().numpy().view(np.int32)[b.valid == 1],
                     [wl.bits(k) for k in Kc], [wl.bits(v) for v in Vc]))
        eng.close()
    assert np.array_equal(outs[0][0], outs[1][0])
    for l in range(cfg["n_layers"]):
        assert np.array_equal(outs[0][1][l], outs[1][1][l]) and np.array_equal(outs[0][2][l], outs[1][2][l])


def test_profile_step_times_every_launch_and_changes_nothing():
    """corun_profile_step: every kernel class the step launches gets a
    positive in-step duration and its launch count (norms 2 L + 1, the other
    per-layer kernels L, lm_head and argmax once); it refuses before the first
    step; and the next step's logits and cache match an engine that never
    profiled, bit for bit."""
    cfg = wl.config("tiny")
    Wg = to_device(wl.make_weights(cfg, seed=74))
    B, cap = 4, 160
    K, V = wl.make_kv_contiguous(cfg, B, cap, seed=75, device=DEV)
    b = wl.make_batch(B, cfg["vocab"], seed=76, len_lo=16, len_hi=128)
    outs = []
    for prof in (True, False):
        Kc, Vc = [k.clone() for k in K], [v.clone() for v in V]
        eng = corun.Engine(cfg, Wg, B, Kc, Vc, opt=corun.options(qkv_epilogue=1))
        logits = torch.empty(B, cfg["vocab"], dtype=torch.float32, device=DEV)
        if prof:
            with pytest.raises(corun.CorunError) as ei:
                eng.profile_step(2)
            assert ei.value.status == corun.E_STATE
        eng.decode_step(b.tokens, b.valid, b.seq_lens, logits)
        if prof:
            p = eng.profile_step(2)
            L = cfg["n_layers"]
            want = {"rmsnorm": 2 * L + 1, "qkv_gemm": L, "qkv_post": L, "attn_split": L, "attn_merge": L,
                    "o_gemm": L, "gate_up_gemm": L, "down_gemm": L, "lm_head": 1, "argmax": 1}
            for name, n in want.items():
                assert name in p and p[name][1] == n and 0.0 < p[name][0] < 1e5, (name, p.get(name))
        eng.decode_step(b.tokens, b.valid, b.seq_lens, logits)
        torch.cuda.synchronize()
        outs.append((logits.cpu().numpy().view(np.int32)[b.valid == 1], [wl.bits(k) for k in Kc]))
        eng.close()
    assert np.array_equal(outs[0][0], outs[1][0])
    assert all(np.array_equal(x, y) for x, y in zip(outs[0][1], outs[1][1]))


def test_page_table_host_copy():
    """A registered host copy of the page table replaces the per-call device
    copy in the host-side checks: the same step gives the same bits with it,
    a page the copy maps out of range is refused (while the device table is
    valid) before anything runs, unregistering goes back to the device
    table, and a contiguous engine refuses a copy."""
    cfg = wl.config("tiny")
    Wg = to_device(wl.make_weights(cfg, seed=85))
    B, mpp = 4, CAP // PS
    num_pages = B * mpp
    pt = wl.make_page_table(B, mpp, num_pages, seed=86)
    K, V = wl.make_kv_paged(cfg, num_pages, PS, seed=87, device=DEV)
    eng = corun.Engine(cfg, Wg, B, K, V, layout=corun.KV_PAGED, page_size=PS,
                       page_table=torch.from_numpy(pt).to(DEV))
    b = wl.make_batch(B, cfg["vocab"], seed=88, len_lo=16, len_hi=CAP - 8)
    la = torch.empty(B, cfg["vocab"], dtype=torch.float32, device=DEV)
    lb = torch.empty_like(la)
    # the step appends at seq_len, so running it again rewrites the same values
    na = eng.decode_step(b.tokens, b.valid, b.seq_lens, la)
    host = pt.copy()
    eng.set_page_table_host(host)
    nb = eng.decode_step(b.tokens, b.valid, b.seq_lens, lb)
    assert np.array_equal(na, nb)
    live = torch.from_numpy(b.valid.astype(bool)).to(DEV)
    assert torch.equal(la[live].view(torch.int32), lb[live].view(torch.int32))
    r = int(np.nonzero(b.valid)[0][0])
    host[r, b.seq_lens[r] // PS] = num_pages          # only the host copy is wrong
    before = [k.clone() for k in K]
    with pytest.raises(corun.CorunError) as ei:
        eng.decode_step(b.tokens, b.valid, b.seq_lens, lb)
    assert ei.value.status == corun.E_CAPACITY
    for l in range(cfg["n_layers"]):                  # refused before anything ran
        assert torch.equal(K[l].view(torch.int16), before[l].view(torch.int16))
    eng.set_page_table_host(None)
    nc = eng.decode_step(b.tokens, b.valid, b.seq_lens, lb)
    assert np.array_equal(na, nc)
    eng.close()
    Kc, Vc = wl.make_kv_contiguous(cfg, B, CAP, seed=89, device=DEV)
    ec = corun.Engine(cfg, Wg, B, Kc, Vc)
    with pytest.raises(corun.CorunError) as ei:
        ec.set_page_table_host(pt.copy())
    assert ei.value.status == corun.E_STATE
    ec.close()
