"""Pins for the CPU oracle: each operator against closed forms, brute force
or an independent library routine; the whole step against a structurally
different library composition and against the invariants the paper's
determinism argument relies on (Sec. IV, "Determinism Argument")."""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2608_14376_amd import workload as wl
from tests import torch_reference as tref

def bf16_bits_of(x: np.ndarray) -> np.ndarray:
    return wl.bits(torch.as_tensor(np.asarray(x, np.float32)).to(torch.bfloat16))


def bf16_val(b) -> np.ndarray:
    b = np.asarray(b, np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# bf16 rounding
# --------------------------------------------------------------------------

def test_bf16_exhaustive_against_torch():
    """All 2^32 binary32 patterns: the oracle's round-to-nearest-even against
    torch's independent float -> bfloat16 conversion (NaNs compared as NaN)."""
    chunk = 1 << 25
    pat = np.arange(chunk, dtype=np.uint32)
    ours = np.empty(chunk, np.uint16)
    ref_t = torch.empty(chunk, dtype=torch.bfloat16)
    ref = ref_t.view(torch.int16).numpy().view(np.uint16)
    src = torch.from_numpy(pat.view(np.float32))
    f32b = oracle.lib().orc_f32bits_to_bf16
    for _ in range((1 << 32) // chunk):
        f32b(pat.ctypes.data, ours.ctypes.data, chunk)
        ref_t.copy_(src)
        if not np.array_equal(ours, ref):
            bad = ours != ref
            # the only allowed difference is the payload of a NaN
            nan_o = ((ours[bad] & 0x7F80) == 0x7F80) & ((ours[bad] & 0x7F) != 0)
            nan_r = ((ref[bad] & 0x7F80) == 0x7F80) & ((ref[bad] & 0x7F) != 0)
            assert (nan_o & nan_r).all(), f"mismatch at pattern {int(pat[bad][~(nan_o & nan_r)][0]):#010x}"
        pat += np.uint32(chunk)


def test_bf16_from_f64_brute_force():
    """binary64 inputs (not representable in binary32): the result is the
    nearest of all bf16 values, ties to the even pattern, found by brute
    force over the two bracketing bf16 bit patterns."""
    r = np.random.default_rng(1)
    xs = list(r.standard_normal(4000) * np.exp(r.uniform(-30, 30, 4000)))
    # exact half-way points between neighbours, and neighbours +- tiny
    for b in [0x3F80, 0x3F81, 0x4049, 0x0001, 0x0080, 0x7F7E, 0x7F7F, 0xBF80]:
        lo, hi = bf16_val(b), bf16_val(b + 1)
        mid = (lo + hi) / 2
        xs += [mid, math.nextafter(mid, math.inf), math.nextafter(mid, -math.inf)]
    for x in xs:
        got = oracle.f64_to_bf16(x)
        ax = abs(x)
        # all non-negative finite bf16 values in order of their bit patterns
        cand = np.arange(0, 0x7F80, dtype=np.uint16)
        vals = bf16_val(cand)
        i = int(np.searchsorted(vals, ax))
        best = None
        for j in (i - 1, i):
            if 0 <= j < len(vals):
                dist = abs(vals[j] - ax)
                if best is None or dist < best[0] or (dist == best[0] and cand[j] % 2 == 0):
                    best = (dist, int(cand[j]))
        if i == len(vals):   # above max finite: overflow threshold is max + half ulp
            mx = vals[-1]
            half = (mx - vals[-2]) / 2
            exp_bits = 0x7F80 if ax >= mx + half else 0x7F7F
        else:
            exp_bits = best[1]
        if x < 0:
            exp_bits |= 0x8000
        assert got == exp_bits, (x, hex(got), hex(exp_bits))


# --------------------------------------------------------------------------
# Operators
# --------------------------------------------------------------------------

def _half_ulp_ok(got_bits, ref):
    """got is a correctly rounded bf16 of ref (within half a bf16 ulp)."""
    got = bf16_val(got_bits)
    ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-300))) - 7)
    return np.all(np.abs(got - ref) <= 0.5 * ulp * (1 + 1e-9))


def test_rmsnorm_closed_forms():
    H, eps = 256, 1e-6
    g = bf16_bits_of(1 + 0.02 * np.random.default_rng(0).standard_normal(H))
    for c in (1.0, -3.5, 1e-3, 7.25):
        y = oracle.rmsnorm(np.full(H, c, np.float32), g, eps)
        ref = np.float64(np.float32(c)) / math.sqrt(np.float64(np.float32(c)) ** 2 + eps) * bf16_val(g)
        assert _half_ulp_ok(y, ref)
    x = np.zeros(H, np.float32)
    x[17] = 5.0
    y = oracle.rmsnorm(x, g, eps)
    assert np.all(bf16_val(y)[np.arange(H) != 17] == 0)
    assert _half_ulp_ok(y[17:18], np.array([5.0 / math.sqrt(25.0 / H + eps) * bf16_val(g[17])]))


def test_rmsnorm_against_torch():
    r = np.random.default_rng(2)
    for H in (64, 256, 4096):
        x = (r.standard_normal(H) * 3).astype(np.float32)
        g = bf16_bits_of(1 + 0.02 * r.standard_normal(H))
        ref = F.rms_norm(torch.from_numpy(x).double(), (H,), weight=torch.from_numpy(bf16_val(g)),
                         eps=1e-6).numpy()
        assert _half_ulp_ok(oracle.rmsnorm(x, g, 1e-6), ref)


def test_linear_identity_onehot_and_torch():
    r = np.random.default_rng(3)
    n = 64
    I = bf16_bits_of(np.eye(n))
    h = bf16_bits_of(r.standard_normal(n))
    assert np.array_equal(oracle.linear(h, I), bf16_val(h))
    W = bf16_bits_of(r.standard_normal((48, n)))
    e = np.zeros(n)
    e[5] = 1.0
    assert np.array_equal(oracle.linear(bf16_bits_of(e), W), bf16_val(W[:, 5]))
    for (o, i) in ((48, 64), (300, 688), (17, 4096)):
        W = bf16_bits_of(r.standard_normal((o, i)) * 0.02)
        h = bf16_bits_of(r.standard_normal(i))
        ref = (torch.from_numpy(bf16_val(W)) @ torch.from_numpy(bf16_val(h))).numpy()
        np.testing.assert_allclose(oracle.linear(h, W), ref, rtol=1e-12, atol=1e-14)


def test_rope_pins():
    d, theta = 64, 10000.0
    r = np.random.default_rng(4)
    x = r.standard_normal(d)
    assert np.array_equal(oracle.rope(x, 0, theta), x)            # position 0 is the identity
    e0 = np.zeros(d)
    e0[0] = 1.0
    for p in (1, 5, 1000, 32767):                                  # pair 0 turns by p radians
        y = oracle.rope(e0, p, theta)
        exp = np.zeros(d)
        exp[0], exp[d // 2] = np.cos(p), np.sin(p)
        np.testing.assert_allclose(y, exp, atol=1e-12)
    eq = np.zeros(d)
    eq[d // 4] = 1.0                                               # theta^(-1/2) = 0.01 rad per step
    y = oracle.rope(eq, 100, theta)
    np.testing.assert_allclose([y[d // 4], y[d // 4 + d // 2]], [np.cos(1.0), np.sin(1.0)], atol=1e-12)
    for p in (3, 77, 4095):                                        # rotation preserves pair norms
        y = oracle.rope(x, p, theta)
        n0 = x[: d // 2] ** 2 + x[d // 2:] ** 2
        n1 = y[: d // 2] ** 2 + y[d // 2:] ** 2
        np.testing.assert_allclose(n1, n0, rtol=1e-12)
    np.testing.assert_allclose(oracle.rope(oracle.rope(x, 11, theta), 30, theta),
                               oracle.rope(x, 41, theta), atol=1e-10)
    k = r.standard_normal(d)
    base = np.dot(oracle.rope(x, 50, theta), oracle.rope(k, 20, theta))
    for s in (1, 100, 2000):                                       # depends only on m - n
        np.testing.assert_allclose(np.dot(oracle.rope(x, 50 + s, theta), oracle.rope(k, 20 + s, theta)),
                                   base, rtol=1e-9)


def test_attention_pins():
    r = np.random.default_rng(5)
    d = 64
    q = bf16_bits_of(r.standard_normal(d))
    K = bf16_bits_of(r.standard_normal((1, d)))
    V = bf16_bits_of(r.standard_normal((1, d)))
    assert np.array_equal(oracle.attention(q, K, V), bf16_val(V[0]))        # one key -> its value
    n = 37
    K = bf16_bits_of(r.standard_normal((n, d)))
    V = bf16_bits_of(r.standard_normal((n, d)))
    zero_q = np.zeros(d, np.uint16)                                          # equal scores -> mean
    np.testing.assert_allclose(oracle.attention(zero_q, K, V), bf16_val(V).mean(0), rtol=1e-12)
    Vsame = np.repeat(V[:1], n, axis=0)                                      # identical values
    np.testing.assert_allclose(oracle.attention(q, K, Vsame), bf16_val(V[0]), rtol=1e-13)
    # two keys whose scores differ by ln 3 -> weights 1/4 and 3/4
    qv = np.zeros(d)
    qv[0] = 1.0
    K2 = np.zeros((2, d))
    K2[1, 0] = math.log(3.0) * math.sqrt(d)
    Kb = bf16_bits_of(K2)
    gap = bf16_val(Kb[1, 0]) / math.sqrt(d)
    w1 = math.exp(gap) / (1 + math.exp(gap))
    V2 = bf16_bits_of(r.standard_normal((2, d)))
    np.testing.assert_allclose(oracle.attention(bf16_bits_of(qv), Kb, V2),
                               (1 - w1) * bf16_val(V2[0]) + w1 * bf16_val(V2[1]), rtol=1e-12)
    assert abs(w1 - 0.75) < 2e-3
    for n in (1, 2, 129, 1000):
        q = bf16_bits_of(r.standard_normal(d))
        K = bf16_bits_of(r.standard_normal((n, d)))
        V = bf16_bits_of(r.standard_normal((n, d)))
        ref = F.scaled_dot_product_attention(torch.from_numpy(bf16_val(q))[None, None, None],
                                             torch.from_numpy(bf16_val(K))[None, None],
                                             torch.from_numpy(bf16_val(V))[None, None])[0, 0, 0]
        np.testing.assert_allclose(oracle.attention(q, K, V), ref.numpy(), rtol=1e-11, atol=1e-13)


def test_silu_and_argmax():
    assert oracle.silu(0.0) == 0.0
    for z in np.linspace(-30, 30, 61):
        assert abs(oracle.silu(z) - F.silu(torch.tensor(z, dtype=torch.float64)).item()) <= 1e-15 * max(1, abs(z))
    v = np.zeros(100, np.float32)
    v[42] = 1.0
    assert oracle.argmax_f32(v) == 42
    v[:] = 0.5
    assert oracle.argmax_f32(v) == 0                # all tied -> lowest index
    v[7] = v[70] = 2.0
    assert oracle.argmax_f32(v) == 7
    r = np.random.default_rng(6)
    for _ in range(50):
        w = r.standard_normal(1000).astype(np.float32)
        w[r.integers(0, 1000, 3)] = w.max()         # crafted ties at the maximum
        assert oracle.argmax_f32(w) == int(np.argmax(w))   # numpy: first occurrence


def test_route_pins():
    sel, w = oracle.route(np.zeros(16), 4)          # equal logits: lowest ids, equal weights
    assert list(sel) == [0, 1, 2, 3] and np.allclose(w, 0.25)
    logits = np.zeros(16)
    logits[9] = 50.0
    sel, w = oracle.route(logits, 1)                # one dominant expert, weight exactly 1
    assert list(sel) == [9] and w[0] == 1.0
    r = np.random.default_rng(7)
    for E, k in ((16, 4), (128, 8)):
        lg = r.standard_normal(E)
        sel, w = oracle.route(lg, k)
        p = torch.softmax(torch.from_numpy(lg), -1)
        tp, te = torch.topk(p, k)
        assert list(sel) == te.tolist()
        np.testing.assert_allclose(w, (tp / tp.sum()).numpy(), rtol=1e-12)


def test_fig3_sum_trees_golden():
    """Sec. III, Fig. 3: two reduction trees of one row give different
    binary32 results (the premise behind every invariance test)."""
    path = os.path.join(os.path.dirname(__file__), "golden", "fig3_sum_trees.txt")
    rows = [ln.split() for ln in open(path) if ln.strip() and not ln.startswith("#")]
    for row in rows:
        a, b, c, d, split, seq = [np.frombuffer(bytes.fromhex(h)[::-1], np.float32)[0] for h in row]
        f = np.float32
        assert f(f(a + b) + f(c + d)) == split
        assert f(f(f(a + b) + c) + d) == seq
        assert split != seq


# --------------------------------------------------------------------------
# Whole step
# --------------------------------------------------------------------------

def _host_model(W: wl.Weights) -> oracle.Model:
    b = wl.bits
    return oracle.Model(W.cfg, b(W.embed), b(W.final_norm), b(W.lm_head),
                        [b(t) for t in W.attn_norm], [b(t) for t in W.w_qkv], [b(t) for t in W.w_o],
                        [b(t) for t in W.mlp_norm], [b(t) for t in W.w_gate_up],
                        [b(t) for t in W.w_down], [b(t) for t in W.w_router],
                        [b(t) for t in W.w_exp_gate_up], [b(t) for t in W.w_exp_down])


def _contig_kv(cfg, slots, S, seed):
    K, V = wl.make_kv_contiguous(cfg, slots, S, seed)
    return oracle.KVCache([wl.bits(t) for t in K], [wl.bits(t) for t in V], oracle.KV_CONTIGUOUS,
                          slots, S)


@pytest.mark.parametrize("name", ["tiny", "tiny_moe"])
def test_decode_row_against_torch_composition(name):
    cfg = wl.config(name)
    W = wl.make_weights(cfg, seed=3)
    m = _host_model(W)
    S, slot, pos = 64, 1, 23
    kv = _contig_kv(cfg, 2, S, seed=4)
    kpre = [torch.from_numpy(np.ascontiguousarray(k[slot, :, :pos]).view(np.int16)).view(torch.bfloat16) for k in kv.k]
    vpre = [torch.from_numpy(np.ascontiguousarray(v[slot, :, :pos]).view(np.int16)).view(torch.bfloat16)
            for v in kv.v]
    tok = 517
    logits = oracle.decode_row(m, kv, slot, tok, pos)
    ref, kn, vn = tref.forward_chunk(cfg, W, [tok], pos, kpre, vpre)
    scale = np.abs(ref.numpy()).max()
    assert np.abs(logits - ref.numpy()[0]).max() <= 1e-10 * scale
    for l in range(cfg["n_layers"]):   # the appended KV entries are the same bf16 values
        assert np.array_equal(kv.k[l][slot, :, pos], wl.bits(kn[l][:, 0]))
        assert np.array_equal(kv.v[l][slot, :, pos], wl.bits(vn[l][:, 0]))


@pytest.mark.parametrize("name", ["tiny", "tiny_moe"])
def test_prefill_against_torch_composition(name):
    cfg = wl.config(name)
    W = wl.make_weights(cfg, seed=5)
    m = _host_model(W)
    Lp = 19
    kv = _contig_kv(cfg, 1, 32, seed=6)
    prompt = wl.make_prompt(cfg["vocab"], Lp, seed=7)
    logits, tok = oracle.prefill(m, kv, 0, prompt)
    empty = [torch.zeros(cfg["n_kv_heads"], 0, cfg["head_dim"], dtype=torch.bfloat16)] * cfg["n_layers"]
    ref, kn, vn = tref.forward_chunk(cfg, W, prompt, 0, empty, empty)
    ref_last = ref.numpy()[-1]
    assert np.abs(logits - ref_last).max() <= 1e-10 * np.abs(ref_last).max()
    assert tok == int(np.argmax(ref_last.astype(np.float32)))
    for l in range(cfg["n_layers"]):
        assert np.array_equal(kv.k[l][0, :, :Lp], wl.bits(kn[l]))
        assert np.array_equal(kv.v[l][0, :, :Lp], wl.bits(vn[l]))


def test_decode_equals_prefill_bitwise():
    """prefill(p ++ [t]) at its last row == prefill(p) then decode(t)."""
    cfg = wl.config("tiny")
    m = _host_model(wl.make_weights(cfg, seed=8))
    p = wl.make_prompt(cfg["vocab"], 12, seed=9)
    t = 333
    kv1 = _contig_kv(cfg, 1, 16, seed=10)
    l1, _ = oracle.prefill(m, kv1, 0, np.append(p, t))
    kv2 = _contig_kv(cfg, 1, 16, seed=11)
    oracle.prefill(m, kv2, 0, p)
    l2 = oracle.decode_row(m, kv2, 0, t, len(p))
    assert np.array_equal(l1, l2)
    for l in range(cfg["n_layers"]):
        assert np.array_equal(kv1.k[l][0, :, :13], kv2.k[l][0, :, :13])
        assert np.array_equal(kv1.v[l][0, :, :13], kv2.v[l][0, :, :13])


def test_paged_equals_contiguous_bitwise():
    cfg = wl.config("tiny")
    m = _host_model(wl.make_weights(cfg, seed=12))
    S, ps, slots = 64, 16, 3
    ckv = _contig_kv(cfg, slots, S, seed=13)
    mpp = S // ps
    num_pages = slots * mpp + 5
    pt = wl.make_page_table(slots, mpp, num_pages, seed=14)
    pk, pv = [], []
    for l in range(cfg["n_layers"]):      # scatter the same contents into permuted pages
        k = np.zeros((num_pages, cfg["n_kv_heads"], ps, cfg["head_dim"]), np.uint16)
        v = np.zeros((num_pages, cfg["n_kv_heads"], ps, cfg["head_dim"]), np.uint16)
        for s_ in range(slots):
            for j in range(mpp):
                k[pt[s_, j]] = ckv.k[l][s_, :, j * ps:(j + 1) * ps]
                v[pt[s_, j]] = ckv.v[l][s_, :, j * ps:(j + 1) * ps]
        pk.append(k)
        pv.append(v)
    pkv = oracle.KVCache(pk, pv, oracle.KV_PAGED, slots, S, ps, num_pages, mpp, pt)
    batch = wl.make_batch(slots, cfg["vocab"], seed=15, len_lo=10, len_hi=60, n_live=slots)
    la, na = oracle.decode_batch(m, ckv, batch.tokens, batch.valid, batch.seq_lens)
    lb, nb = oracle.decode_batch(m, pkv, batch.tokens, batch.valid, batch.seq_lens)
    assert np.array_equal(la, lb) and np.array_equal(na, nb)


def test_gqa_equals_mha_with_duplicated_kv_heads():
    cfg = wl.config("tiny")
    W = wl.make_weights(cfg, seed=16)
    nq, nkv, d = cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    cfg_mha = dict(cfg, n_kv_heads=nq)
    W2 = wl.make_weights(cfg, seed=16)
    W2.cfg = cfg_mha
    rep = nq // nkv
    for l in range(cfg["n_layers"]):
        q = W.w_qkv[l][: nq * d]
        k = W.w_qkv[l][nq * d:(nq + nkv) * d].reshape(nkv, d, -1).repeat_interleave(rep, 0).reshape(nq * d, -1)
        v = W.w_qkv[l][(nq + nkv) * d:].reshape(nkv, d, -1).repeat_interleave(rep, 0).reshape(nq * d, -1)
        W2.w_qkv[l] = torch.cat([q, k, v]).contiguous()
    m1, m2 = _host_model(W), _host_model(W2)
    kv1 = _contig_kv(cfg, 1, 40, seed=17)
    kv2 = oracle.KVCache([np.ascontiguousarray(np.repeat(k, rep, axis=1)) for k in kv1.k],
                         [np.ascontiguousarray(np.repeat(v, rep, axis=1)) for v in kv1.v],
                         oracle.KV_CONTIGUOUS, 1, 40)
    a = oracle.decode_row(m1, kv1, 0, 77, 30)
    b = oracle.decode_row(m2, kv2, 0, 77, 30)
    assert np.array_equal(a, b)


def test_moe_top1_equals_dense_expert_bitwise():
    """A router with equal logits and top_k = 1 picks expert 0 with weight
    exactly 1, so the layer is the dense SwiGLU MLP of expert 0."""
    cm = wl.config("tiny_moe", top_k=1)
    Wm = wl.make_weights(cm, seed=18)
    for l in range(cm["n_layers"]):
        Wm.w_router[l] = torch.zeros_like(Wm.w_router[l])
    cd = wl.config("tiny", ffn=cm["expert_ffn"])
    Wd = wl.make_weights(cm, seed=18)
    Wd.cfg = cd
    Wd.w_gate_up = [Wm.w_exp_gate_up[l][0].contiguous() for l in range(cm["n_layers"])]
    Wd.w_down = [Wm.w_exp_down[l][0].contiguous() for l in range(cm["n_layers"])]
    Wd.w_router, Wd.w_exp_gate_up, Wd.w_exp_down = [], [], []
    kva = _contig_kv(cm, 1, 32, seed=19)
    kvb = _contig_kv(cm, 1, 32, seed=19)
    a = oracle.decode_row(_host_model(Wm), kva, 0, 5, 20)
    b = oracle.decode_row(_host_model(Wd), kvb, 0, 5, 20)
    assert np.array_equal(a, b)


def test_routed_decode_records_and_forcing():
    """The routing records and overrides of the MoE oracle, pinned three ways:
    * its router logits and own top-k equal those of the torch composition
      (matrix form, torch.topk on torch.softmax) at every layer;
    * forcing each layer to the oracle's own choice changes no bit;
    * forcing other expert sets (the 2nd..k+1-th ranked experts, a shuffled
      order) gives the torch composition run with the same sets."""
    cfg = wl.config("tiny_moe")
    W = wl.make_weights(cfg, seed=30)
    m = _host_model(W)
    L, E, k = cfg["n_layers"], cfg["n_experts"], cfg["top_k"]
    S, slot, pos, tok = 48, 0, 29, 211
    kv = _contig_kv(cfg, 1, S, seed=31)
    kpre = [torch.from_numpy(np.ascontiguousarray(x[slot, :, :pos]).view(np.int16)).view(torch.bfloat16) for x in kv.k]
    vpre = [torch.from_numpy(np.ascontiguousarray(x[slot, :, :pos]).view(np.int16))
            .view(torch.bfloat16) for x in kv.v]
    plain = oracle.decode_row(m, kv, slot, tok, pos)
    lg, rl, own = oracle.decode_row_routed(m, kv, slot, tok, pos)
    assert np.array_equal(lg, plain)
    routing = []
    ref, _, _ = tref.forward_chunk(cfg, W, [tok], pos, kpre, vpre, routing=routing)
    for l in range(L):
        trl, tsel = routing[l]
        np.testing.assert_allclose(rl[l], trl.numpy()[0], rtol=0, atol=1e-12 * np.abs(rl[l]).max())
        assert list(own[l]) == tsel[0].tolist(), l
    # the oracle's own choice, forced: bit-identical
    lg2, _, own2 = oracle.decode_row_routed(m, kv, slot, tok, pos, force=own)
    assert np.array_equal(lg2, plain) and np.array_equal(own2, own)
    # other sets: drop the top expert for the (k+1)-th, and reverse the order
    force = np.empty((L, k), np.int32)
    for l in range(L):
        order = np.argsort(-rl[l], kind="stable")
        force[l] = order[1:k + 1][::-1]
    lg3, rl3, own3 = oracle.decode_row_routed(m, kv, slot, tok, pos, force=force)
    ref3, _, _ = tref.forward_chunk(cfg, W, [tok], pos, kpre, vpre, force=force[:, None, :])
    scale = np.abs(ref3.numpy()).max()
    assert np.abs(lg3 - ref3.numpy()[0]).max() <= 1e-10 * scale
    assert np.abs(lg3 - plain).max() > 1e-6 * scale        # the forced sets do change the result
    assert np.array_equal(rl3[0], rl[0])                   # layer 0's router input is unchanged
    with pytest.raises(ValueError):                        # malformed sets are refused
        bad = own.copy()
        bad[0, 1] = bad[0, 0]
        oracle.decode_row_routed(m, kv, slot, tok, pos, force=bad)


def test_routed_prefill_matches_routed_decode_rows():
    """Forced prefill routing [L][Lp][k] is the per-position forced decode:
    the prefill of p with forced sets equals, at its last position, the
    forced decode of p's last token after the forced prefill of the rest
    (the routed form of decode == prefill), bit for bit; the records of both
    agree."""
    cfg = wl.config("tiny_moe")
    W = wl.make_weights(cfg, seed=32)
    m = _host_model(W)
    L, k = cfg["n_layers"], cfg["top_k"]
    Lp = 12
    prompt = wl.make_prompt(cfg["vocab"], Lp, seed=33)
    kva = _contig_kv(cfg, 1, 32, seed=34)
    _, _, rl, own = oracle.prefill_routed(m, kva, 0, prompt)
    force = np.empty_like(own)
    for l in range(L):
        for t in range(Lp):
            force[l, t] = np.argsort(-rl[l, t], kind="stable")[1:k + 1]
    kvb = _contig_kv(cfg, 1, 32, seed=34)
    la, ta, rla, owna = oracle.prefill_routed(m, kvb, 0, prompt, force=force)
    kvc = _contig_kv(cfg, 1, 32, seed=34)
    oracle.prefill_routed(m, kvc, 0, prompt[:-1], force=force[:, :-1])
    lb, rlb, ownb = oracle.decode_row_routed(m, kvc, 0, int(prompt[-1]), Lp - 1, force=force[:, -1])
    assert np.array_equal(la, lb)
    assert np.array_equal(rla[:, -1], rlb) and np.array_equal(owna[:, -1], ownb)
    for l in range(L):
        assert np.array_equal(kvb.k[l], kvc.k[l]) and np.array_equal(kvb.v[l], kvc.v[l])


def test_route_forced_weights():
    """Weights of a forced set: softmax over all experts, renormalised over
    the set (torch), in the set's order."""
    r = np.random.default_rng(35)
    lg = r.standard_normal(128)
    f = np.array([5, 77, 3, 120, 64, 9, 100, 31], np.int32)
    p = torch.softmax(torch.from_numpy(lg), -1)[torch.from_numpy(f).long()]
    np.testing.assert_allclose(oracle.route_forced(lg, f), (p / p.sum()).numpy(), rtol=1e-13)
    sel, w = oracle.route(lg, 8)
    assert np.array_equal(oracle.route_forced(lg, sel), w)   # the own choice: the same weights, bit for bit
    with pytest.raises(ValueError):
        oracle.route_forced(lg, np.array([1, 1], np.int32))
    with pytest.raises(ValueError):
        oracle.route_forced(lg, np.array([0, 128], np.int32))


def test_thread_count_invariance():
    cfg = wl.config("tiny")
    m = _host_model(wl.make_weights(cfg, seed=20))
    batch = wl.make_batch(4, cfg["vocab"], seed=21, len_lo=16, len_hi=128, n_live=4)
    outs = []
    n0 = oracle.get_threads()
    try:
        for n in (1, max(2, os.cpu_count() or 2)):
            oracle.set_threads(n)
            kv = _contig_kv(cfg, 4, 160, seed=22)
            outs.append(oracle.decode_batch(m, kv, batch.tokens, batch.valid, batch.seq_lens))
    finally:
        oracle.set_threads(n0)
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])


def test_padding_rows_ignored():
    """Padding rows (valid = 0) may carry any token and length; they get -1
    and do not change live rows (row-by-row definition)."""
    cfg = wl.config("tiny")
    m = _host_model(wl.make_weights(cfg, seed=23))
    b = wl.make_batch(4, cfg["vocab"], seed=24, len_lo=16, len_hi=100, n_live=2)
    kv = _contig_kv(cfg, 4, 128, seed=25)
    lg, nx = oracle.decode_batch(m, kv, b.tokens, b.valid, b.seq_lens)
    assert all(nx[i] == -1 for i in range(4) if not b.valid[i])
    assert all(0 <= nx[i] < cfg["vocab"] for i in range(4) if b.valid[i])
    assert np.isnan(lg[b.valid == 0]).all() and np.isfinite(lg[b.valid == 1]).all()
