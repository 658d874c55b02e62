"""Chunked isolated prefill (corun_prefill_chunk; Sec. IV, "Isolated
Prefill": a long prompt divided into fixed-size chunks that run alone, one
iteration each, in order).

* Against the oracle's prefill of the whole prompt.  The chunk boundaries
  change nothing in the definition (every position attends to its prefix;
  the cached k/v are the same bf16 storage points), so the same tolerance
  applies: the last position's logits to 2e-2 relative, every cached k and
  v position to 2e-2 of the layer's largest value, the greedy token unless
  a near tie.  Chunk sizes split the 32-query blocks and 64-key tiles
  unevenly (64, 100, and 333 = one chunk), on small128 (head_dim 128),
  tiny (head_dim 64) and the tiny mixture of experts, contiguous and paged.
* Determinism: the same chunk sequence into another slot, after other
  traffic, gives bit-identical k/v and logits.
* One chunk at start 0 is corun_prefill, bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_14376_amd import corun
from paper_2608_14376_amd import workload as wl
from tests.gpu_helpers import DEV, check_routing, check_tokens, host_model, oracle_kv, row_rel_err, to_device

pytestmark = pytest.mark.gpu
TOL = 2e-2
CAP = 400
LP = 333
PS = 16


@pytest.fixture(scope="module", params=["small128", "tiny", "tiny_moe"])
def model(request):
    cfg = wl.config(request.param)
    Wc = wl.make_weights(cfg, seed=41)
    return cfg, to_device(Wc), host_model(Wc)


def chunked(eng, prompt, slot, C, last, trace=None):
    """Run `prompt` as chunks of C tokens (the last shorter), in order.
    trace (a list, mixture of experts): receives each chunk's routing record."""
    start, tok = 0, None
    while start < len(prompt):
        n = min(C, len(prompt) - start)
        fin = start + n == len(prompt)
        tok = eng.prefill_chunk(prompt[start:start + n], start, slot, last if fin else None, want_token=fin)
        if trace is not None:
            trace.append(eng.routing_trace(1))
        start += n
    return tok


def oracle_prefill(cfg, m, okv, slot, prompt, trace):
    """The oracle's whole-prompt prefill; for a mixture of experts it follows
    the GPU's expert sets (the chunks' routing records, in order) where
    check_routing admits them as near-ties.  Returns the last logits."""
    if not cfg["n_experts"]:
        return oracle.prefill(m, okv, slot, prompt)[0]
    gsel = np.concatenate([t[0] for t in trace], axis=1)
    glog = np.concatenate([t[1] for t in trace], axis=1)
    assert gsel.shape[1] == len(prompt)
    ref, _, rl, own = oracle.prefill_routed(m, okv, slot, prompt, force=gsel)
    ties = []
    for t in range(len(prompt)):
        ties += check_routing(gsel[:, t], glog[:, t], rl[:, t], own[:, t], t)
    print(f"routing near-ties followed: {ties}")
    return ref


def contiguous(cfg, B, seed):
    K, V = wl.make_kv_contiguous(cfg, B, CAP, seed)
    return [k.to(DEV) for k in K], [v.to(DEV) for v in V]


def bf16_as_f32(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32)


def check_kv_against_oracle(cfg, gpu_k, gpu_v, okv, slot_sel):
    """Every cached position of the prompt, k and v, within TOL of the
    layer's largest oracle value.  slot_sel maps an array to the prompt's
    [nkv, LP, d] view (k and v alike)."""
    for l in range(cfg["n_layers"]):
        for g, o, axis in ((gpu_k[l], okv.k[l], "k"), (gpu_v[l], okv.v[l], "v")):
            a = bf16_as_f32(slot_sel(wl.bits(g), axis))
            b = bf16_as_f32(slot_sel(o, axis))
            err = np.abs(a - b).max(axis=(0, 2))
            bad = np.nonzero(err > TOL * np.abs(b).max())[0]
            assert bad.size == 0, (l, axis, bad[:8].tolist(), float(err.max()))


@pytest.mark.parametrize("C", [64, 100, LP])
def test_chunked_prefill_matches_oracle(model, C):
    cfg, Wg, m = model
    K, V = contiguous(cfg, 4, 990)
    okv = oracle_kv(K, V)
    # the prefill workspace only needs one chunk
    moe = bool(cfg["n_experts"])
    eng = corun.Engine(cfg, Wg, 4, K, V, opt=corun.options(max_prefill_len=C, record_routing=moe))
    prompt = wl.make_prompt(cfg["vocab"], LP, seed=991)
    last = torch.empty(cfg["vocab"], dtype=torch.float32, device=DEV)
    trace = []
    tok = chunked(eng, prompt, 1, C, last, trace if moe else None)
    ref = oracle_prefill(cfg, m, okv, 1, prompt, trace)
    g = last.cpu().numpy()
    assert row_rel_err(g, ref) <= TOL
    check_tokens([tok], ref[None], g[None], [1], [])
    check_kv_against_oracle(cfg, K, V, okv, lambda a, ax: a[1, :, :LP])
    eng.close()


def test_chunked_prefill_paged_matches_oracle(model):
    """Chunks of 100 cross the 16-token pages of a permuted page table."""
    cfg, Wg, m = model
    mpp = CAP // PS
    num_pages = 4 * mpp + 5
    pt = wl.make_page_table(4, mpp, num_pages, seed=992)
    K, V = wl.make_kv_paged(cfg, num_pages, PS, seed=993)
    K = [k.to(DEV) for k in K]
    V = [v.to(DEV) for v in V]
    okv = oracle_kv(K, V, layout=oracle.KV_PAGED, page_size=PS, page_table=pt)
    moe = bool(cfg["n_experts"])
    eng = corun.Engine(cfg, Wg, 4, K, V, layout=corun.KV_PAGED, page_size=PS,
                       page_table=torch.from_numpy(pt).to(DEV),
                       opt=corun.options(max_prefill_len=100, record_routing=moe))
    prompt = wl.make_prompt(cfg["vocab"], LP, seed=994)
    last = torch.empty(cfg["vocab"], dtype=torch.float32, device=DEV)
    trace = []
    tok = chunked(eng, prompt, 2, 100, last, trace if moe else None)
    ref = oracle_prefill(cfg, m, okv, 2, prompt, trace)
    g = last.cpu().numpy()
    assert row_rel_err(g, ref) <= TOL
    check_tokens([tok], ref[None], g[None], [1], [])
    pages = pt[2, :(LP + PS - 1) // PS]

    def sel(a, ax):   # gather the slot's pages into position order, first LP positions
        return np.concatenate([a[p] for p in pages], axis=1)[:, :LP]
    check_kv_against_oracle(cfg, K, V, okv, sel)
    eng.close()


def test_chunked_prefill_is_deterministic_and_one_chunk_is_prefill(model):
    cfg, Wg, m = model
    K, V = contiguous(cfg, 4, 995)
    eng = corun.Engine(cfg, Wg, 4, K, V, opt=corun.options(max_prefill_len=LP))
    prompt = wl.make_prompt(cfg["vocab"], LP, seed=996)
    la = torch.empty(cfg["vocab"], dtype=torch.float32, device=DEV)
    lb = torch.empty_like(la)
    ta = chunked(eng, prompt, 0, 100, la)
    # other traffic: another prompt in slot 2, a decode step over every slot
    eng.prefill(wl.make_prompt(cfg["vocab"], 150, seed=997), 2, None)
    b = wl.make_batch(4, cfg["vocab"], seed=998, len_lo=16, len_hi=300)
    b.valid[0] = 0                                             # leave the first copy alone
    eng.decode_step(b.tokens, b.valid, b.seq_lens)
    tb = chunked(eng, prompt, 3, 100, lb)
    assert ta == tb and torch.equal(la.view(torch.int32), lb.view(torch.int32))
    for l in range(cfg["n_layers"]):
        assert torch.equal(K[l][0, :, :LP].view(torch.int16), K[l][3, :, :LP].view(torch.int16)), l
        assert torch.equal(V[l][0, :, :LP].view(torch.int16), V[l][3, :, :LP].view(torch.int16)), l
    # one chunk at start 0 is the whole-prompt prefill, bit for bit
    tc = eng.prefill(prompt, 1, la)
    td = eng.prefill_chunk(prompt, 0, 2, lb)
    assert tc == td and torch.equal(la.view(torch.int32), lb.view(torch.int32))
    for l in range(cfg["n_layers"]):
        assert torch.equal(K[l][1, :, :LP].view(torch.int16), K[l][2, :, :LP].view(torch.int16)), l
        assert torch.equal(V[l][1, :, :LP].view(torch.int16), V[l][2, :, :LP].view(torch.int16)), l
    eng.close()
