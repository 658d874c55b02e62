"""Batched prefill with batch-invariant kernels (corun_prefill_batch; Sec.
VIII, "Batch-Invariant Kernels for Prefill": prefill batches run through
batch-invariant kernels while decode keeps its fixed-shape kernels).

* Every prompt of a batch gets k/v and last-position logits bit-identical
  to its own corun_prefill on the same engine, in another slot, whatever
  its batch-mates and their order: small128 (head_dim 128, the pipelined
  projections), tiny (head_dim 64, a K tail) and the two small mixtures
  of experts.
* Against the oracle (relative 2e-2 on the logits, greedy token unless a
  near tie).
* Refusals: an engine without batch-invariant prefill, a slot given twice,
  more tokens than the prefill workspace.
"""
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
B = 10
LENS = [1, 33, 200, 64, 17]


@pytest.fixture(scope="module", params=["small128", "tiny", "tiny_moe", "small_moe"])
def model(request):
    cfg = wl.config(request.param)
    Wc = wl.make_weights(cfg, seed=51)
    return cfg, to_device(Wc), host_model(Wc)


def engine(cfg, Wg, seed, bi_prefill=True, pf=512):
    K, V = wl.make_kv_contiguous(cfg, B, CAP, seed)
    K = [k.to(DEV) for k in K]
    V = [v.to(DEV) for v in V]
    eng = corun.Engine(cfg, Wg, B, K, V, opt=corun.options(max_prefill_len=pf, bi_prefill=bi_prefill))
    return eng, K, V


def kv_bits(K, V, slot, n):
    return [(k[slot, :, :n].clone().view(torch.int16), v[slot, :, :n].clone().view(torch.int16))
            for k, v in zip(K, V)]


def same(a, b):
    return all(torch.equal(x[0], y[0]) and torch.equal(x[1], y[1]) for x, y in zip(a, b))


def test_batched_prefill_is_bit_identical_to_isolated(model):
    cfg, Wg, m = model
    V_ = cfg["vocab"]
    prompts = [wl.make_prompt(V_, L, seed=520 + i) for i, L in enumerate(LENS)]
    eng, K, V = engine(cfg, Wg, 521)
    lg = torch.empty(len(prompts), V_, dtype=torch.float32, device=DEV)
    toks = eng.prefill_batch(prompts, [0, 1, 2, 3, 4], lg)
    batched = [(int(toks[i]), lg[i].clone(), kv_bits(K, V, i, L)) for i, L in enumerate(LENS)]
    # each prompt alone, in slot 9
    last = torch.empty(V_, dtype=torch.float32, device=DEV)
    for i, p in enumerate(prompts):
        t = eng.prefill(p, 9, last)
        assert t == batched[i][0], i
        assert torch.equal(last.view(torch.int32), batched[i][1].view(torch.int32)), i
        assert same(kv_bits(K, V, 9, LENS[i]), batched[i][2]), i
    # other batch-mates and another order, other slots
    extra = wl.make_prompt(V_, 90, seed=529)
    lg2 = torch.empty(3, V_, dtype=torch.float32, device=DEV)
    toks2 = eng.prefill_batch([prompts[3], extra, prompts[0]], [6, 5, 8], lg2)
    for j, (i, slot) in enumerate(((3, 6), (0, 8))):
        row = 0 if j == 0 else 2
        assert int(toks2[row]) == batched[i][0]
        assert torch.equal(lg2[row].view(torch.int32), batched[i][1].view(torch.int32))
        assert same(kv_bits(K, V, slot, LENS[i]), batched[i][2])
    eng.close()


def test_batched_prefill_against_the_oracle(model):
    cfg, Wg, m = model
    V_ = cfg["vocab"]
    prompts = [wl.make_prompt(V_, L, seed=530 + i) for i, L in enumerate((200, 45))]
    eng, K, V = engine(cfg, Wg, 531)
    okv = oracle_kv(K, V)
    lg = torch.empty(2, V_, dtype=torch.float32, device=DEV)
    toks = eng.prefill_batch(prompts, [3, 7], lg)
    for i, (p, slot) in enumerate(zip(prompts, (3, 7))):
        ref, _ = oracle.prefill(m, okv, slot, p)
        g = lg[i].cpu().numpy()
        assert row_rel_err(g, ref) <= TOL, i
        check_tokens([int(toks[i])], ref[None], g[None], [1], [])
    eng.close()


def test_batched_prefill_refusals(model):
    cfg, Wg, m = model
    V_ = cfg["vocab"]
    p = [wl.make_prompt(V_, 40, seed=540), wl.make_prompt(V_, 30, seed=541)]
    plain, _, _ = engine(cfg, Wg, 542, bi_prefill=False)
    with pytest.raises(corun.CorunError):
        plain.prefill_batch(p, [0, 1])
    plain.close()
    eng, _, _ = engine(cfg, Wg, 543, pf=64)
    with pytest.raises(corun.CorunError):
        eng.prefill_batch(p, [2, 2])                      # slot twice
    with pytest.raises(corun.CorunError):
        eng.prefill_batch(p, [0, 1])                      # 70 tokens > 64
    assert len(eng.prefill_batch([p[0][:20], p[1]], [0, 1])) == 2
    eng.close()
