"""The decode step's QKV epilogue inside the attention kernel (qkv_epilogue
= 2; the default for B <= 8) against the same epilogue as its own kernel
(qkv_epilogue = 1):
every block rebuilds its group's q from the QKV split partials, and the
block holding the new token makes that token's k and v, appends them to the
cache and patches them into the step tile it has just loaded.  Both run the
same device function in the same order, so decode must be bit-identical:
logits, greedy tokens and the whole cache over three steps.

* small128 (head_dim 128) and tiny (head_dim 64), the tiny mixture of
  experts; B = 1, 5 and 40 (split-K 1 to 8 on the QKV projection);
* contiguous and paged caches;
* a 256-token attention chunk, so that the new token often sits in a later
  128-token step of its split than the first."""
import numpy as np
import pytest
import torch

from paper_2608_14376_amd import corun
from paper_2608_14376_amd import workload as wl
from tests.gpu_helpers import DEV, to_device

pytestmark = pytest.mark.gpu
CAP = 400
PS = 16


@pytest.fixture(scope="module", params=["small128", "tiny", "tiny_moe"])
def model(request):
    cfg = wl.config(request.param)
    return cfg, to_device(wl.make_weights(cfg, seed=71))


def caches(cfg, B, paged):
    if not paged:
        K, V = wl.make_kv_contiguous(cfg, B, CAP, seed=710)
        return [k.to(DEV) for k in K], [v.to(DEV) for v in V], {}
    mpp = CAP // PS
    num_pages = B * mpp + 3
    pt = wl.make_page_table(B, mpp, num_pages, seed=711)
    K, V = wl.make_kv_paged(cfg, num_pages, PS, seed=712)
    return ([k.to(DEV) for k in K], [v.to(DEV) for v in V],
            dict(layout=corun.KV_PAGED, page_size=PS, page_table=torch.from_numpy(pt).to(DEV)))


def run(cfg, Wg, B, paged, where, chunk):
    K, V, kw = caches(cfg, B, paged)
    eng = corun.Engine(cfg, Wg, B, K, V, opt=corun.options(qkv_epilogue=where, attn_chunk=chunk), **kw)
    b = wl.make_batch(B, cfg["vocab"], seed=713, len_lo=16, len_hi=CAP - 4)
    logits = torch.empty(B, cfg["vocab"], dtype=torch.float32, device=DEV)
    tok, seq, out = b.tokens.copy(), b.seq_lens.copy(), []
    for _ in range(3):
        nxt = eng.decode_step(tok, b.valid, seq, logits)
        out.append((nxt.copy(), logits.clone().view(torch.int32)))
        tok = np.where(b.valid == 1, nxt, tok).astype(np.int32)
        seq = seq + b.valid.astype(np.int32)
    eng.close()
    return out, [k.view(torch.int16) for k in K], [v.view(torch.int16) for v in V]


@pytest.mark.parametrize("paged", [False, True])
@pytest.mark.parametrize("B,chunk", [(1, 0), (5, 256), (40, 0)])
def test_fused_qkv_epilogue_is_bit_identical(model, B, chunk, paged):
    cfg, Wg = model
    fused = run(cfg, Wg, B, paged, 2, chunk)
    split = run(cfg, Wg, B, paged, 1, chunk)
    for (na, la), (nb, lb) in zip(fused[0], split[0]):
        assert np.array_equal(na, nb)
        assert torch.equal(la, lb)
    for l in range(cfg["n_layers"]):
        assert torch.equal(fused[1][l], split[1][l]), ("k", l)
        assert torch.equal(fused[2][l], split[2][l]), ("v", l)
