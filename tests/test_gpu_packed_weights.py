"""Tile-packed weight copies (corun_options.no_weight_pack = 0, the
default): for plans of up to 64 rows the engine streams its projections from
a copy laid out in contiguous 128 x 64 tiles.  The kernel meets the same
elements in the same order, so everything must be bit-identical to an engine
that reads the caller's row-major weights:

* decode logits, greedy tokens and appended k/v over two steps at B = 1, 24
  and 48 (32- and 64-row tiles; split-K on the narrow projections; at B = 1
  with the small-batch layer off, which would otherwise stream copies of
  its own: tests/test_gpu_small_batch_layer.py);
* prefill of a 40-token prompt (its projections take the packed copies) and
  a 100-token prompt (they do not; the last-row lm_head does);
* the packed copies exist: creating the engine takes the memory they need
  (small128).

small128 (every K a multiple of 64), tiny (down K = 688 stays row-major),
the tiny mixture of experts (router, attention, lm_head and expert gate/up
packed) and small_moe (expert down packed too, SwiGLU fused into the expert
gate/up)."""
import numpy as np
import pytest
import torch

from paper_2608_14376_amd import corun
from paper_2608_14376_amd import workload as wl
from tests.gpu_helpers import DEV, to_device

pytestmark = pytest.mark.gpu
CAP = 256


@pytest.fixture(scope="module", params=["small128", "tiny", "tiny_moe", "small_moe"])
def model(request):
    cfg = wl.config(request.param)
    return cfg, to_device(wl.make_weights(cfg, seed=61))


def engine(cfg, Wg, B, pack):
    K, V = wl.make_kv_contiguous(cfg, B, CAP, seed=610)
    K = [k.to(DEV) for k in K]
    V = [v.to(DEV) for v in V]
    eng = corun.Engine(cfg, Wg, B, K, V, opt=corun.options(max_prefill_len=128, no_weight_pack=not pack,
                                                           small_batch_layer=2))
    return eng, K, V


def bits(t):
    return t.view(torch.int32) if t.dtype == torch.float32 else t.view(torch.int16)


@pytest.mark.parametrize("B", [1, 24, 48])
def test_packed_decode_is_bit_identical(model, B):
    cfg, Wg = model
    runs = []
    for pack in (True, False):
        eng, K, V = engine(cfg, Wg, B, pack)
        b = wl.make_batch(B, cfg["vocab"], seed=611, len_lo=16, len_hi=CAP - 4)
        logits = torch.empty(B, cfg["vocab"], dtype=torch.float32, device=DEV)
        out = []
        tok, seq = b.tokens.copy(), b.seq_lens.copy()
        for _ in range(2):
            nxt = eng.decode_step(tok, b.valid, seq, logits)
            out.append((nxt.copy(), logits.clone()))
            tok = np.where(b.valid == 1, nxt, tok).astype(np.int32)
            seq = seq + b.valid.astype(np.int32)
        runs.append((out, [k.clone() for k in K], [v.clone() for v in V]))
        eng.close()
    (oa, Ka, Va), (ob, Kb, Vb) = runs
    for (na, la), (nb, lb) in zip(oa, ob):
        assert np.array_equal(na, nb)
        assert torch.equal(bits(la), bits(lb))
    for l in range(cfg["n_layers"]):
        assert torch.equal(bits(Ka[l]), bits(Kb[l])) and torch.equal(bits(Va[l]), bits(Vb[l])), l


@pytest.mark.parametrize("Lp", [40, 100])
def test_packed_prefill_is_bit_identical(model, Lp):
    cfg, Wg = model
    prompt = wl.make_prompt(cfg["vocab"], Lp, seed=612)
    res = []
    for pack in (True, False):
        eng, K, V = engine(cfg, Wg, 4, pack)
        last = torch.empty(cfg["vocab"], dtype=torch.float32, device=DEV)
        tok = eng.prefill(prompt, 2, last)
        res.append((tok, last.clone(), [k[2].clone() for k in K], [v[2].clone() for v in V]))
        eng.close()
    a, b = res
    assert a[0] == b[0] and torch.equal(bits(a[1]), bits(b[1]))
    for l in range(cfg["n_layers"]):
        assert torch.equal(bits(a[2][l]), bits(b[2][l])) and torch.equal(bits(a[3][l]), bits(b[3][l])), l


def packed_bytes(cfg):
    """What the B = 1 split-K plan packs: every projection with K % 64 == 0."""
    H, d = cfg["hidden"], cfg["head_dim"]
    nqkv = (cfg["n_heads"] + 2 * cfg["n_kv_heads"]) * d
    shapes = [(nqkv, H), (H, cfg["n_heads"] * d)]
    if cfg["n_experts"]:
        shapes.append((cfg["n_experts"], H))
    else:
        shapes += [(2 * cfg["ffn"], H), (H, cfg["ffn"])]
    per_layer = sum(-(-N // 128) * 128 * K * 2 for N, K in shapes if K % 64 == 0)
    return cfg["n_layers"] * per_layer + -(-cfg["vocab"] // 128) * 128 * H * 2


def test_packed_copies_are_made():
    """The engine's own allocations, with and without the copies (small128:
    the tiny models' copies fall below the allocator's 2 MB granularity)."""
    cfg = wl.config("small128")
    Wg = to_device(wl.make_weights(cfg, seed=62))
    K, V = wl.make_kv_contiguous(cfg, 1, CAP, seed=613)
    K = [k.to(DEV) for k in K]
    V = [v.to(DEV) for v in V]
    used = []
    for pack in (False, True):
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        eng = corun.Engine(cfg, Wg, 1, K, V, opt=corun.options(no_weight_pack=not pack, small_batch_layer=2))
        torch.cuda.synchronize()
        used.append(free0 - torch.cuda.mem_get_info()[0])
        eng.close()
    assert used[1] - used[0] >= packed_bytes(cfg)
