"""corun_sample_noalloc, the allocation-free variant of corun_sample: on the
same logits and arguments it returns corun_sample's token and
log-probability bits, on two calls in a row (the second smaller: fewer rows,
a narrower vocabulary and another row stride), so nothing the first call
left in the shared static staging reaches the second; its size checks
reject what the staging cannot hold."""
import numpy as np
import pytest
import torch

from paper_2608_14376_amd import corun
from paper_2608_14376_amd import workload as wl
from tests.gpu_helpers import DEV, to_device

pytestmark = pytest.mark.gpu


def _args(rows, seed):
    r = np.random.default_rng(seed)
    valid = (r.random(rows) < 0.8).astype(np.uint8)
    valid[0] = 1
    pos = r.integers(0, 5000, rows).astype(np.int32)
    seeds = r.integers(0, 1 << 63, rows, dtype=np.uint64)
    temp = np.where(r.random(rows) < 0.3, 0.0, r.uniform(0.3, 1.5, rows)).astype(np.float32)
    return valid, pos, seeds, temp


def test_noalloc_sampler_matches_engine_sampler():
    cfg = wl.config("tiny")
    Wg = to_device(wl.make_weights(cfg, seed=90))
    B = 64
    K, V = wl.make_kv_contiguous(cfg, B, 32, seed=91, device=DEV)
    eng = corun.Engine(cfg, Wg, B, K, V)
    g = torch.Generator(device=DEV)
    g.manual_seed(92)
    for rows, vocab, ld, seed in ((64, 1024, 1024, 93), (17, 640, 700, 94)):
        logits = (3.0 * torch.randn(rows, ld, generator=g, device=DEV)).contiguous()
        valid, pos, seeds, temp = _args(rows, seed)
        # the engine's sampler samples `vocab` = the model's 1024 columns; give it
        # a copy whose columns past `vocab` can never win (-inf) for the narrow case
        ref_in = logits.clone()
        if vocab < cfg["vocab"]:
            ref_in = torch.full((rows, cfg["vocab"]), float("-inf"), device=DEV)
            ref_in[:, :vocab] = logits[:, :vocab]
        tok_a, lp_a = eng.sample(ref_in.contiguous(), valid, pos, seeds, temp)
        tok_b, lp_b = corun.sample_noalloc(logits, valid, pos, seeds, temp, vocab=vocab)
        assert np.array_equal(tok_a, tok_b), (rows, vocab)
        assert np.array_equal(lp_a.view(np.int32), lp_b.view(np.int32)), (rows, vocab)
        assert (tok_b[valid == 0] == -1).all() and (tok_b[valid == 1] < vocab).all()
    eng.close()


def test_noalloc_sampler_rejects_oversized_calls():
    logits = torch.zeros(corun.SAMPLE_NOALLOC_MAX_ROWS + 1, 16, device=DEV)
    n = logits.shape[0]
    with pytest.raises(corun.CorunError) as ei:
        corun.sample_noalloc(logits, np.ones(n), np.zeros(n), np.zeros(n), np.zeros(n))
    assert ei.value.status == corun.E_SHAPE
    small = torch.zeros(2, 16, device=DEV)
    with pytest.raises(corun.CorunError) as ei:
        corun.sample_noalloc(small, np.ones(2), np.zeros(2), np.zeros(2), np.zeros(2), vocab=17)
    assert ei.value.status == corun.E_SHAPE
