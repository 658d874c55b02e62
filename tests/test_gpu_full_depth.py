"""Full-depth parity: the whole 36-layer 8B-shaped decoder (hidden 4096,
32/8 heads of 128, FFN 12288, vocabulary 151936) against the oracle, at the
decode benchmark's plans and cache capacity, B = 1 and B = 256.

The other 8B parity tests run two-layer slices at the 2e-2 row-relative
tolerance.  Over 36 layers this random-weight model amplifies
rounding-level differences: one bf16 ulp added to a single element of the
input embedding moves the oracle's own logits by about 4e-2 (row-relative),
against under 1e-2 at two layers.  Two correct implementations that round
their bf16 storage points from different fp32/fp64 sums therefore drift apart
by that much too, so at full depth the bound is taken from that envelope,
measured on each sampled row:
    env = max over two single-element one-ulp input perturbations of
          row_rel_err(oracle_perturbed, oracle),
    GPU error <= max(2e-2, 2 env).
The GPU's batch-invariant plan (no split-K, other tiles: a second valid
summation order) is held to the same bound and its distance to the default
plan is printed beside it.

Sampled live rows are recomputed by the oracle row by row from a host copy of
their own cache taken before the step (about 0.6 GB per row)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_14376_amd import corun
from paper_2608_14376_amd import workload as wl
from tests.gpu_helpers import DEV, check_tokens, host_model, row_rel_err

pytestmark = pytest.mark.gpu
TOL = 2e-2
CAP = 4144          # the decode benchmark's capacity (contexts up to 4096 plus its steps)


@pytest.fixture(scope="module")
def model36():
    cfg = wl.config("8b")
    Wg = wl.make_weights(cfg, seed=0, device=DEV)
    m = host_model(Wg)            # 15 GB of host bf16 bit patterns
    yield cfg, Wg, m
    del Wg
    torch.cuda.empty_cache()


def own_cache(K, V, r):
    return oracle.KVCache([wl.bits(k[r:r + 1]) for k in K], [wl.bits(v[r:r + 1]) for v in V],
                          oracle.KV_CONTIGUOUS, 1, CAP)


def envelope(m, kv, token, pos, ref):
    """Largest row-relative change of the oracle's logits when one element
    of the token's embedding moves by one bf16 ulp (two elements tried)."""
    env = 0.0
    row = m.embed[token]
    for j in (17, 2900):
        keep = row[j]
        row[j] = keep + 1            # the next bf16 value of the same sign
        try:
            p = oracle.decode_row(m, kv, 0, token, pos)
        finally:
            row[j] = keep
        env = max(env, row_rel_err(p, ref))
    return env


@pytest.mark.parametrize("B,seed", [(1, 1), (256, 2)])
def test_full_depth_decode_against_oracle(model36, B, seed):
    cfg, Wg, m = model36
    print(f"full depth: B={B} seed={seed}: making the {B}-slot cache", flush=True)
    K, V = wl.make_kv_contiguous(cfg, B, CAP, seed=1000 + B, device=DEV)
    b = wl.make_batch(B, cfg["vocab"], seed=seed, len_lo=512, len_hi=4096)
    live = np.nonzero(b.valid)[0]
    order = live[np.argsort(b.seq_lens[live], kind="stable")]
    sample = sorted({int(order[0]), int(order[len(order) // 2]), int(order[-1])})
    kv = {r: own_cache(K, V, r) for r in sample}
    logits = torch.empty(B, cfg["vocab"], dtype=torch.float32, device=DEV)
    gl = {}
    for mode in ("default", "bi"):
        # every step writes a row's new k, v at its position before reading
        # it, so the second engine sees the same cache state as the first
        eng = corun.Engine(cfg, Wg, B, K, V, opt=corun.options(batch_invariant=(mode == "bi")))
        nxt = eng.decode_step(b.tokens, b.valid, b.seq_lens, logits)
        gl[mode] = (logits[sample].cpu().numpy(), nxt)
        eng.close()
        del eng
    del K, V
    torch.cuda.empty_cache()
    near = []
    for i, r in enumerate(sample):
        tok, pos = int(b.tokens[r]), int(b.seq_lens[r])
        print(f"full depth: B={B} row {r} (context {pos}): oracle", flush=True)
        ref = oracle.decode_row(m, kv[r], 0, tok, pos)
        env = envelope(m, kv[r], tok, pos, ref)
        bound = max(TOL, 2 * env)
        err = row_rel_err(gl["default"][0][i], ref)
        err_bi = row_rel_err(gl["bi"][0][i], ref)
        spread = row_rel_err(gl["default"][0][i], gl["bi"][0][i].astype(np.float64))
        print(f"full depth: B={B} row {r}: GPU {err:.3e}, GPU batch-invariant plan {err_bi:.3e}, "
              f"between the two plans {spread:.3e}; oracle one-ulp envelope {env:.3e} -> bound {bound:.3e}",
              flush=True)
        assert err <= bound and err_bi <= bound, (B, r, err, err_bi, env)
        check_tokens([gl["default"][1][r]], ref[None], gl["default"][0][i][None], [1], near)
    assert len(near) <= 1, near
