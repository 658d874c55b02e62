"""GPU tests of the request-bound seeded sampler (Sec. IV, "Shape-Aligned
Sampling"; y_t = S(l_t, R(s, t)) in Sec. IV, "Determinism Argument").

* the kernel against the oracle on given logits (the tiny vocabulary and
  the 8B one): the token exactly, the log-probability to float rounding;
* a request's draw does not move when co-runners or padding rows change;
* the paper's validation protocol (Sec. V, "Determinism Validation") on the
  tiny model: 32 prompts, temperature 0.6, seed 42, up to 8 output tokens,
  each prompt alone (at another slot) and in a batch of 32: identical token
  sequences and bit-identical sampled-token log-probabilities."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_14376_amd import corun
from paper_2608_14376_amd import workload as wl
from tests.gpu_helpers import DEV, to_device

pytestmark = pytest.mark.gpu
B = 32


def engine(cfg, seed, cap, prefill=0):
    Wg = to_device(wl.make_weights(cfg, seed=seed))
    K, V = wl.make_kv_contiguous(cfg, B, cap, seed + 1)
    K = [k.to(DEV) for k in K]
    V = [v.to(DEV) for v in V]
    return corun.Engine(cfg, Wg, B, K, V, opt=corun.options(max_prefill_len=prefill)), (Wg, K, V)


@pytest.mark.parametrize("vocab", [1024, 151936])
def test_sampler_matches_oracle(vocab):
    cfg = dict(wl.config("tiny"), vocab=vocab)
    eng, keep = engine(cfg, 70, 64)
    rng = np.random.default_rng(71)
    logits = torch.from_numpy(rng.normal(0, 3, (B, vocab)).astype(np.float32)).to(DEV)
    valid = (rng.random(B) < 0.8).astype(np.uint8)
    pos = rng.integers(0, 1 << 20, B).astype(np.int32)
    seeds = rng.integers(0, 1 << 63, B, dtype=np.uint64)
    temp = rng.choice([0.0, 0.3, 0.6, 1.0, 1.7], B).astype(np.float32)
    tok, lp = eng.sample(logits, valid, pos, seeds, temp)
    host = logits.cpu().numpy()
    for r in range(B):
        if not valid[r]:
            assert tok[r] == -1
            continue
        ot, olp = oracle.sample(host[r], int(seeds[r]), int(pos[r]), float(temp[r]))
        assert tok[r] == ot, (r, tok[r], ot)
        assert abs(float(lp[r]) - olp) <= 1e-6 * max(1.0, abs(olp)), (r, lp[r], olp)
    eng.close()


def test_draw_is_bound_to_the_request():
    cfg = wl.config("tiny")
    eng, keep = engine(cfg, 72, 64)
    rng = np.random.default_rng(73)
    logits = torch.from_numpy(rng.normal(0, 2, (B, cfg["vocab"])).astype(np.float32)).to(DEV)
    valid = np.zeros(B, np.uint8)
    valid[[3, 17]] = 1
    pos = np.zeros(B, np.int32)
    pos[3], pos[17] = 40, 99
    seeds = np.zeros(B, np.uint64)
    seeds[3], seeds[17] = 42, 7
    temp = np.full(B, 0.6, np.float32)
    t0, l0 = eng.sample(logits, valid, pos, seeds, temp)
    for trial in range(5):
        v2 = valid.copy()
        others = rng.choice([i for i in range(B) if i != 3], 10, replace=False)
        v2[others] = rng.integers(0, 2, 10)
        p2 = pos.copy()
        s2 = seeds.copy()
        T2 = temp.copy()
        mask = np.arange(B) != 3
        p2[mask] = rng.integers(0, 1000, mask.sum())
        s2[mask] = rng.integers(0, 1 << 63, mask.sum(), dtype=np.uint64)
        T2[mask] = rng.random(mask.sum()).astype(np.float32)
        t1, l1 = eng.sample(logits, v2, p2, s2, T2)
        assert t1[3] == t0[3] and l1.view(np.int32)[3] == l0.view(np.int32)[3]
    eng.close()


def test_paper_protocol_alone_vs_batch_of_32():
    cfg = wl.config("tiny")
    T, SEED, N_OUT = 0.6, 42, 8
    eng, keep = engine(cfg, 74, 80, prefill=64)
    rng = np.random.default_rng(75)
    prompts = [wl.make_prompt(cfg["vocab"], int(rng.integers(4, 49)), seed=100 + i) for i in range(B)]
    V = cfg["vocab"]
    last = torch.empty(V, dtype=torch.float32, device=DEV)
    logits = torch.empty(B, V, dtype=torch.float32, device=DEV)

    def first_token(p, slot):
        eng.prefill(p, slot, last)
        t, l = eng.sample(last, [1], [len(p)], [SEED], [T])
        return int(t[0]), l.view(np.int32)[0]

    # alone: one live request at a slot other than its batched one, every other row padding
    alone = []
    for i, p in enumerate(prompts):
        slot = (7 * i + 3) % B
        toks, lps = [], []
        t, l = first_token(p, slot)
        toks.append(t)
        lps.append(l)
        for k in range(1, N_OUT):
            tokens = rng.integers(0, V, B).astype(np.int32)          # padding rows hold garbage
            seq = rng.integers(0, 70, B).astype(np.int32)
            valid = np.zeros(B, np.uint8)
            tokens[slot], seq[slot], valid[slot] = toks[-1], len(p) + k - 1, 1
            eng.decode_step(tokens, valid, seq, logits)
            pos = seq + 1
            t, l = eng.sample(logits, valid, pos, np.full(B, SEED, np.uint64), np.full(B, T, np.float32))
            toks.append(int(t[slot]))
            lps.append(l.view(np.int32)[slot])
        alone.append((toks, lps))

    # batched: every prompt prefilled alone into slot i, then all 32 decode together
    cur = [first_token(p, i) for i, p in enumerate(prompts)]
    batched = [([c[0]], [c[1]]) for c in cur]
    valid = np.ones(B, np.uint8)
    for k in range(1, N_OUT):
        tokens = np.array([batched[i][0][-1] for i in range(B)], np.int32)
        seq = np.array([len(p) + k - 1 for p in prompts], np.int32)
        eng.decode_step(tokens, valid, seq, logits)
        t, l = eng.sample(logits, valid, seq + 1, np.full(B, SEED, np.uint64), np.full(B, T, np.float32))
        for i in range(B):
            batched[i][0].append(int(t[i]))
            batched[i][1].append(l.view(np.int32)[i])

    for i in range(B):
        assert alone[i][0] == batched[i][0], (i, alone[i][0], batched[i][0])
        assert [int(x) for x in alone[i][1]] == [int(x) for x in batched[i][1]], i
    eng.close()
