"""The C ABI without a GPU: the library loads, exports every entry point the
header declares, and its host-side checks reject bad input before anything
is enqueued.  No compute call is made here."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2608_14376_amd import corun
from paper_2608_14376_amd import workload as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "corun.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(corun_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = corun.load()
    syms = declared_symbols()
    assert set(syms) == set(corun.EXPORTS), syms
    for s in syms:
        assert hasattr(lib, s), f"{s} not exported"


def _kv(layout=corun.KV_CONTIGUOUS, n_slots=4, max_seq_len=256, page_size=16, num_pages=64, mpp=16):
    keep = []
    null2 = (C.c_void_p * 1)(None)
    keep.append(null2)
    kv = corun.KV(layout, n_slots, max_seq_len, page_size, num_pages, mpp, C.cast(null2, corun._PP),
                  C.cast(null2, corun._PP), None)
    kv._keep = keep
    return kv


def test_check_config_accepts_the_dense_configs():
    for name in ("tiny", "8b", "32b"):
        c = wl.config(name)
        assert corun.check_config(c, _kv(n_slots=256, max_seq_len=4224), 256) == corun.OK
        assert corun.check_config(c, _kv(corun.KV_PAGED, n_slots=32, num_pages=4096, mpp=2048), 32) == corun.OK


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 96, corun.E_SHAPE),
    ("n_kv_heads", 3, corun.E_SHAPE),
    ("hidden", 200, corun.E_SHAPE),
    ("vocab", 1000, corun.E_SHAPE),
    ("ffn", 0, corun.E_SHAPE),
])
def test_check_config_rejects_bad_shapes(field, value, status):
    c = wl.config("tiny", **{field: value})
    assert corun.check_config(c, _kv(), 4) == status
    assert corun.last_error()


def test_check_config_capacity():
    c = wl.config("tiny")
    assert corun.check_config(c, _kv(n_slots=2), 4) == corun.E_CAPACITY
    assert corun.check_config(c, _kv(max_seq_len=0), 4) == corun.E_CAPACITY
    assert corun.check_config(c, _kv(layout=7), 4) == corun.E_INVAL
    assert corun.check_config(c, _kv(), 0) == corun.E_SHAPE


def test_check_batch_rows():
    c = wl.config("tiny")
    kv = _kv(max_seq_len=128)
    ok = dict(tokens=[1, 2, 3, 4], valid=[1, 1, 1, 1], seq_lens=[0, 5, 100, 127])
    assert corun.check_batch(c, kv, **ok) == corun.OK
    assert corun.check_batch(c, kv, [1, 2, 3, 1024], [1, 1, 1, 1], [0, 0, 0, 0]) == corun.E_INVAL
    assert corun.check_batch(c, kv, [1, 2, 3, -1], [1, 1, 1, 1], [0, 0, 0, 0]) == corun.E_INVAL
    assert corun.check_batch(c, kv, [1, 2, 3, 4], [1, 1, 1, 1], [0, 0, 0, -3]) == corun.E_INVAL
    assert corun.check_batch(c, kv, [1, 2, 3, 4], [1, 1, 1, 1], [0, 0, 0, 128]) == corun.E_CAPACITY
    # padding rows are never validated: any token and length
    assert corun.check_batch(c, kv, [1, -99, 3, 10**9], [1, 0, 1, 0], [0, -5, 3, 2**31 - 1]) == corun.OK
    # multi-step runs need room for every step
    assert corun.check_batch(c, kv, **ok, n_steps=2) == corun.E_CAPACITY
    assert corun.check_batch(c, kv, [1], [1], [100], n_steps=28) == corun.OK
    assert corun.check_batch(c, kv, [1], [1], [100], n_steps=29) == corun.E_CAPACITY


def test_check_batch_pages():
    c = wl.config("tiny")
    kv = _kv(corun.KV_PAGED, n_slots=2, page_size=16, num_pages=8, mpp=4)
    pt = np.array([[0, 1, 2, 3], [4, 5, 6, 99]], np.int32)
    assert corun.check_batch(c, kv, [1, 1], [1, 1], [40, 40], page_table_host=pt) == corun.OK
    assert corun.check_batch(c, kv, [1, 1], [1, 1], [40, 48], page_table_host=pt) == corun.E_CAPACITY
    assert corun.check_batch(c, kv, [1, 1], [1, 0], [40, 63], page_table_host=pt) == corun.OK
    assert corun.check_batch(c, kv, [1, 1], [1, 1], [40, 64], page_table_host=pt) == corun.E_CAPACITY


def test_plan_is_a_function_of_shape_only():
    """The launch plan depends on (model, B, capacity) -- there is no input
    through which the live rows could reach it -- and differs across B."""
    c = wl.config("8b")
    plans = {B: corun.describe_plan(c, _kv(n_slots=256, max_seq_len=4224), B) for B in (1, 8, 16, 64, 256)}
    for B, p in plans.items():
        assert p["B"] == B and p["Mp"] % 64 == 0 and p["Mp"] >= B
        for name in ("qkv", "o", "gate_up", "down", "lm_head"):
            pr = p[name]
            assert pr["k_chunk"] % 32 == 0 and pr["split_k"] * pr["k_chunk"] >= pr["K"]
            assert (pr["split_k"] - 1) * pr["k_chunk"] < pr["K"]
        assert p["lm_head"]["split_k"] == 1
        assert p["attn_chunk"] % 64 == 0 and p["attn_max_splits"] * p["attn_chunk"] >= 4224
    assert plans[1] == corun.describe_plan(c, _kv(n_slots=256, max_seq_len=4224), 1)
    assert plans[16]["qkv"]["split_k"] >= plans[256]["qkv"]["split_k"]
    forced = corun.describe_plan(c, _kv(n_slots=256, max_seq_len=4224), 16, corun.options(split_k_override=3))
    assert forced["qkv"]["split_k"] == 3 and forced["down"]["split_k"] == 3


def test_attention_chunk_rule():
    """The split-KV chunk: the smallest power of two from 128 up to 1024 with
    B * kv_heads * ceil(capacity / chunk) <= 2048, fixed per engine (the
    decode benchmark's capacity 4144: 128 / 256 / 512 / 1024 tokens at
    B = 1 / 8 / 16 / 32 and up); an explicit chunk wins."""
    c = wl.config("8b")
    got = {B: corun.describe_plan(c, _kv(n_slots=256, max_seq_len=4144), B)["attn_chunk"]
           for B in (1, 2, 4, 8, 16, 32, 64, 256)}
    assert got == {1: 128, 2: 128, 4: 128, 8: 256, 16: 512, 32: 1024, 64: 1024, 256: 1024}, got
    for B, ch in got.items():
        assert B * c["n_kv_heads"] * -(-4144 // ch) <= 2048 or ch == 1024
        assert ch == 128 or B * c["n_kv_heads"] * -(-4144 // (ch // 2)) > 2048
    assert corun.describe_plan(c, _kv(n_slots=256, max_seq_len=4144), 8,
                               corun.options(attn_chunk=192))["attn_chunk"] == 192


def _small_batch_layer(p):
    return all((p[n]["m_tile"], p[n]["n_tile"], p[n]["split_k"]) == (16, 16, 1)
               for n in ("qkv", "o", "gate_up", "down"))


def test_small_batch_layer_plan():
    """Dense models at B = 1 run the small-batch layer by default, up to B =
    8 when asked (small_batch_layer = 1): every projection on 16-column
    fragment-packed tiles over the whole of K (no split-K), K padded to 32 in
    the description; the lm_head keeps the pipelined kernel.  It needs the
    packed copies and the default epilogue placement; batch-invariant mode
    and mixture-of-experts models never take it, and small_batch_layer = 2
    turns it off."""
    kv = _kv(n_slots=256, max_seq_len=4224)
    for name in ("8b", "tiny", "small128", "32b"):
        c = wl.config(name)
        p = corun.describe_plan(c, kv, 1)
        assert _small_batch_layer(p), name
        for n in ("qkv", "o", "gate_up", "down"):
            assert p[n]["k_chunk"] == (p[n]["K"] + 31) // 32 * 32
        assert p["lm_head"]["n_tile"] != 16
        assert not _small_batch_layer(corun.describe_plan(c, kv, 1, corun.options(small_batch_layer=2)))
        for B in (2, 8, 16, 64):
            assert not _small_batch_layer(corun.describe_plan(c, kv, B)), (name, B)
        for B in (2, 5, 8):
            assert _small_batch_layer(corun.describe_plan(c, kv, B, corun.options(small_batch_layer=1))), (name, B)
        for opt in (corun.options(no_weight_pack=True), corun.options(qkv_epilogue=1),
                    corun.options(qkv_epilogue=2), corun.options(batch_invariant=True),
                    corun.options(split_k_override=2)):
            assert not _small_batch_layer(corun.describe_plan(c, kv, 1, opt)), name
        for B, kw in ((9, {}), (1, dict(no_weight_pack=True)), (1, dict(batch_invariant=True))):
            with pytest.raises(corun.CorunError):
                corun.describe_plan(c, kv, B, corun.options(small_batch_layer=1, **kw))
    for name in ("tiny_moe", "moe"):
        assert not _small_batch_layer(corun.describe_plan(wl.config(name), kv, 1)), name
    with pytest.raises(corun.CorunError):
        corun.describe_plan(wl.config("tiny"), kv, 1, corun.options(small_batch_layer=3))


def test_batch_invariant_plan_ignores_the_batch_size():
    """Batch-invariant mode (Sec. III, Fig. 3b and Definition 1): for every
    B no split-K, one kernel per projection (the pipelined one when K % 64
    == 0, else the 128-row LDS-tiled one) and split-KV off, so every element
    is one MFMA chain over K in the same order; only the tile follows B.
    The default plans split K differently across B."""
    for name in ("8b", "tiny", "32b"):
        c = wl.config(name)
        kv = _kv(n_slots=256, max_seq_len=4224)
        bi = corun.options(batch_invariant=True)
        plans = [corun.describe_plan(c, kv, B, bi) for B in (1, 3, 8, 64, 65, 200, 256)]
        for p in plans:
            for proj in ("qkv", "o", "gate_up", "down", "lm_head"):
                pr = p[proj]
                assert pr["split_k"] == 1 and pr["k_chunk"] >= pr["K"], (name, proj)
                if pr["K"] % 64 == 0:
                    assert pr["n_tile"] > 0 and pr["m_tile"] > 0, (name, proj)
                else:
                    assert pr["n_tile"] == 0 and pr["m_tile"] == 128, (name, proj)
            assert p["attn_max_splits"] == 1 and p["attn_chunk"] >= 4224
    std = [corun.describe_plan(wl.config("8b"), _kv(n_slots=256, max_seq_len=4224), B) for B in (1, 256)]
    assert std[0]["qkv"] != std[1]["qkv"] and std[0]["attn_chunk"] != std[1]["attn_chunk"]


def test_batch_invariant_rejects_plan_overrides():
    c = wl.config("tiny")
    kv = _kv(n_slots=4, max_seq_len=128)
    for extra in (dict(attn_chunk=128), dict(split_k_override=2), dict(gemm_bm=128)):
        with pytest.raises(corun.CorunError):
            corun.describe_plan(c, kv, 4, corun.options(batch_invariant=True, **extra))


def test_options_take_only_flags():
    """no_weight_pack, batch_invariant and bi_prefill are 0 or 1,
    qkv_epilogue 0, 1 or 2."""
    c = wl.config("tiny")
    kv = _kv(n_slots=4, max_seq_len=128)
    for bad in (dict(no_weight_pack=2), dict(no_weight_pack=-1), dict(bi_prefill=3), dict(qkv_epilogue=3),
                dict(qkv_epilogue=-1)):
        opt = corun.options()
        for k, v in bad.items():
            setattr(opt, k, v)
        with pytest.raises(corun.CorunError):
            corun.describe_plan(c, kv, 4, opt)
    corun.describe_plan(c, kv, 4, corun.options(no_weight_pack=True, qkv_epilogue=2))


def test_prefill_tiles_follow_the_wave_estimate():
    """M > 256 takes the tile and split-K of least estimated time (waves of
    256 workgroups, per-tile wave costs, split partials' traffic): the
    choices the standalone measurements favour at these 8B shapes.  The
    decode plan at B = 512 and 1024 runs the same rule as a prefill of that
    many rows (describe_plan stops at B = 1024)."""
    c = wl.config("8b")

    def plan(M):
        p = corun.describe_plan(c, _kv(n_slots=M, max_seq_len=4224), M)
        return {k: (p[k]["m_tile"], p[k]["n_tile"], p[k]["split_k"]) for k in ("qkv", "o", "gate_up", "down")}

    p512, p1024 = plan(512), plan(1024)
    assert p512["gate_up"] == (256, 256, 1)          # 192 tiles in one wave beat 384 of 256 x 128
    assert p512["qkv"] == (256, 128, 2)
    assert p1024["gate_up"] == (256, 128, 1)         # three full waves beat 1.5 waves of 256 x 256
    assert p1024["o"] == (256, 128, 2)
    for p in (p512, p1024):                          # every split keeps at least 512 K elements
        for name, K in (("qkv", 4096), ("o", 4096), ("gate_up", 4096), ("down", 12288)):
            assert K // p[name][2] >= 512, (name, p[name])


def test_prefill_plan_is_a_function_of_the_length_only():
    """The prefill plan takes no workspace size: the 8B shape's projections
    split K at lengths where the estimate asks for it (so an engine-size cap
    would have changed them), never in batch-invariant mode; every
    projection of the plan covers its K exactly."""
    c = wl.config("8b")
    split = set()
    for n in (1, 7, 64, 100, 300, 600, 2048, 8192, 32768):
        p = corun.describe_prefill_plan(c, n)
        bi = corun.describe_prefill_plan(c, n, corun.options(bi_prefill=True))
        for name in ("qkv", "o", "gate_up", "down"):
            pr = p[name]
            assert pr["split_k"] >= 1 and pr["split_k"] * pr["k_chunk"] >= pr["K"] > (pr["split_k"] - 1) * pr["k_chunk"]
            if pr["split_k"] > 1:
                split.add(n)
            assert bi[name]["split_k"] == 1
        assert p["router"]["N"] == 0
    assert {300, 600} & split, split
    moe = corun.describe_prefill_plan(wl.config("moe"), 300)
    assert moe["router"]["N"] == 128 and moe["gate_up"]["N"] == 0
