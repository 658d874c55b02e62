"""CPU oracle for CoRun's padded decode step and isolated prefill.

TEST INFRASTRUCTURE ONLY: imported by the test-suite, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP library; the two meet only through the seeded inputs of
``paper_2608_14376_amd.workload``, which holds none of the method's arithmetic.

The arithmetic lives in ``corun_oracle.c`` (plain C, fp64 between the model's
bf16/fp32 storage points, sequential sums).  This module marshals numpy arrays
into it through ctypes.  Arrays of bf16 values are carried as ``numpy.uint16``
bit patterns.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "corun_oracle.c")
_LIB = os.path.join(_HERE, "libcorun_oracle.so")

KV_CONTIGUOUS = 0
KV_PAGED = 1


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (portable flags: the library also runs on
    hosts other than the one that built it; no fp contraction, so every sum
    is the plain sequential one)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
               "-shared", "-fPIC", "-o", _LIB + ".tmp", _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(_LIB + ".tmp", _LIB)
    return _LIB


class _Cfg(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "n_layers", "hidden", "n_heads", "n_kv_heads", "head_dim", "ffn", "vocab",
        "n_experts", "top_k", "expert_ffn")] + [("rms_eps", C.c_double), ("rope_theta", C.c_double)]


_PP = C.POINTER(C.c_void_p)


class _Weights(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("final_norm", C.c_void_p), ("lm_head", C.c_void_p)] + [
        (n, _PP) for n in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down",
                           "w_router", "w_exp_gate_up", "w_exp_down")]


class _KV(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "layout", "n_slots", "max_seq_len", "page_size", "num_pages", "max_pages_per_seq")] + [
        ("k", _PP), ("v", _PP), ("page_table", C.c_void_p)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = C.CDLL(_LIB)
        u16p = C.c_void_p
        L.orc_bf16_to_f64.restype = C.c_double
        L.orc_bf16_to_f64.argtypes = [C.c_uint16]
        L.orc_f64_to_bf16.restype = C.c_uint16
        L.orc_f64_to_bf16.argtypes = [C.c_double]
        L.orc_f32bits_to_bf16.argtypes = [C.c_void_p, C.c_void_p, C.c_int64]
        L.orc_linear.argtypes = [u16p, C.c_int, u16p, C.c_int, C.c_void_p]
        L.orc_rmsnorm.argtypes = [C.c_void_p, C.c_int, u16p, C.c_double, u16p]
        L.orc_rope.argtypes = [C.c_void_p, C.c_int, C.c_int, C.c_double, C.c_void_p]
        L.orc_attention.argtypes = [u16p, C.c_void_p, C.c_void_p, C.c_int, C.c_int, C.c_void_p]
        L.orc_silu.restype = C.c_double
        L.orc_silu.argtypes = [C.c_double]
        L.orc_argmax_f32.restype = C.c_int
        L.orc_argmax_f32.argtypes = [C.c_void_p, C.c_int]
        L.orc_route.argtypes = [C.c_void_p, C.c_int, C.c_int, C.c_void_p, C.c_void_p]
        L.orc_decode_row.restype = C.c_int
        L.orc_decode_row.argtypes = [C.POINTER(_Cfg), C.POINTER(_Weights), C.POINTER(_KV),
                                     C.c_int, C.c_int, C.c_int, C.c_void_p]
        L.orc_decode_row_routed.restype = C.c_int
        L.orc_decode_row_routed.argtypes = [C.POINTER(_Cfg), C.POINTER(_Weights), C.POINTER(_KV),
                                            C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_void_p, C.c_void_p,
                                            C.c_void_p]
        L.orc_prefill_routed.restype = C.c_int
        L.orc_prefill_routed.argtypes = [C.POINTER(_Cfg), C.POINTER(_Weights), C.POINTER(_KV), C.c_int,
                                         C.c_void_p, C.c_int, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                         C.c_void_p]
        L.orc_route_forced.restype = C.c_int
        L.orc_route_forced.argtypes = [C.c_void_p, C.c_int, C.c_int, C.c_void_p, C.c_void_p]
        L.orc_decode_batch.restype = C.c_int
        L.orc_decode_batch.argtypes = [C.POINTER(_Cfg), C.POINTER(_Weights), C.POINTER(_KV), C.c_int,
                                       C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.orc_prefill.restype = C.c_int
        L.orc_prefill.argtypes = [C.POINTER(_Cfg), C.POINTER(_Weights), C.POINTER(_KV), C.c_int,
                                  C.c_void_p, C.c_int, C.c_void_p, C.c_void_p]
        L.orc_philox4x32_10.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p]
        L.orc_uniform.restype = C.c_double
        L.orc_uniform.argtypes = [C.c_uint32, C.c_uint32]
        L.orc_gumbel.restype = C.c_double
        L.orc_gumbel.argtypes = [C.c_uint64, C.c_int32, C.c_int32]
        L.orc_sample.restype = C.c_int
        L.orc_sample.argtypes = [C.c_void_p, C.c_int, C.c_uint64, C.c_int32, C.c_float, C.c_void_p, C.c_void_p]
        L.orc_set_threads.argtypes = [C.c_int]
        L.orc_get_threads.restype = C.c_int
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data


def set_threads(n: int) -> None:
    lib().orc_set_threads(int(n))


def get_threads() -> int:
    return int(lib().orc_get_threads())


# --------------------------------------------------------------------------
# Per-operator entry points (used by the pins in tests/test_oracle_*.py)
# --------------------------------------------------------------------------

def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return np.array([lib().orc_bf16_to_f64(int(x)) for x in b.ravel()]).reshape(b.shape)


def f64_to_bf16(x) -> int:
    return int(lib().orc_f64_to_bf16(float(x)))


def f32bits_to_bf16(bits: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint32)
    out = np.empty(b.shape, np.uint16)
    lib().orc_f32bits_to_bf16(_ptr(b), _ptr(out), b.size)
    return out


def linear(h: np.ndarray, W: np.ndarray) -> np.ndarray:
    h = np.ascontiguousarray(h, np.uint16)
    W = np.ascontiguousarray(W, np.uint16)
    out_f, in_f = W.shape
    assert h.shape == (in_f,)
    y = np.empty(out_f, np.float64)
    lib().orc_linear(_ptr(h), in_f, _ptr(W), out_f, _ptr(y))
    return y


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    x = np.ascontiguousarray(x, np.float32)
    g = np.ascontiguousarray(g, np.uint16)
    y = np.empty(x.shape, np.uint16)
    lib().orc_rmsnorm(_ptr(x), x.size, _ptr(g), float(eps), _ptr(y))
    return y


def rope(x: np.ndarray, pos: int, theta: float) -> np.ndarray:
    x = np.ascontiguousarray(x, np.float64)
    y = np.empty_like(x)
    lib().orc_rope(_ptr(x), x.size, int(pos), float(theta), _ptr(y))
    return y


def attention(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """One head: q [d] bf16 bits, K, V [n, d] bf16 bits -> fp64 [d]."""
    q = np.ascontiguousarray(q, np.uint16)
    K = np.ascontiguousarray(K, np.uint16)
    V = np.ascontiguousarray(V, np.uint16)
    n, d = K.shape
    kp = (C.c_void_p * max(n, 1))(*[K.ctypes.data + 2 * d * t for t in range(n)])
    vp = (C.c_void_p * max(n, 1))(*[V.ctypes.data + 2 * d * t for t in range(n)])
    out = np.empty(d, np.float64)
    lib().orc_attention(_ptr(q), kp, vp, n, d, _ptr(out))
    return out


def silu(z: float) -> float:
    return float(lib().orc_silu(float(z)))


def argmax_f32(v: np.ndarray) -> int:
    v = np.ascontiguousarray(v, np.float32)
    return int(lib().orc_argmax_f32(_ptr(v), v.size))


def philox4x32_10(ctr, key) -> np.ndarray:
    """Philox4x32-10 block: four 32-bit counter words, two key words."""
    c = np.ascontiguousarray(ctr, np.uint32)
    k = np.ascontiguousarray(key, np.uint32)
    out = np.empty(4, np.uint32)
    lib().orc_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def uniform(w0: int, w1: int) -> float:
    return float(lib().orc_uniform(w0, w1))


def gumbel(seed: int, t: int, v: int) -> float:
    """g_v = -ln(-ln u_v) of R(seed, t)."""
    return float(lib().orc_gumbel(seed, t, v))


def sample(logits: np.ndarray, seed: int, t: int, temperature: float):
    """S(l, R(seed, t)): (token, log-probability) by the Gumbel-max rule."""
    l = np.ascontiguousarray(logits, np.float32)
    tok = np.empty(1, np.int32)
    lp = np.empty(1, np.float64)
    if lib().orc_sample(_ptr(l), l.size, seed, t, temperature, _ptr(tok), _ptr(lp)):
        raise ValueError("empty logits")
    return int(tok[0]), float(lp[0])


def route(logits: np.ndarray, top_k: int):
    logits = np.ascontiguousarray(logits, np.float64)
    sel = np.empty(top_k, np.int32)
    w = np.empty(top_k, np.float64)
    lib().orc_route(_ptr(logits), logits.size, top_k, _ptr(sel), _ptr(w))
    return sel, w


def route_forced(logits: np.ndarray, force) -> np.ndarray:
    """Weights of a given expert set: softmax over all experts, renormalised
    over the set, in the set's order."""
    logits = np.ascontiguousarray(logits, np.float64)
    f = np.ascontiguousarray(force, np.int32)
    w = np.empty(f.size, np.float64)
    if lib().orc_route_forced(_ptr(logits), logits.size, f.size, _ptr(f), _ptr(w)):
        raise ValueError("malformed expert set")
    return w


# --------------------------------------------------------------------------
# Whole model
# --------------------------------------------------------------------------

@dataclass
class Model:
    """Host-side model: config dict plus numpy uint16 (bf16 bits) weights."""
    cfg: dict
    embed: np.ndarray
    final_norm: np.ndarray
    lm_head: np.ndarray
    attn_norm: list
    w_qkv: list
    w_o: list
    mlp_norm: list
    w_gate_up: list = field(default_factory=list)
    w_down: list = field(default_factory=list)
    w_router: list = field(default_factory=list)
    w_exp_gate_up: list = field(default_factory=list)
    w_exp_down: list = field(default_factory=list)


@dataclass
class KVCache:
    """Host KV cache: per-layer uint16 arrays, keys and values by token:
    contiguous K, V [slots, nkv, S, d]; paged K, V [pages, nkv, page_size, d]
    with an int32 page table [slots, max_pages_per_seq]."""
    k: list
    v: list
    layout: int = KV_CONTIGUOUS
    n_slots: int = 0
    max_seq_len: int = 0
    page_size: int = 16
    num_pages: int = 0
    max_pages_per_seq: int = 0
    page_table: np.ndarray | None = None


class _Bound:
    """ctypes views that keep the numpy arrays alive for one call."""

    def __init__(self, m: Model, kv: KVCache):
        c = m.cfg
        self.cfg = _Cfg(c["n_layers"], c["hidden"], c["n_heads"], c["n_kv_heads"], c["head_dim"],
                        c["ffn"], c["vocab"], c.get("n_experts", 0), c.get("top_k", 0),
                        c.get("expert_ffn", 0), float(c["rms_eps"]), float(c["rope_theta"]))
        L = c["n_layers"]
        keep = []

        def arr(lst):
            if not lst:
                return C.cast(None, _PP)
            for a in lst:
                assert a.dtype == np.uint16 and a.flags["C_CONTIGUOUS"]
            keep.extend(lst)
            t = (C.c_void_p * L)(*[a.ctypes.data for a in lst])
            keep.append(t)
            return C.cast(t, _PP)

        for a in (m.embed, m.final_norm, m.lm_head):
            assert a.dtype == np.uint16 and a.flags["C_CONTIGUOUS"]
        self.w = _Weights(m.embed.ctypes.data, m.final_norm.ctypes.data, m.lm_head.ctypes.data,
                          arr(m.attn_norm), arr(m.w_qkv), arr(m.w_o), arr(m.mlp_norm),
                          arr(m.w_gate_up), arr(m.w_down), arr(m.w_router),
                          arr(m.w_exp_gate_up), arr(m.w_exp_down))
        pt = None
        if kv.layout == KV_PAGED:
            assert kv.page_table is not None and kv.page_table.dtype == np.int32
            pt = kv.page_table.ctypes.data
        self.kv = _KV(kv.layout, kv.n_slots, kv.max_seq_len, kv.page_size, kv.num_pages,
                      kv.max_pages_per_seq, arr(kv.k), arr(kv.v), pt)
        self._keep = keep
        self._m, self._kvref = m, kv


def decode_row(m: Model, kv: KVCache, slot: int, token: int, pos: int) -> np.ndarray:
    b = _Bound(m, kv)
    logits = np.empty(m.cfg["vocab"], np.float64)
    rc = lib().orc_decode_row(C.byref(b.cfg), C.byref(b.w), C.byref(b.kv), slot, token, pos,
                              _ptr(logits))
    if rc:
        raise ValueError("oracle rejected the row")
    return logits


def decode_row_routed(m: Model, kv: KVCache, slot: int, token: int, pos: int, force=None):
    """decode_row of a mixture of experts with its routing exposed:
    (logits [V], router logits [L, E] fp64, own top-k [L, k]).  force
    ([L, k] int32, optional) makes layer l follow that expert set instead of
    its own top-k (the records still hold the oracle's own choice)."""
    c = m.cfg
    L, E, k = c["n_layers"], c["n_experts"], c["top_k"]
    b = _Bound(m, kv)
    logits = np.empty(c["vocab"], np.float64)
    rl = np.empty((L, E), np.float64)
    own = np.empty((L, k), np.int32)
    f = None if force is None else np.ascontiguousarray(force, np.int32).reshape(L, k)
    rc = lib().orc_decode_row_routed(C.byref(b.cfg), C.byref(b.w), C.byref(b.kv), slot, token, pos,
                                     _ptr(logits), None if f is None else _ptr(f), _ptr(rl), _ptr(own))
    if rc:
        raise ValueError("oracle rejected the row or the forced routing")
    return logits, rl, own


def prefill_routed(m: Model, kv: KVCache, slot: int, prompt, force=None):
    """prefill of a mixture of experts with its routing exposed: (logits of
    the last position [V], token, router logits [L, Lp, E], own top-k
    [L, Lp, k]); force [L, Lp, k] optional, as in decode_row_routed."""
    c = m.cfg
    L, E, k = c["n_layers"], c["n_experts"], c["top_k"]
    prompt = np.ascontiguousarray(prompt, np.int32)
    Lp = prompt.size
    b = _Bound(m, kv)
    logits = np.empty(c["vocab"], np.float64)
    tok = np.empty(1, np.int32)
    rl = np.empty((L, Lp, E), np.float64)
    own = np.empty((L, Lp, k), np.int32)
    f = None if force is None else np.ascontiguousarray(force, np.int32).reshape(L, Lp, k)
    rc = lib().orc_prefill_routed(C.byref(b.cfg), C.byref(b.w), C.byref(b.kv), slot, _ptr(prompt), Lp,
                                  _ptr(logits), _ptr(tok), None if f is None else _ptr(f), _ptr(rl), _ptr(own))
    if rc:
        raise ValueError("oracle rejected the prompt or the forced routing")
    return logits, int(tok[0]), rl, own


def decode_batch(m: Model, kv: KVCache, tokens, valid, seq_lens):
    """Padded decode step, row by row.  Returns (logits [B, V] fp64 with NaN
    in padding rows, next [B] int32 with -1 for padding rows)."""
    tokens = np.ascontiguousarray(tokens, np.int32)
    valid = np.ascontiguousarray(valid, np.uint8)
    seq_lens = np.ascontiguousarray(seq_lens, np.int32)
    B = tokens.size
    b = _Bound(m, kv)
    logits = np.full((B, m.cfg["vocab"]), np.nan, np.float64)
    nxt = np.empty(B, np.int32)
    rc = lib().orc_decode_batch(C.byref(b.cfg), C.byref(b.w), C.byref(b.kv), B, _ptr(tokens),
                                _ptr(valid), _ptr(seq_lens), _ptr(logits), _ptr(nxt))
    if rc:
        raise ValueError("oracle rejected the batch")
    return logits, nxt


def prefill(m: Model, kv: KVCache, slot: int, prompt):
    """Isolated prefill: writes KV[0, Lp) of `slot`; returns (logits of the
    last position [V] fp64, greedy token)."""
    prompt = np.ascontiguousarray(prompt, np.int32)
    b = _Bound(m, kv)
    logits = np.empty(m.cfg["vocab"], np.float64)
    tok = np.empty(1, np.int32)
    rc = lib().orc_prefill(C.byref(b.cfg), C.byref(b.w), C.byref(b.kv), slot, _ptr(prompt),
                           prompt.size, _ptr(logits), _ptr(tok))
    if rc:
        raise ValueError("oracle rejected the prompt")
    return logits, int(tok[0])
