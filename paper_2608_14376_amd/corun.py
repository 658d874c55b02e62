"""ctypes binding of the C ABI declared in ``include/corun.h``.

Argument marshalling only: every step of the decode and prefill path runs in
the HIP kernels of ``libcorun.so``.  There is no fallback -- if the library
is missing, :func:`load` raises.  Torch tensors are accepted where the ABI
takes device or host pointers; torch is used for device memory and streams.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcorun.so")

OK, E_INVAL, E_SHAPE, E_CAPACITY, E_HIP, E_STATE = 0, -1, -2, -3, -4, -5
KV_CONTIGUOUS, KV_PAGED = 0, 1

EXPORTS = ("corun_engine_create", "corun_engine_destroy", "corun_decode_step", "corun_decode_run",
           "corun_prefill", "corun_prefill_chunk", "corun_prefill_batch", "corun_check_config", "corun_check_batch",
           "corun_describe_plan", "corun_describe_prefill_plan",
           "corun_last_error", "corun_time_kernel", "corun_profile_step", "corun_sample", "corun_sample_noalloc", "corun_engine_info",
           "corun_engine_set_page_table_host",
           "corun_routing_trace",
           "corun_sched_create", "corun_sched_destroy", "corun_sched_add_request", "corun_sched_step",
           "corun_sched_output", "corun_sched_state", "corun_sched_last_error")

# kernel ids of corun_time_kernel
K_QKV_GEMM, K_O_GEMM, K_GATE_UP_GEMM, K_DOWN_GEMM, K_LM_HEAD, K_ATTN_SPLIT, K_ATTN_MERGE, K_RMSNORM, \
    K_QKV_POST, K_SWIGLU, K_ARGMAX, K_MOE_ROUTER = range(12)
KERNEL_NAMES = ("qkv_gemm", "o_gemm", "gate_up_gemm", "down_gemm", "lm_head", "attn_split", "attn_merge",
                "rmsnorm", "qkv_post", "swiglu", "argmax", "moe_router")


class ModelCfg(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "n_layers", "hidden", "n_heads", "n_kv_heads", "head_dim", "ffn", "vocab",
        "n_experts", "top_k", "expert_ffn")] + [("rms_eps", C.c_float), ("rope_theta", C.c_float)]


_PP = C.POINTER(C.c_void_p)


class Weights(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("final_norm", C.c_void_p), ("lm_head", C.c_void_p)] + [
        (n, _PP) for n in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down",
                           "w_router", "w_exp_gate_up", "w_exp_down")]


class KV(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "layout", "n_slots", "max_seq_len", "page_size", "num_pages", "max_pages_per_seq")] + [
        ("k", _PP), ("v", _PP), ("page_table", C.c_void_p)]


class Options(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "attn_chunk", "max_prefill_len", "no_graph", "poison_workspace", "split_k_override", "gemm_bm",
        "batch_invariant", "bi_prefill", "no_weight_pack", "qkv_epilogue", "record_routing",
        "small_batch_layer")]


class CorunError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"corun status {status}: {msg}")
        self.status = status


_lib = None


def load():
    """Open libcorun.so (built by ``python -m paper_2608_14376_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_14376_amd.build`")
    L = C.CDLL(LIB_PATH)
    st = C.c_int
    L.corun_engine_create.restype = st
    L.corun_engine_create.argtypes = [C.POINTER(ModelCfg), C.POINTER(Weights), C.POINTER(KV), C.c_int32,
                                      C.POINTER(Options), C.c_void_p, C.POINTER(C.c_void_p)]
    L.corun_engine_destroy.restype = None
    L.corun_engine_destroy.argtypes = [C.c_void_p]
    L.corun_decode_step.restype = st
    L.corun_decode_step.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
    L.corun_decode_run.restype = st
    L.corun_decode_run.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
    L.corun_prefill.restype = st
    L.corun_prefill.argtypes = [C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p]
    L.corun_prefill_batch.restype = st
    L.corun_prefill_batch.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p,
                                      C.c_void_p]
    L.corun_prefill_chunk.restype = st
    L.corun_prefill_chunk.argtypes = [C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_int32, C.c_void_p,
                                      C.c_void_p]
    L.corun_check_config.restype = st
    L.corun_check_config.argtypes = [C.POINTER(ModelCfg), C.POINTER(KV), C.c_int32]
    L.corun_check_batch.restype = st
    L.corun_check_batch.argtypes = [C.POINTER(ModelCfg), C.POINTER(KV), C.c_void_p, C.c_int32, C.c_void_p,
                                    C.c_void_p, C.c_void_p, C.c_int32]
    L.corun_describe_plan.restype = C.c_int32
    L.corun_describe_plan.argtypes = [C.POINTER(ModelCfg), C.POINTER(KV), C.c_int32, C.POINTER(Options),
                                      C.c_void_p, C.c_int32]
    L.corun_describe_prefill_plan.restype = C.c_int32
    L.corun_describe_prefill_plan.argtypes = [C.POINTER(ModelCfg), C.c_int32, C.POINTER(Options), C.c_void_p,
                                              C.c_int32]
    L.corun_time_kernel.restype = st
    L.corun_time_kernel.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.c_int32, C.POINTER(C.c_float)]
    L.corun_profile_step.restype = st
    L.corun_profile_step.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p]
    L.corun_sample.restype = st
    L.corun_sample.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p,
                               C.c_void_p, C.c_void_p, C.c_void_p]
    L.corun_sample_noalloc.restype = st
    L.corun_sample_noalloc.argtypes = [C.c_void_p, C.c_int64, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p,
                                       C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
    L.corun_engine_info.restype = st
    L.corun_engine_info.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
    L.corun_engine_set_page_table_host.restype = st
    L.corun_engine_set_page_table_host.argtypes = [C.c_void_p, C.c_void_p]
    L.corun_routing_trace.restype = st
    L.corun_routing_trace.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.POINTER(C.c_int32)]
    L.corun_sched_create.restype = st
    L.corun_sched_create.argtypes = [C.c_void_p, C.POINTER(SchedCfg), C.POINTER(C.c_void_p)]
    L.corun_sched_destroy.restype = None
    L.corun_sched_destroy.argtypes = [C.c_void_p]
    L.corun_sched_add_request.restype = st
    L.corun_sched_add_request.argtypes = [C.c_void_p, C.c_int64, C.c_void_p, C.c_int32, C.c_int32, C.c_uint64,
                                          C.c_float]
    L.corun_sched_step.restype = st
    L.corun_sched_step.argtypes = [C.c_void_p, C.POINTER(C.c_int32)]
    L.corun_sched_output.restype = st
    L.corun_sched_output.argtypes = [C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p, C.c_int32,
                                     C.POINTER(C.c_int32), C.POINTER(C.c_int32)]
    L.corun_sched_state.restype = st
    L.corun_sched_state.argtypes = [C.c_void_p, C.POINTER(C.c_int32), C.POINTER(C.c_int32), C.POINTER(C.c_int32),
                                    C.POINTER(C.c_int32), C.c_void_p]
    L.corun_sched_last_error.restype = C.c_char_p
    L.corun_sched_last_error.argtypes = []
    L.corun_last_error.restype = C.c_char_p
    L.corun_last_error.argtypes = []
    _lib = L
    return L


def last_error() -> str:
    return load().corun_last_error().decode()


def _check(status: int):
    if status != OK:
        raise CorunError(status, last_error())


def model_cfg(c: dict) -> ModelCfg:
    return ModelCfg(c["n_layers"], c["hidden"], c["n_heads"], c["n_kv_heads"], c["head_dim"], c["ffn"],
                    c["vocab"], c.get("n_experts", 0), c.get("top_k", 0), c.get("expert_ffn", 0),
                    float(c["rms_eps"]), float(c["rope_theta"]))


def _ptr_array(tensors, keep):
    if not tensors:
        return C.cast(None, _PP)
    arr = (C.c_void_p * len(tensors))(*[t.data_ptr() for t in tensors])
    keep.append(arr)
    return C.cast(arr, _PP)


def kv_struct(layout: int, n_slots: int, k, v, keep, max_seq_len=0, page_size=0, num_pages=0,
              max_pages_per_seq=0, page_table=None) -> KV:
    return KV(layout, n_slots, max_seq_len, page_size, num_pages, max_pages_per_seq,
              _ptr_array(k, keep), _ptr_array(v, keep),
              page_table.data_ptr() if page_table is not None else None)


def options(attn_chunk=0, max_prefill_len=0, no_graph=False, poison_workspace=False, split_k_override=0,
            gemm_bm=0, batch_invariant=False, bi_prefill=False, no_weight_pack=False, qkv_epilogue=0,
            record_routing=False, small_batch_layer=0):
    return Options(attn_chunk, max_prefill_len, int(no_graph), int(poison_workspace), split_k_override, gemm_bm,
                   int(batch_invariant), int(bi_prefill), int(no_weight_pack), int(qkv_epilogue),
                   int(record_routing), int(small_batch_layer))


def _np(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def check_config(cfg: dict, kv: KV, B: int) -> int:
    c = model_cfg(cfg)
    return load().corun_check_config(C.byref(c), C.byref(kv), B)


def check_batch(cfg: dict, kv: KV, tokens, valid, seq_lens, n_steps=1, page_table_host=None) -> int:
    c = model_cfg(cfg)
    t, vm, s = _np(tokens, np.int32), _np(valid, np.uint8), _np(seq_lens, np.int32)
    pt = None if page_table_host is None else _np(page_table_host, np.int32)
    return load().corun_check_batch(C.byref(c), C.byref(kv), None if pt is None else pt.ctypes.data, t.size,
                                    t.ctypes.data, vm.ctypes.data, s.ctypes.data, n_steps)


def describe_plan(cfg: dict, kv: KV, B: int, opt: Options | None = None) -> dict:
    c = model_cfg(cfg)
    out = np.zeros(64, np.int32)
    n = load().corun_describe_plan(C.byref(c), C.byref(kv), B, C.byref(opt) if opt else None,
                                   out.ctypes.data, 64)
    if n < 0:
        raise CorunError(n, last_error())
    v = out[:n].tolist()
    plan = {"B": v[0], "Mp": v[1]}
    for i, name in enumerate(("qkv", "o", "gate_up", "down", "lm_head")):
        N, K, S, Kc, bm, bn = v[2 + 6 * i: 8 + 6 * i]
        plan[name] = {"N": N, "K": K, "split_k": S, "k_chunk": Kc, "m_tile": bm, "n_tile": bn}
    plan["attn_chunk"], plan["attn_max_splits"] = v[32], v[33]
    return plan


def describe_prefill_plan(cfg: dict, n: int, opt: Options | None = None) -> dict:
    """Projection plan of a prefill call over n rows (a function of the
    model, n and the batch-invariant flags only)."""
    c = model_cfg(cfg)
    out = np.zeros(30, np.int32)
    k = load().corun_describe_prefill_plan(C.byref(c), n, C.byref(opt) if opt else None, out.ctypes.data, 30)
    if k < 0:
        raise CorunError(k, last_error())
    v = out[:k].tolist()
    plan = {}
    for i, name in enumerate(("qkv", "o", "gate_up", "down", "router")):
        N, K, S, Kc, bm, bn = v[6 * i: 6 * i + 6]
        plan[name] = {"N": N, "K": K, "split_k": S, "k_chunk": Kc, "m_tile": bm, "n_tile": bn}
    return plan


SAMPLE_NOALLOC_MAX_ROWS = 1024


def sample_noalloc(logits, valid, positions, seeds, temperature, vocab=None, stream=None):
    """corun_sample_noalloc: seeded sampling of the rows of a device fp32
    logits tensor ([rows, ld] or [ld]) with no engine and no allocation;
    returns (tokens int32[rows], logprobs float32[rows])."""
    import torch
    assert logits.is_cuda and logits.dtype == torch.float32 and logits.is_contiguous()
    rows = 1 if logits.dim() == 1 else logits.shape[0]
    ld = logits.shape[-1]
    vocab = ld if vocab is None else vocab
    vm = _np(valid, np.uint8).reshape(rows)
    pos = _np(positions, np.int32).reshape(rows)
    sd = np.ascontiguousarray(np.asarray(seeds, dtype=np.uint64).reshape(rows))
    tp = np.ascontiguousarray(np.asarray(temperature, dtype=np.float32).reshape(rows))
    tok = np.empty(rows, np.int32)
    lp = np.empty(rows, np.float32)
    if stream is None:
        stream = torch.cuda.current_stream()
    _check(load().corun_sample_noalloc(logits.data_ptr(), ld, rows, vocab, vm.ctypes.data, pos.ctypes.data,
                                       sd.ctypes.data, tp.ctypes.data, tok.ctypes.data, lp.ctypes.data,
                                       C.c_void_p(stream.cuda_stream)))
    return tok, lp


class SchedCfg(C.Structure):
    _fields_ = [("max_num_reqs", C.c_int32), ("n_slots", C.c_int32), ("max_seq_len", C.c_int32),
                ("page_size", C.c_int32), ("num_pages", C.c_int32), ("max_pages_per_seq", C.c_int32),
                ("prefill_chunk", C.c_int32), ("prefill_batch_tokens", C.c_int32)]


class Scheduler:
    """Host scheduler over an Engine (or a dry run with engine=None):
    isolated prefill (Algorithms 1 and 2), fixed-shape decode and
    request-bound sampling, with slot reuse and full-sequence admission."""

    IDLE, PREFILL, DECODE = 0, 1, 2

    def __init__(self, engine=None, max_num_reqs=0, n_slots=0, max_seq_len=0, page_size=0, num_pages=0,
                 max_pages_per_seq=0, prefill_chunk=0, prefill_batch_tokens=0):
        self._L = load()
        self.engine = engine
        cfg = SchedCfg(max_num_reqs, n_slots, max_seq_len, page_size, num_pages, max_pages_per_seq, prefill_chunk,
                       prefill_batch_tokens)
        h = C.c_void_p()
        st = self._L.corun_sched_create(engine._h if engine is not None else None, C.byref(cfg), C.byref(h))
        if st != 0:
            raise CorunError(st, self._L.corun_sched_last_error().decode())
        self._h = h
        self.B = engine.B if engine is not None else n_slots

    def _ok(self, st):
        if st != 0:
            raise CorunError(st, self._L.corun_sched_last_error().decode())

    def add_request(self, rid: int, prompt, max_new_tokens: int, seed: int = 0, temperature: float = 0.0):
        p = _np(prompt, np.int32)
        self._ok(self._L.corun_sched_add_request(self._h, rid, p.ctypes.data, p.size, max_new_tokens, seed,
                                                 temperature))

    def step(self) -> int:
        ev = C.c_int32()
        self._ok(self._L.corun_sched_step(self._h, C.byref(ev)))
        return ev.value

    def output(self, rid: int):
        n = C.c_int32()
        fin = C.c_int32()
        self._ok(self._L.corun_sched_output(self._h, rid, None, None, 0, C.byref(n), C.byref(fin)))
        tok = np.empty(max(n.value, 1), np.int32)
        lp = np.empty(max(n.value, 1), np.float32)
        self._ok(self._L.corun_sched_output(self._h, rid, tok.ctypes.data, lp.ctypes.data, n.value, C.byref(n),
                                            C.byref(fin)))
        return tok[:n.value], lp[:n.value], bool(fin.value)

    def state(self) -> dict:
        r, w, fs, fp = C.c_int32(), C.c_int32(), C.c_int32(), C.c_int32()
        owner = np.empty(self.B, np.int64)
        self._ok(self._L.corun_sched_state(self._h, C.byref(r), C.byref(w), C.byref(fs), C.byref(fp),
                                           owner.ctypes.data))
        return dict(running=r.value, waiting=w.value, free_slots=fs.value, free_pages=fp.value, slot_owner=owner)

    def run_until_idle(self, max_steps: int = 1 << 20) -> list:
        events = []
        for _ in range(max_steps):
            ev = self.step()
            if ev == self.IDLE:
                return events
            events.append(ev)
        raise RuntimeError("scheduler did not drain")

    def close(self):
        if getattr(self, "_h", None):
            self._L.corun_sched_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def torch_float32():
    import torch
    return torch.float32


class Engine:
    """One fixed-B engine.  `weights` is a workload.Weights of device bf16
    tensors; `k`, `v` lists of per-layer device bf16 cache tensors."""

    def __init__(self, cfg: dict, weights, B: int, k, v, layout=KV_CONTIGUOUS, page_size=0, page_table=None,
                 opt: Options | None = None, stream=None):
        import torch
        L = load()
        self.cfg, self.B = cfg, B
        self._keep = [weights, k, v, page_table]
        keep = self._keep
        w = weights
        self._w = Weights(w.embed.data_ptr(), w.final_norm.data_ptr(), w.lm_head.data_ptr(),
                          _ptr_array(w.attn_norm, keep), _ptr_array(w.w_qkv, keep), _ptr_array(w.w_o, keep),
                          _ptr_array(w.mlp_norm, keep), _ptr_array(w.w_gate_up, keep), _ptr_array(w.w_down, keep),
                          _ptr_array(w.w_router, keep), _ptr_array(w.w_exp_gate_up, keep),
                          _ptr_array(w.w_exp_down, keep))
        if layout == KV_PAGED:
            num_pages, _, ps, _ = k[0].shape
            assert ps == page_size
            n_slots, mpp = page_table.shape
            self._kv = kv_struct(layout, n_slots, k, v, keep, 0, page_size, num_pages, mpp, page_table)
            self.capacity = mpp * page_size
        else:
            n_slots, _, S, _ = k[0].shape
            self._kv = kv_struct(layout, n_slots, k, v, keep, max_seq_len=S)
            self.capacity = S
        self._cfg = model_cfg(cfg)
        self._opt = opt if opt is not None else options()
        if stream is None:
            stream = torch.cuda.current_stream()
        self._stream = stream
        h = C.c_void_p()
        _check(L.corun_engine_create(C.byref(self._cfg), C.byref(self._w), C.byref(self._kv), B,
                                     C.byref(self._opt), C.c_void_p(stream.cuda_stream), C.byref(h)))
        self._h = h
        self._L = L

    def close(self):
        if getattr(self, "_h", None):
            self._L.corun_engine_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def plan(self) -> dict:
        return describe_plan(self.cfg, self._kv, self.B, self._opt)

    def set_page_table_host(self, pt) -> None:
        """Register a host int32 [n_slots, max_pages_per_seq] copy of the
        device page table for the host-side checks (None unregisters); the
        array is kept alive here and must be kept equal to the device table."""
        if pt is None:
            self._pt_host = None
            _check(self._L.corun_engine_set_page_table_host(self._h, None))
            return
        assert isinstance(pt, np.ndarray) and pt.dtype == np.int32 and pt.flags.c_contiguous
        self._pt_host = pt
        _check(self._L.corun_engine_set_page_table_host(self._h, pt.ctypes.data))

    def decode_step(self, tokens, valid, seq_lens, logits=None) -> np.ndarray:
        t, vm, s = _np(tokens, np.int32), _np(valid, np.uint8), _np(seq_lens, np.int32)
        assert t.size == vm.size == s.size == self.B
        nxt = np.empty(self.B, np.int32)
        if logits is not None:
            assert logits.is_cuda and logits.dtype.is_floating_point and logits.numel() == self.B * self.cfg["vocab"]
        _check(self._L.corun_decode_step(self._h, t.ctypes.data, vm.ctypes.data, s.ctypes.data, nxt.ctypes.data,
                                         None if logits is None else logits.data_ptr()))
        return nxt

    def decode_run(self, n_steps, tokens, valid, seq_lens) -> np.ndarray:
        t, vm, s = _np(tokens, np.int32), _np(valid, np.uint8), _np(seq_lens, np.int32)
        out = np.empty((n_steps, self.B), np.int32)
        _check(self._L.corun_decode_run(self._h, n_steps, t.ctypes.data, vm.ctypes.data, s.ctypes.data,
                                        out.ctypes.data))
        return out

    def routing_trace(self, source: int = 0):
        """(sel int32 [L, rows, top_k], router logits float32 [L, rows, E]) of
        the last decode step (source 0) or prefill call (source 1); needs an
        engine created with record_routing."""
        L, k, E = self.cfg["n_layers"], self.cfg["top_k"], self.cfg["n_experts"]
        rows = C.c_int32()
        _check(self._L.corun_routing_trace(self._h, source, None, None, C.byref(rows)))
        n = rows.value
        sel = np.empty((L, n, k), np.int32)
        lg = np.empty((L, n, E), np.float32)
        _check(self._L.corun_routing_trace(self._h, source, sel.ctypes.data, lg.ctypes.data, C.byref(rows)))
        return sel, lg

    def time_kernel(self, kernel: int, layer: int = 0, n_iters: int = 20) -> float:
        """Mean launch duration in microseconds (HIP events, engine stream)."""
        us = C.c_float()
        _check(self._L.corun_time_kernel(self._h, kernel, layer, n_iters, C.byref(us)))
        return float(us.value)

    def profile_step(self, n_steps: int = 3):
        """{kernel name: (mean in-step launch duration in us, launches per
        step)} over n_steps eagerly launched steps with HIP events around
        every launch (corun_profile_step)."""
        us = np.zeros(len(KERNEL_NAMES), np.float32)
        n = np.zeros(len(KERNEL_NAMES), np.int32)
        _check(self._L.corun_profile_step(self._h, n_steps, us.ctypes.data, n.ctypes.data))
        return {KERNEL_NAMES[k]: (float(us[k]), int(n[k])) for k in range(len(KERNEL_NAMES)) if n[k]}

    def sample(self, logits, valid, positions, seeds, temperature):
        """Seeded sampling of the rows of a device fp32 logits tensor
        ([rows, vocab] or [vocab] for one row): (tokens int32[rows],
        logprobs float32[rows])."""
        assert logits.is_cuda and logits.dtype == torch_float32() and logits.is_contiguous()
        rows = 1 if logits.dim() == 1 else logits.shape[0]
        ld = logits.shape[-1]
        vm = _np(valid, np.uint8).reshape(rows)
        pos = _np(positions, np.int32).reshape(rows)
        sd = np.ascontiguousarray(np.asarray(seeds, dtype=np.uint64).reshape(rows))
        tp = np.ascontiguousarray(np.asarray(temperature, dtype=np.float32).reshape(rows))
        tok = np.empty(rows, np.int32)
        lp = np.empty(rows, np.float32)
        _check(self._L.corun_sample(self._h, logits.data_ptr(), ld, rows, vm.ctypes.data, pos.ctypes.data,
                                    sd.ctypes.data, tp.ctypes.data, tok.ctypes.data, lp.ctypes.data))
        return tok, lp

    def prefill(self, prompt, slot: int, last_logits=None) -> int:
        p = _np(prompt, np.int32)
        tok = np.empty(1, np.int32)
        _check(self._L.corun_prefill(self._h, p.ctypes.data, p.size, slot, tok.ctypes.data,
                                     None if last_logits is None else last_logits.data_ptr()))
        return int(tok[0])

    def prefill_batch(self, prompts, slots, last_logits=None) -> np.ndarray:
        """Several whole prompts in one batch-invariant pass (engine created
        with bi_prefill or batch_invariant); returns their first tokens.
        last_logits: a device fp32 tensor [len(prompts), vocab], or None."""
        ps = [_np(p, np.int32) for p in prompts]
        toks = np.ascontiguousarray(np.concatenate(ps), np.int32)
        lens = np.array([p.size for p in ps], np.int32)
        sl = _np(slots, np.int32)
        out = np.empty(len(ps), np.int32)
        _check(self._L.corun_prefill_batch(self._h, toks.ctypes.data, lens.ctypes.data, sl.ctypes.data, len(ps),
                                           out.ctypes.data,
                                           None if last_logits is None else last_logits.data_ptr()))
        return out

    def prefill_chunk(self, tokens, start: int, slot: int, last_logits=None, want_token=True):
        """Positions start .. start+len(tokens)-1 of a prompt whose earlier
        positions are already cached in `slot`; returns the greedy token of
        the chunk's last position (None for an inner chunk: want_token False
        and no last_logits)."""
        p = _np(tokens, np.int32)
        tok = np.empty(1, np.int32)
        _check(self._L.corun_prefill_chunk(self._h, p.ctypes.data, p.size, start, slot,
                                           tok.ctypes.data if want_token else None,
                                           None if last_logits is None else last_logits.data_ptr()))
        return int(tok[0]) if want_token else None
