#!/usr/bin/env python3
"""Decode throughput of the padded fixed-shape step on one MI355X.

Workload: the 8B-shaped dense decoder (36 layers, hidden 4096, 32 query / 8
KV heads, head_dim 128, SwiGLU 12288, vocab 151936) with seeded random bf16
weights; a fixed padded batch B whose live-row fraction is uniform in
[0.25, 1] (live slots a random subset); contiguous per-slot KV cache with
context lengths uniform in [512, 4096] and N(0, 1) contents.  A "step" is one
padded decode step over all B slots (the whole path: embedding, 36 layers,
lm_head, greedy argmax), replayed from the captured graph with device-side
feedback between steps.  Throughput counts live rows only (padding is the
method's cost).

The headline is B = 256 (the paper's capture size); --sweep adds further
fixed sizes.  Alongside: per-kernel durations measured with HIP events on the
engine's stream, the roofline of the dominant kernel (against the published
peak, and against what a plain device copy reaches here), a bit-exactness
check across two batch mixes, and the CPU oracle timed on a bounded sample.
Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16
METRIC = "decode tokens/s at fixed padded B + % HBM/MFMA roofline; bit-exact across batch mixes"
LEN_LO, LEN_HI = 512, 4096


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_bytes_flops(cfg, B, lens_live, plan, swiglu_fused=False):
    """Algorithmic bytes (read + written) and flops of one launch of each
    kernel class (per-layer kernels repeat n_layers times per step), for the
    engine's plan (split-K factors, attention chunk).  A projection reads its
    weights once and its bf16 input rows, and writes its outputs: fp32
    split-K partials (split x rows x N), or bf16 activations where the
    gate/up epilogue applies SwiGLU; the consumers read those partials back
    (RMSNorm folds the O or down partials into the fp32 residual, the QKV
    epilogue folds the QKV partials, SwiGLU the gate/up partials).  Decode
    attention reads each live row's cached keys and values (seq_len + 1
    tokens per kv head) and q, and writes one (max, sum, acc[G][d]) fp32
    partial per (row, kv head, split); the merge reads them and writes o.
    The argmax reads the lm_head epilogue's per-64-column (value, index)
    partials.  Padding rows are counted in the projections (padding is the
    method's cost).  Mixture-of-experts projections count every expert's
    weights: at B = 128 with top-8 of 128 experts nearly all are touched."""
    from paper_2608_14376_amd import corun
    H, d, nq, nkv, F, V = (cfg[k] for k in ("hidden", "head_dim", "n_heads", "n_kv_heads", "ffn", "vocab"))
    E, k, Fe = cfg["n_experts"], cfg["top_k"], cfg["expert_ffn"]
    G = nq // nkv
    nqkv = (nq + 2 * nkv) * d
    S = {n: plan[n]["split_k"] for n in ("qkv", "o", "gate_up", "down", "lm_head")}
    chunk = plan["attn_chunk"]

    def gemm(N, K, out_bytes, rows=B, mats=1):
        return 2 * N * K * mats + 2 * rows * K + out_bytes * rows * N, 2 * rows * N * K

    n_live = len(lens_live)
    kv_read = sum(int(L) + 1 for L in lens_live) * nkv * d * 2 * 2
    n_part = sum((int(L) + chunk) // chunk for L in lens_live) * nkv     # (row, kv head, split) partials
    part_bytes = n_part * G * (d + 2) * 4
    fold = lambda s_: B * H * 4 * (s_ + 1) + (B * H * 4 if s_ else 0) + B * H * 2 + H * 2   # x, partials in; x, h out
    dense_S = 0 if E else S["down"]
    bf = {
        corun.K_QKV_GEMM: gemm(nqkv, H, 4 * S["qkv"]),
        corun.K_O_GEMM: gemm(H, nq * d, 4 * S["o"]),
        corun.K_LM_HEAD: (2 * V * H + 2 * B * H + 4 * B * V + 8 * B * ((V + 63) // 64), 2 * B * V * H),
        corun.K_ATTN_SPLIT: (kv_read + 2 * n_live * nq * d + part_bytes,
                             4 * n_live * nq * d * (sum(lens_live) / max(n_live, 1) + 1)),
        corun.K_ATTN_MERGE: (part_bytes + 2 * B * nq * d, 0),
        # the 2 L + 1 norms of a step: L fold the O partials, L + 1 the down partials (or the expert combine)
        corun.K_RMSNORM: ((cfg["n_layers"] * fold(S["o"]) + (cfg["n_layers"] + 1) * fold(dense_S))
                          // (2 * cfg["n_layers"] + 1), 0),
        corun.K_QKV_POST: (4 * S["qkv"] * B * nqkv + 2 * B * nq * d + n_live * 2 * nkv * d * 2, 0),
        corun.K_ARGMAX: (8 * B * ((V + 63) // 64) + 4 * B, 0),
    }
    gv = all((plan[n]["m_tile"], plan[n]["n_tile"]) == (16, 16) for n in ("qkv", "o", "gate_up", "down"))
    if gv:
        # the small-batch layer: projections from fragment-packed copies (K
        # padded to 32), no split-K; qkv and gate/up read the fp32 residual,
        # the gain and the 16-column sums of squares (their norm), qkv writes
        # q and the appended k, v, gate/up the bf16 activations; o and down
        # read and write the residual and write the sums of squares; the one
        # RMSNorm of the step (the final one) reads x and writes h
        Kp = lambda K: (K + 31) // 32 * 32
        norm_in = 4 * B * H + 2 * H + 4 * B * (H // 16)
        resid = 8 * B * H + 4 * B * (H // 16)
        bf[corun.K_QKV_GEMM] = (2 * nqkv * Kp(H) + norm_in + 2 * B * nq * d + n_live * 2 * nkv * d * 2,
                                2 * B * nqkv * H)
        bf[corun.K_O_GEMM] = (2 * H * Kp(nq * d) + 2 * B * nq * d + resid, 2 * B * H * nq * d)
        bf[corun.K_GATE_UP_GEMM] = (2 * 2 * F * Kp(H) + norm_in + 2 * B * F, 2 * B * 2 * F * H)
        bf[corun.K_DOWN_GEMM] = (2 * H * Kp(F) + 2 * B * F + resid, 2 * B * H * F)
        bf[corun.K_RMSNORM] = (4 * B * H + 2 * B * H + 2 * H, 0)
        return bf
    if E:
        bf[corun.K_MOE_ROUTER] = gemm(E, H, 4)
        bf[corun.K_GATE_UP_GEMM] = gemm(2 * Fe, H, 4, rows=n_live * k, mats=E)
        bf[corun.K_SWIGLU] = (n_live * k * (2 * Fe * 4 + Fe * 2), 0)
        bf[corun.K_DOWN_GEMM] = gemm(H, Fe, 4, rows=n_live * k, mats=E)
    else:
        # with SwiGLU in its epilogue the gate/up projection writes the bf16 activations instead
        bf[corun.K_GATE_UP_GEMM] = (gemm(2 * F, H, 0)[0] + 2 * B * F, gemm(2 * F, H, 0)[1]) if swiglu_fused else \
            gemm(2 * F, H, 4 * S["gate_up"])
        bf[corun.K_SWIGLU] = (4 * S["gate_up"] * B * 2 * F + B * F * 2, 0)
        bf[corun.K_DOWN_GEMM] = gemm(H, F, 4 * S["down"])
    return bf


def make_paged(cfg, B, lens, extra, seed):
    """Paged cache sized to the draw: each slot gets ceil((len + extra) / 16)
    pages from a seeded permutation of the page pool; unused table entries
    point at page 0."""
    import torch

    from paper_2608_14376_amd import workload as wl
    ps = 16
    need = [(int(L) + extra + ps - 1) // ps for L in lens]
    mpp = max(need)
    num_pages = sum(need)
    perm = np.random.default_rng(seed).permutation(num_pages).astype(np.int32)
    pt = np.zeros((B, mpp), np.int32)
    o = 0
    for b in range(B):
        pt[b, :need[b]] = perm[o:o + need[b]]
        o += need[b]
    K, V = wl.make_kv_paged(cfg, num_pages, ps, seed=2000 + B, device="cuda")
    return K, V, torch.from_numpy(pt).to("cuda"), ps


def run_B(cfg, W, B, args, seeds, measure_kernels, paged=False, len_lo=LEN_LO, len_hi=LEN_HI,
          log_uniform=False, live_frac=(0.25, 1.0)):
    import torch

    from paper_2608_14376_amd import corun
    from paper_2608_14376_amd import workload as wl

    extra = args.warmup + args.steps + 1
    t0 = time.time()
    batches = [wl.make_batch(B, cfg["vocab"], seed=sd, len_lo=len_lo, len_hi=len_hi, log_uniform=log_uniform,
                             live_frac=live_frac) for sd in seeds]
    if paged:
        assert len(seeds) == 1, "the paged cache is sized to one draw"
        K, V, pt, ps = make_paged(cfg, B, np.where(batches[0].valid == 1, batches[0].seq_lens, 0), extra, 3000 + B)
        eng = corun.Engine(cfg, W, B, K, V, layout=corun.KV_PAGED, page_size=ps, page_table=pt)
    else:
        K, V = wl.make_kv_contiguous(cfg, B, (len_hi + extra + 15) // 16 * 16, seed=1000 + B, device="cuda")
        eng = corun.Engine(cfg, W, B, K, V)
    torch.cuda.synchronize()
    log(f"[bench] {cfg['n_layers']}L H={cfg['hidden']} B={B} {'paged' if paged else 'contiguous'}: KV cache "
        f"{2 * len(K) * K[0].numel() * 2 / 1e9:.1f} GB ready in {time.time() - t0:.1f}s")
    runs = []
    for sd, b in zip(seeds, batches):
        n_live = int(b.valid.sum())
        eng.decode_run(args.warmup, b.tokens, b.valid, b.seq_lens)
        torch.cuda.synchronize()
        t = time.perf_counter()
        eng.decode_run(args.steps, b.tokens, b.valid, b.seq_lens)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t
        runs.append(dict(seed=sd, n_live=n_live, step_ms=1e3 * dt / args.steps,
                         live_tok_s=n_live * args.steps / dt, slot_tok_s=B * args.steps / dt,
                         lens=b.seq_lens[b.valid == 1].tolist(), batch=b))
        log(f"[bench] B={B} seed={sd} live={n_live} step={runs[-1]['step_ms']:.3f} ms "
            f"live tok/s={runs[-1]['live_tok_s']:.0f}")
    runs.sort(key=lambda r: r["live_tok_s"])
    med = runs[len(runs) // 2]
    kv_tok = wl.kv_bytes_per_token(cfg)
    res = dict(B=B, n_live=med["n_live"], step_ms=round(med["step_ms"], 4), live_tok_s=round(med["live_tok_s"], 1),
               slot_tok_s=round(med["slot_tok_s"], 1), seeds=[r["seed"] for r in runs],
               mean_context=round(float(np.mean(med["lens"])), 1),
               step_bytes_algorithmic=int(wl.streamed_weight_params(cfg) * 2 + kv_tok * (sum(med["lens"]) + 2 * len(med["lens"]))))
    res["step_hbm_frac"] = round(res["step_bytes_algorithmic"] / (med["step_ms"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
    if measure_kernels:
        # re-run the median seed's batch so the workspace holds its state;
        # every kernel is timed inside eagerly launched steps of that batch
        # (HIP events around each launch on the engine's stream)
        b = med["batch"]
        eng.decode_run(1, b.tokens, b.valid, b.seq_lens)
        prof = eng.profile_step(n_steps=args.profile_steps)
        bf = kernel_bytes_flops(cfg, B, med["lens"], eng.plan(), swiglu_fused=not cfg["n_experts"] and "swiglu" not in prof)
        kern = {}
        for k in bf:
            name = corun.KERNEL_NAMES[k]
            if name not in prof:
                continue        # runs inside a neighbouring kernel at this B (QKV epilogue, SwiGLU)
            us, per = prof[name]
            by, fl = bf[k]
            kern[name] = dict(us=round(us, 2), per_step=per, bytes=by, flops=fl, gbs=round(by / us / 1e3, 1),
                              tflops=round(fl / us / 1e6, 2))
            if by / us / 1e3 > HBM_PEAK_GBS:
                raise AssertionError(f"{name}: {by} algorithmic bytes in {us} us exceed the HBM peak")
        dom = max(kern, key=lambda n: kern[n]["us"] * kern[n]["per_step"])
        res["dominant_isolated_us"] = round(eng.time_kernel(corun.KERNEL_NAMES.index(dom), 0, args.kernel_iters), 2)
        gem = [corun.KERNEL_NAMES[k] for k in (corun.K_QKV_GEMM, corun.K_O_GEMM, corun.K_GATE_UP_GEMM,
                                               corun.K_DOWN_GEMM, corun.K_LM_HEAD)]
        g_us = sum(kern[n]["us"] * kern[n]["per_step"] for n in gem)
        g_by = sum(kern[n]["bytes"] * kern[n]["per_step"] for n in gem)
        g_fl = sum(kern[n]["flops"] * kern[n]["per_step"] for n in gem)
        tot_us = sum(v["us"] * v["per_step"] for v in kern.values())
        res["gemm_phase"] = dict(ms=round(g_us / 1e3, 4), hbm_frac=round(g_by / g_us / 1e3 / HBM_PEAK_GBS, 4),
                                 mfma_frac=round(g_fl / g_us / 1e6 / MFMA_BF16_PEAK_TFLOPS, 4))
        res["kernel_sum_ms"] = round(tot_us / 1e3, 4)
        res["kernels"] = kern
    res["_eng"], res["_K"], res["_V"], res["_med"] = eng, K, V, med
    if paged:
        res["_pt"], res["_ps"] = pt, ps
    return res


def _drop(res):
    for k in ("_eng", "_K", "_V", "_med", "_pt", "_ps"):
        res.pop(k, None)
    return res


def bench_prefill(cfg, W, lens, args):
    """Isolated prefill of one prompt per length (the paper's base case),
    timed end to end through corun_prefill (host prompt in, first token out).
    Algorithmic flops: 2 Lp (weights) + the causal attention's lower
    triangle 2 nq d Lp (Lp + 1) per layer."""
    import torch

    from paper_2608_14376_amd import corun
    from paper_2608_14376_amd import workload as wl
    Lmax = max(lens)
    K, V = wl.make_kv_contiguous(cfg, 1, (Lmax + 15) // 16 * 16, seed=4000, device="cuda")
    eng = corun.Engine(cfg, W, 1, K, V, opt=corun.options(max_prefill_len=Lmax))
    H, d, nq, L = cfg["hidden"], cfg["head_dim"], cfg["n_heads"], cfg["n_layers"]
    w_params = wl.streamed_weight_params(cfg) - cfg["vocab"] * H
    out = []
    eng.prefill(wl.make_prompt(cfg["vocab"], 256, seed=1), 0)          # warm-up
    for Lp in lens:
        prompt = wl.make_prompt(cfg["vocab"], Lp, seed=Lp)
        torch.cuda.synchronize()
        t = time.perf_counter()
        eng.prefill(prompt, 0)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t
        flops = 2 * Lp * w_params + 2 * H * cfg["vocab"] + L * 2 * nq * d * Lp * (Lp + 1)
        out.append(dict(Lp=Lp, ms=round(1e3 * dt, 3), tok_s=round(Lp / dt, 1),
                        tflops=round(flops / dt / 1e12, 1), mfma_frac=round(flops / dt / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)))
        log(f"[bench] prefill Lp={Lp}: {1e3 * dt:.1f} ms, {Lp / dt:.0f} tok/s, {flops / dt / 1e12:.0f} TFLOP/s")
    # chunked prefill of the longest prompt: fixed chunks run alone, in order
    prompt = wl.make_prompt(cfg["vocab"], Lmax, seed=Lmax)
    for C in (2048, 8192):
        if C >= Lmax:
            continue
        torch.cuda.synchronize()
        t = time.perf_counter()
        for start in range(0, Lmax, C):
            n = min(C, Lmax - start)
            eng.prefill_chunk(prompt[start:start + n], start, 0, want_token=start + n == Lmax)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t
        whole = next(o for o in out if o["Lp"] == Lmax)["ms"]
        out.append(dict(Lp=Lmax, chunk=C, ms=round(1e3 * dt, 3), tok_s=round(Lmax / dt, 1),
                        vs_whole=round(1e3 * dt / whole, 3)))
        log(f"[bench] prefill Lp={Lmax} in chunks of {C}: {1e3 * dt:.1f} ms ({1e3 * dt / whole:.2f}x the whole prompt)")
    eng.close()
    return out


def bench_scheduler(cfg, W, n_req=64, B=32, in_len=512, out_len=64, batch_tokens=None):
    """The host scheduler end to end on a synthetic in=512/out=64 workload:
    Algorithms 1 and 2 around the fixed-B decode with request-bound sampling
    (temperature 0.6, own seeds).  batch_tokens None: every request
    prefilled alone with the default prefill plan; else a batch-invariant
    prefill engine, 0 = one prompt per prefill iteration, > 0 = batched
    prefill of up to that many prompt tokens per iteration."""
    import torch

    from paper_2608_14376_amd import corun
    from paper_2608_14376_amd import workload as wl
    cap = (in_len + out_len + 15) // 16 * 16
    K, V = wl.make_kv_contiguous(cfg, B, cap, seed=5000, device="cuda")
    bi = batch_tokens is not None
    pf = max(in_len, batch_tokens or 0, 4096)         # the same prefill workspace in every mode
    eng = corun.Engine(cfg, W, B, K, V, opt=corun.options(max_prefill_len=pf, bi_prefill=bi))
    s = corun.Scheduler(eng, max_num_reqs=B, prefill_batch_tokens=batch_tokens or 0)
    for i in range(2):                                   # warm-up: graph capture, first prefill
        s.add_request(-1 - i, wl.make_prompt(cfg["vocab"], in_len, seed=9000 + i), 2, 1, 0.6)
    s.run_until_idle()
    for i in range(n_req):
        s.add_request(i, wl.make_prompt(cfg["vocab"], in_len, seed=7000 + i), out_len, 1000 + i, 0.6)
    torch.cuda.synchronize()
    t = time.perf_counter()
    events = s.run_until_idle()
    dt = time.perf_counter() - t
    s.close()
    eng.close()
    del K, V
    mode = ("isolated prefill" if not bi else
            "batch-invariant prefill, " + ("one prompt per iteration" if not batch_tokens else
                                           f"batched up to {batch_tokens} tokens"))
    out = dict(mode=mode, requests=n_req, B=B, input_len=in_len, output_len=out_len, seconds=round(dt, 3),
               output_tok_s=round(n_req * out_len / dt, 1), prefill_iterations=events.count(1),
               decode_steps=events.count(2))
    log(f"[bench] scheduler in={in_len}/out={out_len} x{n_req} at B={B}, {mode}: {dt:.2f} s, "
        f"{out['output_tok_s']:.0f} output tok/s ({out['prefill_iterations']} prefill iterations, "
        f"{out['decode_steps']} decode steps)")
    return out


def bench_bi_tradeoff(cfg, W, K, V, args):
    """The paper's trade-off on this GPU (Sec. I, Fig. 2 and Fig. 4b; Sec. V,
    "Ablation Study"), on the 8B-shaped model and the headline cache:

    * step: one decode step of 32 live requests with contexts U[512, 4096]
      under STD (the default plan at B = 32: no padding), BI (batch-invariant
      kernels at B = 32) and CoRun (the default plan at the fixed B = 256,
      224 padding rows), each with its per-kernel-class breakdown;
    * padding: one live request (context 2048) under CoRun at padded sizes
      1..256 against BI at B = 1 (STD is CoRun at B = 1);
    * gemm: each projection's launch time under the default and the
      batch-invariant plan at M = 1..256 (the MatMul panel of Fig. 2);
    * split_kv: the fixed B = 256 step with split-KV on and off, for ragged
      (U[512, 4096]) and similar (U[2000, 2100]) contexts."""
    import torch

    from paper_2608_14376_amd import corun
    from paper_2608_14376_amd import workload as wl

    groups = {"matmul": (corun.K_QKV_GEMM, corun.K_O_GEMM, corun.K_GATE_UP_GEMM, corun.K_DOWN_GEMM,
                         corun.K_LM_HEAD),
              "attention": (corun.K_ATTN_SPLIT, corun.K_ATTN_MERGE), "rmsnorm": (corun.K_RMSNORM,),
              "other": (corun.K_QKV_POST, corun.K_SWIGLU, corun.K_ARGMAX)}
    gemms = {"qkv": corun.K_QKV_GEMM, "o": corun.K_O_GEMM, "gate_up": corun.K_GATE_UP_GEMM,
             "down": corun.K_DOWN_GEMM, "lm_head": corun.K_LM_HEAD}
    cap = K[0].shape[2]

    def timed(B, b, opt=None, breakdown=False, gemm_times=False, rows=None):
        eng = corun.Engine(cfg, W, B, K, V, opt=opt)
        if rows is not None:       # the listed rows' logits of one step, before any timing
            lg = torch.empty(B, cfg["vocab"], dtype=torch.float32, device="cuda")
            eng.decode_step(b.tokens, b.valid, b.seq_lens, lg)
            rows_out = lg[rows].cpu()
            del lg
        eng.decode_run(args.warmup, b.tokens, b.valid, b.seq_lens)
        torch.cuda.synchronize()
        t = time.perf_counter()
        eng.decode_run(args.steps, b.tokens, b.valid, b.seq_lens)
        torch.cuda.synchronize()
        r = dict(step_ms=round(1e3 * (time.perf_counter() - t) / args.steps, 4))
        if breakdown or gemm_times:
            eng.decode_run(1, b.tokens, b.valid, b.seq_lens)
            prof = eng.profile_step(n_steps=args.profile_steps)      # in-step launch durations
        if breakdown:
            r["breakdown_ms"] = {g: round(sum(prof[corun.KERNEL_NAMES[k]][0] * prof[corun.KERNEL_NAMES[k]][1]
                                              for k in ks if corun.KERNEL_NAMES[k] in prof) / 1e3, 3)
                                 for g, ks in groups.items()}
        if gemm_times:
            r["gemm_us"] = {n: round(prof[corun.KERNEL_NAMES[k]][0], 2) for n, k in gemms.items()}
        eng.close()
        if rows is not None:
            r["_rows"] = rows_out
        return r

    def batch_at(B, slots, lens, seed):
        r = np.random.default_rng(seed)
        valid = np.zeros(B, np.uint8)
        valid[slots] = 1
        seq = r.integers(0, 1 << 30, B).astype(np.int32)          # padding rows: garbage
        seq[slots] = lens
        tok = r.integers(0, cfg["vocab"], B).astype(np.int32)
        return wl.Batch(tok, valid, seq)

    bi = corun.options(batch_invariant=True)
    out = {}
    # Fig. 4b: 32 live requests, ragged contexts, in slots 0..31 of the cache
    # under every mode, so each mode sees the same 32 requests
    lens32 = np.random.default_rng(11).integers(LEN_LO, LEN_HI + 1, 32)
    live = np.arange(32)
    b32 = batch_at(32, live, lens32, 12)
    b256 = batch_at(256, live, lens32, 14)
    b256.tokens[:32] = b32.tokens
    s = dict(std=timed(32, b32, breakdown=True, rows=live), bi=timed(32, b32, bi, breakdown=True, rows=live),
             corun_B256=timed(256, b256, breakdown=True, rows=live), bi_B256=timed(256, b256, bi, rows=live))
    same = lambda a, b: int(sum(torch.equal(a["_rows"][i].view(torch.int32), b["_rows"][i].view(torch.int32))
                                for i in range(32)))
    s["identical_rows_of_32"] = dict(default_B32_vs_B256=same(s["std"], s["corun_B256"]),
                                     bi_B32_vs_B256=same(s["bi"], s["bi_B256"]))
    for v in s.values():
        v.pop("_rows", None)
    out["step_32_live"] = s
    log(f"[bench] 32 live requests: STD {s['std']['step_ms']} ms, BI {s['bi']['step_ms']} ms, "
        f"CoRun(B=256) {s['corun_B256']['step_ms']} ms; rows bit-identical between B=32 and B=256: "
        f"default {s['identical_rows_of_32']['default_B32_vs_B256']}/32, "
        f"BI {s['identical_rows_of_32']['bi_B32_vs_B256']}/32")
    # decode padding: one live request; GEMM launch times at each M
    pad, gemm = {}, {}
    for B in (1, 2, 4, 8, 16, 32, 64, 128, 256):
        b = batch_at(B, [B - 1], [2048], 20 + B)
        r = timed(B, b, gemm_times=B in (1, 8, 32, 64, 128, 256))
        pad[B] = dict(step_ms=r["step_ms"], tok_s=round(1e3 / r["step_ms"], 1))
        if "gemm_us" in r:
            rb = timed(B, b, bi, gemm_times=True)
            gemm[B] = dict(std=r["gemm_us"], bi=rb["gemm_us"],
                           bi_over_std={n: round(rb["gemm_us"][n] / r["gemm_us"][n], 2) for n in gemms})
            if B == 1:
                pad["bi_B1"] = dict(step_ms=rb["step_ms"], tok_s=round(1e3 / rb["step_ms"], 1))
    out["padding_1_live"] = pad
    out["gemm_std_vs_bi_us"] = gemm
    log(f"[bench] one live request: CoRun B=1 {pad[1]['tok_s']} tok/s, B=256 {pad[256]['tok_s']} tok/s, "
        f"BI B=1 {pad['bi_B1']['tok_s']} tok/s")
    # split-KV on/off at the fixed B = 256
    sk = {}
    off = corun.options(attn_chunk=(cap + 63) // 64 * 64)
    for name, lo, hi in (("ragged", LEN_LO, LEN_HI), ("similar", 2000, 2100)):
        b = wl.make_batch(256, cfg["vocab"], seed=30, len_lo=lo, len_hi=hi)
        on_ms, off_ms = timed(256, b)["step_ms"], timed(256, b, off)["step_ms"]
        sk[name] = dict(n_live=int(b.valid.sum()), split_on_ms=on_ms, split_off_ms=off_ms,
                        off_cost=round(off_ms / on_ms - 1, 4))
    out["split_kv_B256"] = sk
    log(f"[bench] split-KV off at B=256: ragged {100 * sk['ragged']['off_cost']:+.1f}%, "
        f"similar {100 * sk['similar']['off_cost']:+.1f}%")
    # and at the small fixed sizes, where few rows leave most of the GPU idle without splits
    small = {}
    for Bs in (1, 8, 16):
        b = wl.make_batch(Bs, cfg["vocab"], seed=40 + Bs, len_lo=LEN_LO, len_hi=LEN_HI)
        on_ms, off_ms = timed(Bs, b)["step_ms"], timed(Bs, b, off)["step_ms"]
        small[Bs] = dict(n_live=int(b.valid.sum()), split_on_ms=on_ms, split_off_ms=off_ms,
                         off_cost=round(off_ms / on_ms - 1, 4))
    out["split_kv_small_B"] = small
    log("[bench] split-KV off, ragged contexts: " + ", ".join(f"B={k} {100 * v['off_cost']:+.1f}%"
                                                            for k, v in small.items()))
    return out


def bitexact_check(cfg, res, n_pairs=2):
    """One live request placed in two different batch mixes at two different
    slots: logits rows must be bit-identical."""
    import torch

    from paper_2608_14376_amd import workload as wl
    eng, K, V, B = res["_eng"], res["_K"], res["_V"], res["B"]
    ok = 0
    r = np.random.default_rng(7)
    logits = torch.empty(B, cfg["vocab"], dtype=torch.float32, device="cuda")
    for pair in range(n_pairs):
        tok, L = int(r.integers(0, cfg["vocab"])), int(r.integers(LEN_LO, LEN_HI))
        s1, s2 = (int(x) for x in r.choice(B, 2, replace=False)) if B > 1 else (0, 0)
        rows = []
        saved = [(k[s1].clone(), v[s1].clone()) for k, v in zip(K, V)]
        for slot, seed in ((s1, 500 + pair), (s2, 600 + pair)):
            b = wl.make_batch(B, cfg["vocab"], seed=seed, len_lo=LEN_LO, len_hi=LEN_HI)
            for l in range(len(K)):            # the request's cache, restored into `slot`
                K[l][slot].copy_(saved[l][0])
                V[l][slot].copy_(saved[l][1])
            b.tokens[slot], b.seq_lens[slot], b.valid[slot] = tok, L, 1
            eng.decode_step(b.tokens, b.valid, b.seq_lens, logits)
            rows.append(logits[slot].clone())
        ok += int(torch.equal(rows[0].view(torch.int32), rows[1].view(torch.int32)))
    return dict(pairs=n_pairs, identical=ok)


def time_sampler(cfg, res, iters=20):
    """Request-bound seeded sampling of the headline batch's B rows of
    logits (temperature 0.6, per-row seeds), end to end through
    corun_sample: host arrays in, tokens and log-probabilities out (H2D,
    the sampling kernel, D2H, one synchronisation)."""
    import torch
    eng, B, med = res["_eng"], res["B"], res["_med"]
    b = med["batch"]
    logits = torch.empty(B, cfg["vocab"], dtype=torch.float32, device="cuda")
    eng.decode_step(b.tokens, b.valid, b.seq_lens, logits)
    pos = (b.seq_lens.astype(np.int64) + 1).astype(np.int32)
    seeds = np.arange(B, dtype=np.uint64) * np.uint64(2654435761) + np.uint64(42)
    temp = np.full(B, 0.6, np.float32)
    eng.sample(logits, b.valid, pos, seeds, temp)
    torch.cuda.synchronize()
    t = time.perf_counter()
    for _ in range(iters):
        eng.sample(logits, b.valid, pos, seeds, temp)
    dt = (time.perf_counter() - t) / iters
    del logits
    return dict(B=B, rows_live=int(b.valid.sum()), ms_per_call=round(1e3 * dt, 4), temperature=0.6,
                note="host arrays in, tokens + log-probabilities out; one synchronisation")


def host_cpu():
    """The host the CPU baseline runs on: lscpu's model name, logical CPUs,
    physical cores (distinct (physical id, core id) pairs of /proc/cpuinfo),
    sockets, and the CPUs this process may run on."""
    import subprocess
    info = {}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=20).stdout
        for ln in out.splitlines():
            k, _, v = ln.partition(":")
            info[k.strip()] = v.strip()
    except (OSError, subprocess.SubprocessError):
        pass
    cores, pid, cid = set(), None, None
    try:
        for ln in list(open("/proc/cpuinfo")) + [""]:
            if ln.startswith("physical id"):
                pid = ln.split(":", 1)[1].strip()
            elif ln.startswith("core id"):
                cid = ln.split(":", 1)[1].strip()
            elif not ln.strip():
                if pid is not None or cid is not None:
                    cores.add((pid, cid))
                pid = cid = None
    except OSError:
        pass
    return dict(model=info.get("Model name") or _cpu_name(), logical_cpus=os.cpu_count(),
                physical_cores=len(cores) or None, sockets=info.get("Socket(s)"),
                affinity_cpus=len(os.sched_getaffinity(0)))


def cpu_baseline(cfg, W, res, budget_s=12.0):
    """The oracle (plain C, fp64 between bf16 storage points, row by row,
    OpenMP across output features) on bounded samples of the workloads:

    * decode, extrapolated: live rows of the headline batch with their real
      caches through layers 0-1 plus lm_head (until budget_s), the per-layer
      time scaled to all layers;
    * decode, full depth: one live row through every layer and lm_head,
      measured, which validates that extrapolation;
    * prefill, extrapolated: a 64-token prompt through layer 0 plus the
      last row's lm_head; per token and layer, scaled to a 512-token prompt
      through all layers."""
    import oracle
    from paper_2608_14376_amd import workload as wl
    oracle.build()
    threads = oracle.get_threads()
    L = cfg["n_layers"]
    b = wl.bits

    def model(n):
        c = dict(cfg, n_layers=n)
        return oracle.Model(c, b(W.embed), b(W.final_norm), b(W.lm_head), [b(t) for t in W.attn_norm[:n]],
                            [b(t) for t in W.w_qkv[:n]], [b(t) for t in W.w_o[:n]], [b(t) for t in W.mlp_norm[:n]],
                            [b(t) for t in W.w_gate_up[:n]], [b(t) for t in W.w_down[:n]])

    m2 = model(2)
    K, V, med = res["_K"], res["_V"], res["_med"]
    cap = K[0].shape[2]
    bb = wl.make_batch(res["B"], cfg["vocab"], seed=med["seed"], len_lo=LEN_LO, len_hi=LEN_HI)
    live = np.nonzero(bb.valid)[0]
    h = np.zeros(cfg["hidden"], np.uint16)
    t = time.perf_counter()
    oracle.linear(h, m2.lm_head)
    t_lm = time.perf_counter() - t
    t2, n = 0.0, 0
    t_start = time.perf_counter()
    for slot in live:
        kv = oracle.KVCache([b(K[l][slot:slot + 1]) for l in range(2)], [b(V[l][slot:slot + 1]) for l in range(2)],
                            oracle.KV_CONTIGUOUS, 1, cap)
        t = time.perf_counter()
        oracle.decode_row(m2, kv, 0, int(bb.tokens[slot]), int(bb.seq_lens[slot]))
        t2 += time.perf_counter() - t
        n += 1
        if time.perf_counter() - t_start > budget_s:
            break
    per_row_2 = t2 / n
    per_layer = max(per_row_2 - t_lm, 1e-9) / 2
    full_extrap = per_layer * L + t_lm
    # full depth, measured: the first sampled row again, through every layer
    slot = int(live[0])
    mL = model(L)
    kv = oracle.KVCache([b(K[l][slot:slot + 1]) for l in range(L)], [b(V[l][slot:slot + 1]) for l in range(L)],
                        oracle.KV_CONTIGUOUS, 1, cap)
    t = time.perf_counter()
    oracle.decode_row(mL, kv, 0, int(bb.tokens[slot]), int(bb.seq_lens[slot]))
    full_meas = time.perf_counter() - t
    del mL, kv
    # prefill: 64 tokens through layer 0 and the last row's lm_head
    m1 = model(1)
    lp = 64
    kv1 = oracle.KVCache([np.zeros((1, cfg["n_kv_heads"], lp, cfg["head_dim"]), np.uint16)],
                         [np.zeros((1, cfg["n_kv_heads"], cfg["head_dim"], lp), np.uint16)], oracle.KV_CONTIGUOUS, 1, lp)
    t = time.perf_counter()
    oracle.prefill(m1, kv1, 0, wl.make_prompt(cfg["vocab"], lp, seed=3))
    t_pf = time.perf_counter() - t
    per_tok_layer = max(t_pf - t_lm, 1e-9) / lp
    pf_lp = 512
    pf_tok_s = pf_lp / (pf_lp * L * per_tok_layer + t_lm)
    return dict(value=round(1.0 / full_meas, 4), unit="tokens/s", cores=threads, kind="oracle",
                sample=f"one live row of the B={res['B']} headline batch (context {int(bb.seq_lens[slot])}) through "
                       f"all {L} layers and lm_head, measured: {full_meas:.2f} s per token",
                decode_extrapolated=dict(tok_s=round(1.0 / full_extrap, 4), s_per_token=round(full_extrap, 3),
                                         sample=f"{n} live rows through layers 0-1 + lm_head ({per_row_2:.3f} s/row, "
                                                f"lm_head {t_lm:.3f} s), scaled to {L} layers",
                                         extrapolated_over_measured=round(full_extrap / full_meas, 4)),
                prefill_extrapolated=dict(Lp=pf_lp, tok_s=round(pf_tok_s, 3),
                                          sample=f"{lp}-token prompt through layer 0 + last-row lm_head "
                                                 f"({t_pf:.2f} s), per token and layer scaled to {L} layers"),
                threads=threads, host=host_cpu())


def kernel_source_sha():
    import hashlib
    h = hashlib.sha256()
    for f in ("kernels.hip", "kernels.h"):
        h.update(open(os.path.join(ROOT, "paper_2608_14376_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def read_summary(path):
    """The `key: value` lines of a profiles/ summary, with the kernel-source
    hash from its `# kernel_source_sha256_16:` header line; other comment
    lines are skipped."""
    kv = {}
    for ln in open(path):
        ln = ln.strip()
        if ln.startswith("#"):
            body = ln.lstrip("#").strip()
            if body.startswith("kernel_source_sha256_16:"):
                kv["kernel_source_sha256_16"] = body.split(":", 1)[1].strip()
            continue
        if ":" in ln:
            k, v = ln.split(":", 1)
            kv[k.strip()] = v.strip()
    return kv


def measured_traffic(kernel, B, seed):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary of this workload (FETCH_SIZE and WRITE_SIZE, each scaled by what
    the counter reads for a plain copy of known size), or None when no
    summary exists or the kernels have changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_8b_B{B}_seed{seed}.txt")
    if not os.path.exists(path):
        return None, None
    kv = read_summary(path)
    if kv.get("kernel_source_sha256_16") != kernel_source_sha():
        return None, os.path.relpath(path, ROOT) + " (stale: kernels changed since the counters were taken)"
    return int(float(kv["traffic_bytes_per_launch"])), os.path.relpath(path, ROOT)


def _cpu_name():
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def achievable_peaks():
    """What this device reaches on plain vendor work, reported beside the
    published peaks: HBM reads from a row-wise sum over a 1 GiB fp32 matrix
    (65536 x 4096; the fastest of torch's plain reductions measured here),
    HBM read + write from a 1 GiB device-to-device copy, bf16 matrix-core
    throughput from an 8192^3 bf16 matmul (torch's vendor GEMM); best of 10
    launches each, timed with HIP events on torch's current stream, where
    they run.  1 GiB is four times the last-level cache."""
    import torch

    def best_ms(fn, n=10):
        fn()
        best = float("inf")
        for _ in range(n):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            e1.synchronize()
            best = min(best, e0.elapsed_time(e1))
        return best

    x = torch.ones(65536, 4096, dtype=torch.float32, device="cuda")
    rd = x.numel() * 4 / (best_ms(lambda: x.sum(1)) * 1e-3) / 1e9
    del x
    src = torch.empty(1 << 29, dtype=torch.int16, device="cuda")
    dst = torch.empty_like(src)
    cp = 2 * src.numel() * 2 / (best_ms(lambda: dst.copy_(src)) * 1e-3) / 1e9
    del src, dst
    n = 8192
    g = torch.Generator(device="cuda").manual_seed(0)
    a = torch.randn(n, n, device="cuda", dtype=torch.bfloat16, generator=g)
    b = torch.randn(n, n, device="cuda", dtype=torch.bfloat16, generator=g)
    mfma = 2 * n ** 3 / (best_ms(lambda: torch.matmul(a, b)) * 1e-3) / 1e12
    del a, b
    torch.cuda.empty_cache()
    return dict(hbm_read_gbs=round(rd, 1), hbm_read_source="row sums of a 65536 x 4096 fp32 matrix (1 GiB read)",
                hbm_copy_gbs=round(cp, 1), hbm_copy_source="1 GiB device-to-device copy, (read + written bytes) / time",
                mfma_bf16_tflops=round(mfma, 1), mfma_source="8192^3 bf16 matmul through torch (vendor GEMM)")


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=32)
    ap.add_argument("--warmup", type=int, default=4)
    ap.add_argument("--B", type=int, default=256, help="headline fixed batch size")
    ap.add_argument("--sweep", default="1,8,16,64", help="further fixed batch sizes (comma list, '' for none)")
    ap.add_argument("--seeds", type=int, default=5, help="batch seeds at the headline B (median reported)")
    ap.add_argument("--first-seed", type=int, default=1, help="first batch seed at the headline B")
    ap.add_argument("--kernel-iters", type=int, default=10,
                    help="back-to-back launches of the dominant kernel for its isolated duration (context only)")
    ap.add_argument("--profile-steps", type=int, default=3,
                    help="eagerly launched steps with events around every launch, for the in-step kernel durations")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the 32B paged, MoE and prefill workloads")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run one plain 1 GiB device copy (reference for HBM traffic counters)")
    ap.add_argument("--prefill-only", default="",
                    help="profiling aid: time only the isolated prefill of these prompt lengths (comma list) "
                         "and print their results as one JSON line instead of the decode benchmark")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the decode step and prefill here run on a single MI355X; "
              "multi-GPU sharding is a design note only, so --gpus must be 1.", file=sys.stderr)
        sys.exit(2)
    if args.warmup + args.steps > 127:
        sys.exit("warmup + steps must stay below 128 (cache capacity is 4096 + 128 tokens)")

    import torch

    from paper_2608_14376_amd import corun
    from paper_2608_14376_amd import workload as wl
    corun.load()
    cfg = wl.config("8b")
    t0 = time.time()
    W = wl.make_weights(cfg, seed=0, device="cuda")
    torch.cuda.synchronize()
    log(f"[bench] weights {wl.streamed_weight_params(cfg) * 2 / 1e9:.2f} GB streamed per step, "
        f"made in {time.time() - t0:.1f}s")
    if args.prefill_only:
        lens = [int(x) for x in args.prefill_only.split(",") if x.strip()]
        print(json.dumps({"prefill_8b": bench_prefill(cfg, W, lens, args)}), flush=True)
        return

    head = run_B(cfg, W, args.B, args, seeds=list(range(args.first_seed, args.first_seed + args.seeds)),
                 measure_kernels=True)
    bitexact = bitexact_check(cfg, head)
    log(f"[bench] bit-exact across batch mixes: {bitexact}")
    sampler = time_sampler(cfg, head)
    log(f"[bench] seeded sampler at B={sampler['B']}: {sampler['ms_per_call']} ms per call")
    cpu = None if args.no_cpu_baseline else cpu_baseline(cfg, W, head)
    if cpu:
        log(f"[bench] cpu oracle: {cpu['value']} tok/s measured at full depth on {cpu['cores']} threads "
            f"({cpu['host']['model']}, {cpu['host']['physical_cores']} physical cores); extrapolated "
            f"{cpu['decode_extrapolated']['tok_s']} tok/s, prefill {cpu['prefill_extrapolated']['tok_s']} tok/s")
    tradeoff = None if args.no_extra else bench_bi_tradeoff(cfg, W, head["_K"], head["_V"], args)
    _drop(head)
    torch.cuda.empty_cache()

    sweep = []
    for Bs in [int(x) for x in args.sweep.split(",") if x.strip()]:
        if Bs == args.B:
            continue
        r = _drop(run_B(cfg, W, Bs, args, seeds=[1], measure_kernels=True))
        r.pop("kernels", None)
        sweep.append(r)
        torch.cuda.empty_cache()

    extra = {}
    if tradeoff is not None:
        extra["bi_tradeoff_8b"] = tradeoff
    if not args.no_extra:
        # prefill on the same 8B weights
        extra["prefill_8b"] = bench_prefill(cfg, W, [512, 2048, 8192, 32768], args)
        torch.cuda.empty_cache()
        extra["scheduler_8b"] = bench_scheduler(cfg, W)
        extra["scheduler_8b_bi_prefill"] = bench_scheduler(cfg, W, batch_tokens=0)
        extra["scheduler_8b_batched_prefill"] = bench_scheduler(cfg, W, batch_tokens=4096)
        del W
        torch.cuda.empty_cache()
        # 32B-shaped dense decode at long context on the paged cache
        c32 = wl.config("32b")
        W32 = wl.make_weights(c32, seed=0, device="cuda")
        r32 = run_B(c32, W32, 32, args, seeds=[1], measure_kernels=True, paged=True, len_lo=1024, len_hi=32768,
                    log_uniform=True, live_frac=(1.0, 1.0))
        r32["kernels"] = {k: v for k, v in r32["kernels"].items() if k in ("attn_split", "attn_merge", "gate_up_gemm")}
        # the same batch with split-KV off (one split covers a row's whole capacity): the analogue of
        # the paper's ablation at long, ragged contexts
        b32 = r32["_med"]["batch"]
        cap32 = r32["_pt"].shape[1] * r32["_ps"]
        e_off = corun.Engine(c32, W32, 32, r32["_K"], r32["_V"], layout=corun.KV_PAGED, page_size=r32["_ps"],
                             page_table=r32["_pt"], opt=corun.options(attn_chunk=(cap32 + 63) // 64 * 64))
        e_off.decode_run(args.warmup, b32.tokens, b32.valid, b32.seq_lens)
        torch.cuda.synchronize()
        t = time.perf_counter()
        e_off.decode_run(args.steps, b32.tokens, b32.valid, b32.seq_lens)
        torch.cuda.synchronize()
        off_ms = 1e3 * (time.perf_counter() - t) / args.steps
        e_off.close()
        del e_off                      # it holds the 32B weights and cache
        r32["split_kv_off"] = dict(step_ms=round(off_ms, 4), off_cost=round(off_ms / r32["step_ms"] - 1, 4))
        log(f"[bench] 32B B=32 split-KV off: {off_ms:.3f} ms per step ({100 * (off_ms / r32['step_ms'] - 1):+.1f}%)")
        extra["decode_32b_paged"] = _drop(r32)
        del W32, b32
        torch.cuda.empty_cache()
        # MoE decode
        cm = wl.config("moe")
        Wm = wl.make_weights(cm, seed=0, device="cuda")
        rm = run_B(cm, Wm, 128, args, seeds=[1], measure_kernels=True)
        rm["kernels"] = {k: v for k, v in rm["kernels"].items()
                         if k in ("gate_up_gemm", "down_gemm", "moe_router", "attn_split")}
        extra["decode_moe"] = _drop(rm)
        del Wm
        torch.cuda.empty_cache()
    peaks = achievable_peaks()          # before the calibration copy, which stays the run's last dispatch
    if args.calibrate_copy:
        src = torch.empty(1 << 29, dtype=torch.int16, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log("[bench] calibration copy: 1 GiB read + 1 GiB written")

    log(f"[bench] achievable on this device: HBM read {peaks['hbm_read_gbs']} GB/s (row sums), "
        f"read + write {peaks['hbm_copy_gbs']} GB/s (device copy), "
        f"bf16 MFMA {peaks['mfma_bf16_tflops']} TFLOP/s (vendor GEMM)")
    for r in [head] + sweep:
        r["step_hbm_frac_of_achievable"] = round(r["step_hbm_frac"] * HBM_PEAK_GBS / peaks["hbm_read_gbs"], 4)
        gp = r.get("gemm_phase")
        if gp:
            gp["hbm_frac_of_achievable"] = round(gp["hbm_frac"] * HBM_PEAK_GBS / peaks["hbm_read_gbs"], 4)
    g = head.get("gemm_phase")
    if g:
        g["mfma_frac_of_achievable"] = round(g["mfma_frac"] * MFMA_BF16_PEAK_TFLOPS / peaks["mfma_bf16_tflops"], 4)
    kern = head["kernels"]
    dom_name, dom = max(kern.items(), key=lambda kv: kv[1]["us"] * kv[1]["per_step"])
    traffic, traffic_src = measured_traffic(dom_name, args.B, head["seeds"][len(head["seeds"]) // 2])
    roof = dict(kernel=dom_name, bound="hbm", achieved=dom["gbs"], peak=HBM_PEAK_GBS, unit="GB/s",
                frac=round(dom["gbs"] / HBM_PEAK_GBS, 4), traffic=traffic,
                bytes_per_launch=dom["bytes"], us_per_launch=dom["us"],
                us_source=f"mean of the kernel's launches inside {args.profile_steps} steps of the median batch "
                          f"(HIP events on the engine stream around each launch)",
                us_per_launch_isolated=head.get("dominant_isolated_us"), traffic_source=traffic_src,
                achievable_peak=peaks["hbm_read_gbs"], frac_of_achievable=round(dom["gbs"] / peaks["hbm_read_gbs"], 4))
    out = {
        "metric": METRIC,
        "value": head["live_tok_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["step_ms"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "8B-shaped dense decode, fixed padded B", "B": args.B,
                   "live_fraction": "U[0.25, 1]", "context": f"U[{LEN_LO}, {LEN_HI}]", "kv": "contiguous",
                   "weights": "seeded N(0, 0.02) bf16", "steps_per_seed": args.steps, "seeds": args.seeds},
        "roofline": roof,
        "cpu_baseline": cpu,
        "achievable_peaks": peaks,
        "bitexact_across_batch_mixes": bitexact,
        "sampler": sampler,
        "headline": head,
        "sweep": sweep,
        "extra": extra,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
