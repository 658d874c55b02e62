// engine.cpp -- host side of the C ABI in include/corun.h: validation, the
// per-B launch plan, workspace, and the captured decode graph.
//
// The plan is a pure function of (model shape, B, cache capacity, options):
// it is computed once at creation and never looks at which rows are live.
// That is what makes the fixed-shape step position-invariant end to end
// (Sec. IV, "Fixed-Shape Batched Decode"; Sec. III, Definition 2).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "corun.h"
#include "kernels.h"

using namespace corun;

namespace {

thread_local std::string g_err;

corun_status fail(corun_status s, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

#define HIP_TRY(expr)                                                                            \
    do {                                                                                         \
        hipError_t e_ = (expr);                                                                  \
        if (e_ != hipSuccess) return fail(CORUN_E_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
    } while (0)

#define ST_TRY(expr)                     \
    do {                                 \
        corun_status s_ = (expr);        \
        if (s_ != CORUN_OK) return s_;   \
    } while (0)

int kv_capacity(const corun_kv *kv)
{
    return kv->layout == CORUN_KV_PAGED ? kv->max_pages_per_seq * kv->page_size : kv->max_seq_len;
}

// One projection: N outputs, K inputs, split-K into S chunks of Kc, run by
// the skinny kernel (bm = 0), the LDS-tiled kernel with M tile bm (bn = 0)
// or the pipelined kernel with bm x bn tiles (bn > 0).
struct Proj {
    int N = 0, K = 0, S = 1, Kc = 0, bm = 0, bn = 0;
};

struct Plan {
    int B = 0, Mp = 0, mt = 1;
    // gv: the small-batch layer -- qkv, o, gate/up and down on the
    // fragment-packed projection kernel (launch_gemv), no split-K anywhere:
    // o and down add into the residual, qkv and gate/up normalise their
    // input on the fly, RoPE + KV append and SwiGLU run in their epilogues,
    // so a layer launches no RMSNorm, QKV-epilogue or SwiGLU kernel
    bool gv = false;
    Proj qkv, o, gu, down, lm, router;
    int moe_slots = 0;   // tile slots of the expert projections: E + ceil(B top_k / 16)
    int chunk = 0, max_splits = 0;
};

int mt_for(int M) { return M <= 16 ? 1 : (M <= 32 ? 2 : 4); }

// Kernel, tile and split-K factor from the projection shape and M only.
//  * M <= 64, K % 64 == 0: the pipelined kernel with a 32- or 64-row tile
//    and 128 columns, split-K to about 256 workgroups (each split at least
//    512 K elements).  Against the skinny kernel it streams weights in
//    whole lines and needs a third to a quarter of the split-K partials that
//    the next kernel folds.
//  * M <= 64, K % 64 != 0: the skinny kernel (weights streamed to
//    registers); aim for about 2048 wavefronts (8 per CU) so enough weight
//    bytes are in flight, each split keeping at least 256 K elements.
//  * 64 < M <= 256, K % 64 == 0: the pipelined kernel (one workgroup per
//    CU) with M tile 128 (M <= 128, and the narrower projections up to 256)
//    or 256 and N tile 128; 256 x 256 tiles (eight wavefronts) for wide
//    decode projections (128 < M <= 256, N >= 16384: gate/up, lm_head);
//    split-K up to one round of at most 256 workgroups, each split keeping
//    at least 512 K elements.
//  * M > 256 (prefill), K % 64 == 0: the pipelined kernel with the tile
//    (256 x 256, 256 x 128, 128 x 128) and split-K of least estimated time
//    (waves of 256 workgroups, per-tile wave costs, the partials' traffic).
//  * otherwise (or bm_override > 0): the LDS-tiled kernel with a 128-row
//    tile (or bm_override), split-K to about two workgroups per CU.
// Batch-invariant mode (bi): no split-K and, when K % 64 == 0, the
// pipelined kernel for every M (else the LDS-tiled kernel's 128-row tile),
// so every output element is one chain of v_mfma_f32_32x32x16_bf16 over K in
// order whatever the batch size.  The tile still follows M (occupancy): an
// element's arithmetic does not depend on the tile it sits in.
Proj choose_proj(int N, int K, int M, int split_override, int max_split, int bm_override, bool bi = false)
{
    Proj p;
    p.N = N;
    p.K = K;
    if (N <= 0 || K <= 0 || M <= 0) return p;   // no such projection
    int S, align;
    if (bi) {
        if (K % 64 == 0) return choose_proj(N, K, M, 0, 1, 0, false);
        p.bm = 128;
        p.bn = 0;
        p.Kc = (K + 63) / 64 * 64;
        p.S = 1;
        return p;
    }
    if (M <= 64 && bm_override <= 0 && K % 64 == 0) {
        p.bm = M <= 32 ? 32 : 64;
        p.bn = 128;
        const int tiles = (N + 127) / 128;
        S = std::max(1, 256 / tiles);
        S = std::min(S, std::max(1, K / 512));
        align = 64;
    } else if (M > 256 && bm_override <= 0 && K % 64 == 0) {
        // Prefill-sized M: the tile and split-K with the least estimated
        // time, calibrated on this GPU's pipelined kernel.  A launch runs in
        // waves of 256 workgroups; a wave costs c x K / S with c = 1.69,
        // 1.0, 0.62 for 256 x 256, 256 x 128, 128 x 128 tiles (a 256 x 128
        // wave over 4096 K elements took 68.5 us), and each split beyond the
        // first adds a set of fp32 partials that is written and folded again
        // (8 bytes per output at about 5 TB/s).  Against measured times at
        // M = 512 .. 8192 the estimate picks the fastest tile, or one within
        // a few percent.
        struct Cand {
            int bm, bn;
            double c;
        };
        const Cand cands[] = {{256, 256, 1.69}, {256, 128, 1.0}, {128, 128, 0.62}};
        const int smax = std::max(1, std::min(K / 512, max_split > 0 ? max_split : 64));
        double best = 1e300;
        S = 1;
        for (const Cand &cd : cands) {
            const long long tiles = (long long)((M + cd.bm - 1) / cd.bm) * ((N + cd.bn - 1) / cd.bn);
            for (int s = 1; s <= smax; s *= 2) {
                const double waves = (double)((tiles * s + 255) / 256);
                const double t = waves * cd.c * ((double)K / s) * (68.5 / 4096) + (s - 1) * (double)M * N * 8 / 5e6;
                if (t < best) {
                    best = t;
                    p.bm = cd.bm;
                    p.bn = cd.bn;
                    S = s;
                }
            }
        }
        align = 64;
    } else if (M > 64 && bm_override <= 0 && K % 64 == 0) {
        // 128-row tiles up to M = 256 for the narrower projections (qkv, o,
        // down): about as fast as 256-row tiles there, with half the split-K
        // partials for the next kernel to fold; the decode step is 2% faster
        p.bm = (M <= 128 || (M <= 256 && N < 16384)) ? 128 : 256;
        p.bn = 128;
        const long long t256 = (long long)((M + 255) / 256) * ((N + 255) / 256);
        if ((M > 256 && t256 >= 256) || (M > 128 && M <= 256 && N >= 16384)) p.bn = 256;
        long long tiles = (long long)((M + p.bm - 1) / p.bm) * ((N + p.bn - 1) / p.bn);
        S = tiles >= 256 ? 1 : (int)(256 / tiles);
        S = std::min(S, std::max(1, K / 512));
        if (max_split > 0 && S > max_split && p.bm == 256 && tiles * max_split < 256) {
            // the workspace leaves too little room for split-K: fill the GPU
            // with 128 x 128 tiles instead
            p.bm = 128;
            p.bn = 128;
            tiles = (long long)((M + 127) / 128) * ((N + 127) / 128);
            S = tiles >= 256 ? 1 : (int)(256 / tiles);
            S = std::min(S, std::max(1, K / 512));
        }
        align = 64;
    } else if (M <= 64 && bm_override <= 0) {
        const int col_waves = (N + 63) / 64;
        const int mt = mt_for(M);
        const int m_tiles = (M + 16 * mt - 1) / (16 * mt);
        S = (2048 + col_waves * m_tiles - 1) / (col_waves * m_tiles);
        S = std::min(S, std::max(1, K / 256));
        align = 32;
    } else {
        p.bm = bm_override > 0 ? bm_override : 128;
        const int tiles = ((M + p.bm - 1) / p.bm) * ((N + 127) / 128);
        const int target = p.bm == 256 ? 256 : 512;
        S = (target + tiles - 1) / tiles;
        S = std::min(S, std::max(1, K / 512));
        align = 64;
    }
    if (max_split > 0) S = std::min(S, max_split);
    if (split_override > 0) S = split_override;
    S = std::max(1, std::min(S, (K + align - 1) / align));
    p.Kc = ((K + S - 1) / S + align - 1) / align * align;
    p.S = (K + p.Kc - 1) / p.Kc;
    return p;
}

GemmShape shape_of(const Proj &p, int M) { return GemmShape{M, p.N, p.K, p.S, p.Kc, mt_for(M), p.bm, p.bn, 0}; }

// Attention chunk: fixed per engine from (B, kv heads, capacity): the
// smallest power of two from 128 tokens up to 1024 for which the (row, head,
// split) blocks of a batch at capacity number at most 2048, four rounds of
// the 512 blocks the CUs hold at once (two per CU).  Measured on the
// 8B-shaped decode with contexts U[512, 4096]: B = 1 fastest at 128, B = 8 at
// 256 (4.07 against 4.29 ms at 128; with the QKV epilogue in attention every
// block refolds its q), B = 16 at 512 (1.5% over 256), B = 32 within noise
// from 256 to 1024.
int choose_chunk(int B, int nkv, int cap, int override_chunk)
{
    if (override_chunk > 0) return override_chunk;
    int chunk = 128;   // below 128 tokens some of the four wavefronts get no 32-token block
    while (chunk < 1024 && (long long)B * nkv * ((cap + chunk - 1) / chunk) > 2048) chunk *= 2;
    return chunk;
}

Plan make_plan(const corun_model_cfg *c, const corun_kv *kv, int B, const corun_options &opt)
{
    Plan p;
    p.B = B;
    p.mt = mt_for(B);
    p.Mp = (B + 63) / 64 * 64;
    const int H = c->hidden, d = c->head_dim;
    const int nqkv = (c->n_heads + 2 * c->n_kv_heads) * d;
    const int so = opt.split_k_override, bo = opt.gemm_bm;
    const bool bi = opt.batch_invariant != 0;
    p.qkv = choose_proj(nqkv, H, B, so, 0, bo, bi);
    p.o = choose_proj(H, c->n_heads * d, B, so, 0, bo, bi);
    if (c->n_experts == 0) {
        p.gu = choose_proj(2 * c->ffn, H, B, so, 0, bo, bi);
        p.down = choose_proj(H, c->ffn, B, so, 0, bo, bi);
    } else {
        p.router = choose_proj(c->n_experts, H, B, so, 0, bo, bi);
        p.gu = Proj{2 * c->expert_ffn, H, 1, H, 0};
        p.down = Proj{H, c->expert_ffn, 1, c->expert_ffn, 0};
        p.moe_slots = c->n_experts + (B * c->top_k + 15) / 16;
    }
    // lm_head: never split (its epilogue selects the argmax partials) except
    // under the split override test aid; the 64-row tile has no argmax epilogue
    p.lm = choose_proj(c->vocab, H, B, so > 0 ? so : 1, 0, bo == 64 ? 0 : bo, bi);
    if (p.lm.bm == 64 && p.lm.bn == 0) p.lm = choose_proj(c->vocab, H, 64, so > 0 ? so : 1, 0, 0);
    // lm_head at 128 < M <= 256: 256 x 128 tiles (two wavefronts per 128
    // rows, 64-column wavefront tiles, as the argmax epilogue needs) stream
    // the vocabulary faster than 256 x 256 tiles: 393 against 435 us at
    // M = 256 over 151936 x 4096.  Same K order per element, same bits.
    if (p.lm.bm == 256 && p.lm.bn == 256 && B <= 256 && p.lm.S == 1) p.lm.bn = 128;
    // The small-batch layer (small_batch_layer): automatic for dense models
    // at B = 1 (its kernels stream the fragment-packed copies the engine
    // makes, so not with no_weight_pack, nor under the tuning overrides or
    // batch-invariant mode).  At B = 1 it drops both RMSNorm launches of a
    // layer and the QKV fold in attention: the 8B-shaped step measured 3.58
    // against 3.77 ms.  At B = 8 the eight rows' norm, recomputed by every
    // workgroup, and its projections' in-step rate (the pipelined kernel's
    // 32-row tiles stream faster there) made it 5.3-5.5 against 4.2 ms; it
    // can still be asked for up to B = 8.
    const bool gv_ok = !bi && c->n_experts == 0 && !opt.no_weight_pack && opt.qkv_epilogue == 0 && so == 0 &&
                       bo == 0 && c->hidden % 256 == 0 && c->head_dim % 16 == 0;
    p.gv = opt.small_batch_layer == 1 ? gv_ok && B <= 8 : (opt.small_batch_layer == 0 && gv_ok && B == 1);
    if (p.gv) {
        for (Proj *pr : {&p.qkv, &p.o, &p.gu, &p.down}) {
            pr->S = 1;
            pr->Kc = (pr->K + 31) / 32 * 32;
            pr->bm = 16;
            pr->bn = 16;
        }
    }
    const int cap = kv_capacity(kv);
    // batch-invariant mode turns split-KV off: one split covers the capacity
    p.chunk = bi ? (cap + 63) / 64 * 64 : choose_chunk(B, c->n_kv_heads, cap, opt.attn_chunk);
    p.max_splits = (cap + p.chunk - 1) / p.chunk;
    return p;
}

}  // namespace

namespace {
// Projection weights, for the tile-packed copies the engine may hold.
enum WeightId { W_QKV, W_O, W_GATE_UP, W_DOWN, W_ROUTER, W_LM_HEAD, W_EXP_GATE_UP, W_EXP_DOWN, W_COUNT };
}  // namespace

struct corun_engine {
    corun_model_cfg c{};
    corun_kv kv{};
    corun_options opt{};
    int B = 0;
    Plan plan;
    hipStream_t user = nullptr, st = nullptr;
    hipEvent_t ev = nullptr;

    const uint16_t *embed = nullptr, *final_norm = nullptr, *lm_head = nullptr;
    std::vector<const uint16_t *> attn_norm, w_qkv, w_o, mlp_norm, w_gu, w_down, w_router, w_egu, w_edown;
    // tile-packed copies (per layer; one for lm_head) of the projections
    // whose decode plan streams weights with the small-M pipelined kernel;
    // empty = that projection reads the row-major weight only
    std::vector<const uint16_t *> packed[W_COUNT];
    // fragment-packed copies (per layer) for the small-batch layer (plan.gv):
    // qkv in rotation pairs, o, gate/up in feature pairs, down
    std::vector<const uint16_t *> gvw[4];
    char *pk_buf = nullptr;
    size_t pk_bytes = 0;
    bool gu_fused = false;   // the gate/up copy is interleaved for the fused SwiGLU epilogue
    bool egu_fused = false;  // likewise for every expert's gate/up (mixture of experts)
    bool qkv_in_attn = false;   // decode attention applies the QKV epilogue (no k_qkv_post launch)
    bool moe = false;
    // mixture-of-experts workspace (decode)
    float *p_router = nullptr, *moe_w = nullptr, *moe_gu = nullptr, *moe_y = nullptr;
    int32_t *moe_sel = nullptr, *moe_list = nullptr, *moe_tiles = nullptr;
    uint16_t *moe_act = nullptr;
    // and prefill
    float *pf_moe_w = nullptr, *pf_moe_gu = nullptr, *pf_moe_y = nullptr;
    int32_t *pf_moe_sel = nullptr, *pf_moe_list = nullptr, *pf_moe_tiles = nullptr;
    uint16_t *pf_moe_act = nullptr;
    // routing record (record_routing): [L][B] decode rows, [L][max_prefill_len]
    // prefill rows; pf_trace_rows = the rows of the last prefill call
    int32_t *rt_sel = nullptr, *rt_pf_sel = nullptr;
    float *rt_logit = nullptr, *rt_pf_logit = nullptr;
    int pf_trace_rows = 0;
    bool decoded = false;   // a decode step has uploaded inputs
    // corun_profile_step: every kernel of an eager step timed by events around
    // its own execution; a launch of kernel class `kind` is the recorder's
    // launches [first, end)
    struct ProfRec {
        int kind;
        size_t first, end;
    };
    bool profiling = false;
    std::vector<ProfRec> prof;
    LaunchRecorder rec;
    std::vector<uint16_t *> kc, vc;
    KvView view{};
    // paged caches: the caller's host copy of the page table
    // (corun_engine_set_page_table_host), read by the host-side checks
    // instead of copying the device table back on every call
    const int32_t *pt_host = nullptr;

    // decode workspace (one allocation)
    char *ws = nullptr;
    size_t ws_bytes = 0;
    int32_t *d_tokens = nullptr, *d_seq = nullptr, *d_next = nullptr, *d_hist = nullptr, *d_counter = nullptr;
    int32_t *d_order = nullptr, *h_order = nullptr;   // attention's row dispatch order
    uint8_t *d_valid = nullptr;
    float *gss = nullptr;   // plan.gv: sums of squares of 16-column groups of x, [B][hidden / 16]
    float *x = nullptr, *p_qkv = nullptr, *p_o = nullptr, *p_gu = nullptr, *p_down = nullptr, *attn_ws = nullptr,
          *logits = nullptr, *p_lm = nullptr;
    ArgBest *amax = nullptr;
    uint16_t *h = nullptr, *q = nullptr, *o = nullptr, *a = nullptr;
    float2 *rope = nullptr;
    int hist_cap = 0;

    // pinned host staging
    int32_t *h_tok = nullptr, *h_seq = nullptr, *h_next = nullptr, *h_counter = nullptr, *h_hist = nullptr;
    uint8_t *h_valid = nullptr;
    // seeded sampling: device inputs/outputs [B] and one pinned host block
    uint8_t *d_svalid = nullptr;
    int32_t *d_spos = nullptr, *d_stok = nullptr;
    uint64_t *d_sseed = nullptr;
    float *d_stemp = nullptr, *d_slp = nullptr;
    char *h_samp = nullptr;

    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;

    // prefill workspace
    int pf_max = 0;
    char *pws = nullptr;
    size_t pws_bytes = 0;
    float *pf_x = nullptr, *pf_part = nullptr, *pf_logits = nullptr;
    uint16_t *pf_h = nullptr, *pf_q = nullptr, *pf_o = nullptr, *pf_a = nullptr, *pf_hlast = nullptr;
    int32_t *pf_pos = nullptr, *pf_tok = nullptr, *pf_next = nullptr;
    int32_t *pf_rowpos = nullptr, *pf_rowslot = nullptr, *pf_seq = nullptr;   // batched prefill
    ArgBest *pf_amax = nullptr;
    size_t pf_part_elems = 0;
};

// ---------------------------------------------------------------------------
// Host-side checks
// ---------------------------------------------------------------------------

extern "C" corun_status corun_check_config(const corun_model_cfg *c, const corun_kv *kv, int32_t B)
{
    if (!c || !kv) return fail(CORUN_E_INVAL, "null config");
    if (c->n_layers <= 0 || c->hidden <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 || c->vocab <= 0)
        return fail(CORUN_E_SHAPE, "non-positive model dimension");
    if (c->hidden % 256 != 0) return fail(CORUN_E_SHAPE, "hidden must be a multiple of 256");
    if (c->head_dim != 64 && c->head_dim != 128) return fail(CORUN_E_SHAPE, "head_dim must be 64 or 128");
    if (c->n_heads % c->n_kv_heads != 0) return fail(CORUN_E_SHAPE, "n_heads must be a multiple of n_kv_heads");
    const int G = c->n_heads / c->n_kv_heads;
    if (!(G == 1 || G == 2 || G == 4 || G == 8 || (G == 16 && c->head_dim == 128)))
        return fail(CORUN_E_SHAPE, "unsupported query-group size %d", G);
    if (c->vocab % 16 != 0) return fail(CORUN_E_SHAPE, "vocab must be a multiple of 16");
    if (c->n_experts != 0) {
        if (c->n_experts < 1 || c->n_experts > 256) return fail(CORUN_E_SHAPE, "n_experts must be in [1, 256]");
        if (c->top_k < 1 || c->top_k > 16 || c->top_k > c->n_experts)
            return fail(CORUN_E_SHAPE, "top_k must be in [1, min(16, n_experts)]");
        if (c->expert_ffn <= 0 || c->expert_ffn % 16 != 0)
            return fail(CORUN_E_SHAPE, "expert_ffn must be a positive multiple of 16");
    } else if (c->ffn <= 0 || c->ffn % 16 != 0) {
        return fail(CORUN_E_SHAPE, "ffn must be a positive multiple of 16");
    }
    if (!(c->rms_eps > 0.f) || !(c->rope_theta > 0.f)) return fail(CORUN_E_SHAPE, "bad eps or rope theta");
    if (B <= 0 || B > 1024) return fail(CORUN_E_SHAPE, "B_fixed must be in [1, 1024]");
    if (kv->n_slots < B) return fail(CORUN_E_CAPACITY, "KV cache has %d slots < B_fixed %d", kv->n_slots, B);
    if (kv->layout == CORUN_KV_CONTIGUOUS) {
        if (kv->max_seq_len <= 0 || kv->max_seq_len % 16 != 0)
            return fail(CORUN_E_CAPACITY, "max_seq_len must be a positive multiple of 16");
    } else if (kv->layout == CORUN_KV_PAGED) {
        if (kv->page_size <= 0 || kv->page_size % 16 != 0 || kv->num_pages <= 0 || kv->max_pages_per_seq <= 0)
            return fail(CORUN_E_CAPACITY, "bad paged-cache geometry (page_size must be a multiple of 16)");
    } else {
        return fail(CORUN_E_INVAL, "unknown KV layout %d", kv->layout);
    }
    return CORUN_OK;
}

extern "C" corun_status corun_check_batch(const corun_model_cfg *c, const corun_kv *kv, const int32_t *pt_host,
                                          int32_t B, const int32_t *tokens, const uint8_t *valid,
                                          const int32_t *seq_lens, int32_t n_steps)
{
    if (!c || !kv || !tokens || !valid || !seq_lens) return fail(CORUN_E_INVAL, "null argument");
    if (n_steps < 1) return fail(CORUN_E_INVAL, "n_steps must be >= 1");
    const long long cap = kv_capacity(kv);
    for (int b = 0; b < B; ++b) {
        if (!valid[b]) continue;
        if (tokens[b] < 0 || tokens[b] >= c->vocab)
            return fail(CORUN_E_INVAL, "row %d: token %d outside [0, %d)", b, tokens[b], c->vocab);
        if (seq_lens[b] < 0) return fail(CORUN_E_INVAL, "row %d: negative seq_len %d", b, seq_lens[b]);
        if ((long long)seq_lens[b] + n_steps > cap)
            return fail(CORUN_E_CAPACITY, "row %d: seq_len %d + %d steps exceeds capacity %lld", b, seq_lens[b],
                        n_steps, cap);
        if (kv->layout == CORUN_KV_PAGED && pt_host) {
            const long long last = ((long long)seq_lens[b] + n_steps - 1) / kv->page_size;
            for (long long j = 0; j <= last; ++j) {
                const int32_t pg = pt_host[(long long)b * kv->max_pages_per_seq + j];
                if (pg < 0 || pg >= kv->num_pages)
                    return fail(CORUN_E_CAPACITY, "row %d: page %lld maps to %d outside [0, %d)", b, j, pg,
                                kv->num_pages);
            }
        }
    }
    return CORUN_OK;
}

static corun_status check_options(const corun_options &o)
{
    if (o.attn_chunk < 0 || o.attn_chunk % 64 != 0)
        return fail(CORUN_E_INVAL, "attn_chunk must be a non-negative multiple of 64");
    if (o.max_prefill_len < 0) return fail(CORUN_E_INVAL, "negative max_prefill_len");
    if (o.split_k_override < 0) return fail(CORUN_E_INVAL, "negative split_k_override");
    if (!(o.gemm_bm == 0 || o.gemm_bm == 64 || o.gemm_bm == 128 || o.gemm_bm == 256))
        return fail(CORUN_E_INVAL, "gemm_bm must be 0, 64, 128 or 256");
    if (o.batch_invariant != 0 && o.batch_invariant != 1) return fail(CORUN_E_INVAL, "batch_invariant must be 0 or 1");
    if (o.bi_prefill != 0 && o.bi_prefill != 1) return fail(CORUN_E_INVAL, "bi_prefill must be 0 or 1");
    if (o.no_weight_pack != 0 && o.no_weight_pack != 1) return fail(CORUN_E_INVAL, "no_weight_pack must be 0 or 1");
    if (o.qkv_epilogue < 0 || o.qkv_epilogue > 2) return fail(CORUN_E_INVAL, "qkv_epilogue must be 0, 1 or 2");
    if (o.record_routing != 0 && o.record_routing != 1) return fail(CORUN_E_INVAL, "record_routing must be 0 or 1");
    if (o.small_batch_layer < 0 || o.small_batch_layer > 2)
        return fail(CORUN_E_INVAL, "small_batch_layer must be 0, 1 or 2");
    if (o.batch_invariant && (o.attn_chunk || o.split_k_override || o.gemm_bm))
        return fail(CORUN_E_INVAL, "batch_invariant fixes the plan: attn_chunk, split_k_override and gemm_bm must be 0");
    return CORUN_OK;
}

extern "C" int32_t corun_describe_plan(const corun_model_cfg *c, const corun_kv *kv, int32_t B,
                                       const corun_options *opt, int32_t *out, int32_t cap)
{
    corun_status s = corun_check_config(c, kv, B);
    if (s != CORUN_OK) return s;
    corun_options o{};
    if (opt) o = *opt;
    s = check_options(o);
    if (s != CORUN_OK) return s;
    Plan p = make_plan(c, kv, B, o);
    if (o.small_batch_layer == 1 && !p.gv) return fail(CORUN_E_INVAL, "small_batch_layer = 1 needs a dense model, "
                                                       "B_fixed <= 8, weight packing and no plan overrides");
    std::vector<int32_t> v = {p.B, p.Mp};
    for (const Proj *pr : {&p.qkv, &p.o, &p.gu, &p.down, &p.lm}) {
        v.push_back(pr->N);
        v.push_back(pr->K);
        v.push_back(pr->S);
        v.push_back(pr->Kc);
        v.push_back(pr->bm);
        v.push_back(pr->bn);
    }
    v.push_back(p.chunk);
    v.push_back(p.max_splits);
    const int n = std::min<int>((int)v.size(), cap);
    for (int i = 0; i < n; ++i) out[i] = v[i];
    return n;
}

extern "C" const char *corun_last_error(void) { return g_err.c_str(); }

// The calling thread's error message, for the entry points of other files.
namespace corun {
corun_status set_error(corun_status s, const char *msg)
{
    g_err = msg;
    return s;
}
}  // namespace corun

// ---------------------------------------------------------------------------
// Workspace carving
// ---------------------------------------------------------------------------
namespace {

struct Carver {
    size_t off = 0;
    template <class T>
    size_t take(T **slot, size_t n)
    {
        off = (off + 255) / 256 * 256;
        *slot = reinterpret_cast<T *>(off);   // relative; rebased after allocation
        off += sizeof(T) * n;
        return off;
    }
};

template <class T>
void rebase(T *&p, char *base)
{
    p = reinterpret_cast<T *>(base + reinterpret_cast<size_t>(p));
}

size_t proj_part_elems(const Proj &p, int M) { return (size_t)p.S * M * p.N; }

const uint16_t *row_major_weight(const corun_engine *e, int w, int l)
{
    switch (w) {
    case W_QKV: return e->w_qkv[l];
    case W_O: return e->w_o[l];
    case W_GATE_UP: return e->w_gu[l];
    case W_DOWN: return e->w_down[l];
    case W_ROUTER: return e->w_router[l];
    case W_EXP_GATE_UP: return e->w_egu[l];
    case W_EXP_DOWN: return e->w_edown[l];
    default: return e->lm_head;
    }
}

// Whether a plan's kernel reads tile-packed weights: the pipelined kernel's
// small-M configurations (32 or 64 x 128 tiles, 64-element stages).
bool takes_packed(const Proj &p) { return p.bn == 128 && (p.bm == 32 || p.bm == 64) && p.K % 64 == 0; }

// Projection `w` of layer l over `rows` rows of A: from the engine's
// tile-packed copy where it holds one and the plan's kernel takes it (the
// results are bit-identical), else from the caller's row-major weight.
hipError_t proj(corun_engine *e, const uint16_t *A, int lda, int w, int l, const Proj &pr, int rows, float *out,
                long long split_stride, int ldo, ArgBest *amax = nullptr)
{
    GemmShape g = shape_of(pr, rows);
    const uint16_t *W = row_major_weight(e, w, l);
    const std::vector<const uint16_t *> &pk = e->packed[w];
    if (!pk.empty() && takes_packed(pr) && !(w == W_GATE_UP && e->gu_fused)) {
        g.pk = 1;
        W = pk[w == W_LM_HEAD ? 0 : l];
    }
    return launch_proj(A, lda, W, g, out, split_stride, ldo, e->st, amax);
}

// Whether gate/up and SwiGLU run as one kernel for this plan: the engine
// holds the gate/up-interleaved packed copy and the plan takes it without
// split-K.  The epilogue computes what the SwiGLU kernel computes from the
// same fp32 sums, so both paths give the same bits.
bool gu_fuses(const corun_engine *e, const Proj &pr) { return e->gu_fused && takes_packed(pr) && pr.S == 1; }

// gate/up of layer l over `rows` rows of A with SwiGLU into act [rows][ffn]
hipError_t gate_up_swiglu(corun_engine *e, const uint16_t *A, int l, const Proj &pr, int rows, uint16_t *act)
{
    GemmShape g = shape_of(pr, rows);
    g.pk = 1;
    return launch_gemm_dma(A, e->c.hidden, e->packed[W_GATE_UP][l], g, nullptr, 0, e->c.ffn, e->st, nullptr, act);
}

// Buffers of one mixture-of-experts layer run over `rows` rows.
struct MoeBufs {
    const uint8_t *valid;
    float *router_part, *w, *gu, *y;
    int32_t *sel, *list, *tiles;
    uint16_t *act;
    int slots;
    // routing record (corun_options.record_routing): layer l's choice and
    // router logits at sel_trace + l rows top_k and logit_trace + l rows E
    int32_t *sel_trace = nullptr;
    float *logit_trace = nullptr;
};

corun_status moe_router(corun_engine *e, const MoeBufs &m, const uint16_t *h, int rows, const Proj &pr, int l)
{
    const corun_model_cfg &c = e->c;
    HIP_TRY(proj(e, h, c.hidden, W_ROUTER, l, pr, rows, m.router_part, (long long)rows * c.n_experts, c.n_experts));
    int32_t *st_l = m.sel_trace ? m.sel_trace + (size_t)l * rows * c.top_k : nullptr;
    float *lt_l = m.logit_trace ? m.logit_trace + (size_t)l * rows * c.n_experts : nullptr;
    HIP_TRY(launch_moe_route(m.router_part, pr.S, (long long)rows * c.n_experts, rows, c.n_experts, c.top_k, m.valid,
                             m.sel, m.w, e->st, st_l, lt_l));
    HIP_TRY(launch_moe_dispatch(m.sel, rows * c.top_k, c.n_experts, m.slots, m.list, m.tiles, e->st));
    return CORUN_OK;
}

// Expert gate/up on the pipelined kernel (hidden is a multiple of 64), from
// the packed copies when the engine holds them; with interleaved copies the
// epilogue applies SwiGLU into m.act and no SwiGLU kernel runs.
corun_status moe_expert_gate_up(corun_engine *e, const MoeBufs &m, const uint16_t *h, int l)
{
    const corun_model_cfg &c = e->c;
    const int Fe = c.expert_ffn, H = c.hidden;
    const std::vector<const uint16_t *> &pk = e->packed[W_EXP_GATE_UP];
    if (!pk.empty())
        HIP_TRY(launch_moe_gemm_dma(h, H, c.top_k, pk[l], (long long)packed_weight_elems(2 * Fe, H), true, 2 * Fe, H,
                                    m.list, m.tiles, m.slots, m.gu, e->egu_fused ? m.act : nullptr,
                                    e->egu_fused ? Fe : 2 * Fe, e->st));
    else
        HIP_TRY(launch_moe_gemm_dma(h, H, c.top_k, e->w_egu[l], (long long)2 * Fe * H, false, 2 * Fe, H, m.list,
                                    m.tiles, m.slots, m.gu, nullptr, 2 * Fe, e->st));
    return CORUN_OK;
}

// Expert down: the pipelined kernel when expert_ffn is a multiple of 64
// (packed or row-major), else the register-streaming kernel.
corun_status moe_expert_down(corun_engine *e, const MoeBufs &m, int l)
{
    const corun_model_cfg &c = e->c;
    const int Fe = c.expert_ffn, H = c.hidden;
    const std::vector<const uint16_t *> &pk = e->packed[W_EXP_DOWN];
    if (!pk.empty())
        HIP_TRY(launch_moe_gemm_dma(m.act, Fe, 1, pk[l], (long long)packed_weight_elems(H, Fe), true, H, Fe, m.list,
                                    m.tiles, m.slots, m.y, nullptr, H, e->st));
    else if (Fe % 64 == 0)
        HIP_TRY(launch_moe_gemm_dma(m.act, Fe, 1, e->w_edown[l], (long long)H * Fe, false, H, Fe, m.list, m.tiles,
                                    m.slots, m.y, nullptr, H, e->st));
    else
        HIP_TRY(launch_moe_gemm(m.act, Fe, 1, e->w_edown[l], (long long)H * Fe, H, Fe, m.list, m.tiles, m.slots, m.y,
                                H, e->st));
    return CORUN_OK;
}

MoeBufs decode_moe(corun_engine *e)
{
    return MoeBufs{e->d_valid, e->p_router, e->moe_w,     e->moe_gu,         e->moe_y,         e->moe_sel,
                   e->moe_list, e->moe_tiles, e->moe_act, e->plan.moe_slots, e->rt_sel, e->rt_logit};
}

// The residual fold that opens layer l (l = n_layers: the final norm): the
// previous layer's down-projection partials, or its expert combine.
MoeFold fold_of(corun_engine *e, const MoeBufs &m, int l)
{
    MoeFold f;
    if (e->moe && l > 0) {
        f.y = m.y;
        f.w = m.w;
        f.valid = m.valid;
        f.top_k = e->c.top_k;
    }
    return f;
}

// The small-batch layer's projections (plan.gv): which = 0 qkv (norm of x
// with attn_norm, RoPE + KV append), 1 o (into the residual), 2 gate/up
// (norm of x with mlp_norm, SwiGLU into a), 3 down (into the residual).
hipError_t gemv_proj(corun_engine *e, int which, int l)
{
    const corun_model_cfg &c = e->c;
    const Plan &p = e->plan;
    const int B = e->B, H = c.hidden;
    GemvIn in;
    GemvOut out;
    switch (which) {
    case 0:
        in.x = e->x;
        in.ss = e->gss;
        in.g = e->attn_norm[l];
        in.eps = c.rms_eps;
        out.q = e->q;
        out.kc = e->kc[l];
        out.vc = e->vc[l];
        out.kv = e->view;
        out.rope = e->rope;
        out.valid = e->d_valid;
        out.pos = e->d_seq;
        out.nq = c.n_heads;
        out.nkv = c.n_kv_heads;
        out.d = c.head_dim;
        return launch_gemv(e->gvw[0][l], B, p.qkv.N, H, GV_QKV, in, out, e->st);
    case 1:
        in.a = e->o;
        in.lda = c.n_heads * c.head_dim;
        out.x = e->x;
        out.ss = e->gss;
        return launch_gemv(e->gvw[1][l], B, H, p.o.K, GV_RESID, in, out, e->st);
    case 2:
        in.x = e->x;
        in.ss = e->gss;
        in.g = e->mlp_norm[l];
        in.eps = c.rms_eps;
        out.act = e->a;
        return launch_gemv(e->gvw[2][l], B, p.gu.N, H, GV_SWIGLU, in, out, e->st);
    default:
        in.a = e->a;
        in.lda = c.ffn;
        out.x = e->x;
        out.ss = e->gss;
        return launch_gemv(e->gvw[3][l], B, H, p.down.K, GV_RESID, in, out, e->st);
    }
}

// One kernel of layer l of the decode step; the step is these in order.
corun_status launch_one(corun_engine *e, int which, int l)
{
    const corun_model_cfg &c = e->c;
    const Plan &p = e->plan;
    const int B = e->B, H = c.hidden, d = c.head_dim, nq = c.n_heads, nkv = c.n_kv_heads, F = c.ffn;
    const int nqkv = (nq + 2 * nkv) * d;
    hipStream_t st = e->st;
    if (p.gv) {   // the small-batch layer: four projections, attention and its merge
        switch (which) {
        case CORUN_K_QKV_GEMM: HIP_TRY(gemv_proj(e, 0, l)); return CORUN_OK;
        case CORUN_K_O_GEMM: HIP_TRY(gemv_proj(e, 1, l)); return CORUN_OK;
        case CORUN_K_GATE_UP_GEMM: HIP_TRY(gemv_proj(e, 2, l)); return CORUN_OK;
        case CORUN_K_DOWN_GEMM: HIP_TRY(gemv_proj(e, 3, l)); return CORUN_OK;
        case CORUN_K_QKV_POST:
        case CORUN_K_SWIGLU: return CORUN_OK;
        case CORUN_K_RMSNORM:   // the step's only norm, the final one
            HIP_TRY(launch_rmsnorm(e->x, nullptr, 0, 0, B, H, e->final_norm, c.rms_eps, e->h, st));
            return CORUN_OK;
        default: break;
        }
    }
    switch (which) {
    case CORUN_K_QKV_GEMM: {
        HIP_TRY(proj(e, e->h, H, W_QKV, l, p.qkv, B, e->p_qkv, (long long)B * nqkv, nqkv));
        break;
    }
    case CORUN_K_QKV_POST:   // nothing to launch when attention applies the epilogue
        if (e->qkv_in_attn) break;
        HIP_TRY(launch_qkv_post(e->p_qkv, p.qkv.S, (long long)B * nqkv, B, e->d_valid, e->d_seq, nullptr, -1, nq,
                                nkv, d, e->rope, e->q, e->kc[l], e->vc[l], e->view, st));
        break;
    case CORUN_K_ATTN_SPLIT:
        HIP_TRY(launch_attn_split(e->q, B, e->d_valid, e->d_seq, nullptr, -1, nq, nkv, d, e->kc[l], e->vc[l],
                                  e->view, p.chunk, p.max_splits, e->attn_ws, st,
                                  e->qkv_in_attn ? QkvIn{e->p_qkv, p.qkv.S, (long long)B * nqkv, e->rope}
                                                 : QkvIn{},
                                  e->d_order));
        break;
    case CORUN_K_ATTN_MERGE:
        HIP_TRY(launch_attn_merge(e->attn_ws, B, e->d_valid, e->d_seq, nq, nkv, d, p.chunk, p.max_splits, e->o, st));
        break;
    case CORUN_K_O_GEMM: {
        HIP_TRY(proj(e, e->o, nq * d, W_O, l, p.o, B, e->p_o, (long long)B * H, H));
        break;
    }
    case CORUN_K_RMSNORM:   // the post-attention norm (folds the O partials)
        HIP_TRY(launch_rmsnorm(e->x, e->p_o, p.o.S, (long long)B * H, B, H, e->mlp_norm[l], c.rms_eps, e->h, st));
        break;
    case CORUN_K_MOE_ROUTER:
        if (!e->moe) return fail(CORUN_E_STATE, "dense model has no router");
        ST_TRY(moe_router(e, decode_moe(e), e->h, B, p.router, l));
        break;
    case CORUN_K_GATE_UP_GEMM:
        if (e->moe) {
            ST_TRY(moe_expert_gate_up(e, decode_moe(e), e->h, l));
        } else if (gu_fuses(e, p.gu)) {
            HIP_TRY(gate_up_swiglu(e, e->h, l, p.gu, B, e->a));
        } else {
            HIP_TRY(proj(e, e->h, H, W_GATE_UP, l, p.gu, B, e->p_gu, (long long)B * 2 * F, 2 * F));
        }
        break;
    case CORUN_K_SWIGLU:   // nothing to launch when the gate/up projection's epilogue does it
        if (e->moe) {
            const int Fe = c.expert_ffn;
            if (!e->egu_fused) HIP_TRY(launch_swiglu(e->moe_gu, 1, 0, B * c.top_k, Fe, e->moe_act, Fe, st));
        } else if (!gu_fuses(e, p.gu)) {
            HIP_TRY(launch_swiglu(e->p_gu, p.gu.S, (long long)B * 2 * F, B, F, e->a, F, st));
        }
        break;
    case CORUN_K_DOWN_GEMM:
        if (e->moe) {
            ST_TRY(moe_expert_down(e, decode_moe(e), l));
        } else {
            HIP_TRY(proj(e, e->a, F, W_DOWN, l, p.down, B, e->p_down, (long long)B * H, H));
        }
        break;
    case CORUN_K_LM_HEAD:
        if (p.lm.S == 1) {
            HIP_TRY(proj(e, e->h, H, W_LM_HEAD, 0, p.lm, B, e->logits, 0, c.vocab, e->amax));
        } else {   // test aid only: a split lm_head, reduced in split order
            HIP_TRY(proj(e, e->h, H, W_LM_HEAD, 0, p.lm, B, e->p_lm, (long long)B * c.vocab, c.vocab));
            HIP_TRY(launch_reduce_splits(e->p_lm, p.lm.S, (long long)B * c.vocab, (long long)B * c.vocab, e->logits,
                                         st));
        }
        break;
    case CORUN_K_ARGMAX:
        if (p.lm.S == 1)
            HIP_TRY(launch_argmax_partials(e->amax, B, gemm_col_blocks(c.vocab), e->d_valid, e->d_next, st));
        else
            HIP_TRY(launch_argmax(e->logits, B, c.vocab, e->d_valid, e->d_next, st));
        break;
    default:
        return fail(CORUN_E_INVAL, "unknown kernel id %d", which);
    }
    return CORUN_OK;
}

// Whether launch_one(k) launches anything for this engine (the QKV epilogue
// and SwiGLU may run inside the neighbouring kernels instead).
bool launches(const corun_engine *e, int k)
{
    if (e->plan.gv) return k != CORUN_K_QKV_POST && k != CORUN_K_SWIGLU && k != CORUN_K_RMSNORM;
    if (k == CORUN_K_QKV_POST) return !e->qkv_in_attn;
    if (k == CORUN_K_SWIGLU) return e->moe ? !e->egu_fused : !gu_fuses(e, e->plan.gu);
    return true;
}

// Run f (the launches of kernel class `kind`); while profiling, with a pair
// of events around it on the engine's stream.
template <class F>
corun_status timed(corun_engine *e, int kind, F &&f)
{
    if (!e->profiling) return f();
    const size_t first = e->rec.launches.size();
    set_launch_recorder(&e->rec);
    corun_status s = f();
    set_launch_recorder(nullptr);
    if (s == CORUN_OK) e->prof.push_back({kind, first, e->rec.launches.size()});
    return s;
}

corun_status enqueue_step(corun_engine *e)
{
    const corun_model_cfg &c = e->c;
    const Plan &p = e->plan;
    const int B = e->B, H = c.hidden;
    hipStream_t st = e->st;
    const int OTHER = CORUN_K_COUNT;   // embedding and feedback
    ST_TRY(timed(e, OTHER, [&]() -> corun_status {
        HIP_TRY(launch_embed(e->embed, e->d_tokens, e->d_valid, B, H, e->x, st, p.gv ? e->gss : nullptr));
        return CORUN_OK;
    }));
    const MoeBufs mb = decode_moe(e);
    const int dense_S = e->moe || p.gv ? 0 : p.down.S;
    for (int l = 0; l < c.n_layers; ++l) {
        if (!p.gv)
            ST_TRY(timed(e, CORUN_K_RMSNORM, [&]() -> corun_status {
                HIP_TRY(launch_rmsnorm(e->x, l ? e->p_down : nullptr, l ? dense_S : 0, (long long)B * H, B, H,
                                       e->attn_norm[l], c.rms_eps, e->h, st, fold_of(e, mb, l)));
                return CORUN_OK;
            }));
        for (int k : {CORUN_K_QKV_GEMM, CORUN_K_QKV_POST, CORUN_K_ATTN_SPLIT, CORUN_K_ATTN_MERGE, CORUN_K_O_GEMM,
                      CORUN_K_RMSNORM})
            if (launches(e, k)) ST_TRY(timed(e, k, [&] { return launch_one(e, k, l); }));
        if (e->moe) ST_TRY(timed(e, CORUN_K_MOE_ROUTER, [&] { return launch_one(e, CORUN_K_MOE_ROUTER, l); }));
        for (int k : {CORUN_K_GATE_UP_GEMM, CORUN_K_SWIGLU, CORUN_K_DOWN_GEMM})
            if (launches(e, k)) ST_TRY(timed(e, k, [&] { return launch_one(e, k, l); }));
    }
    ST_TRY(timed(e, CORUN_K_RMSNORM, [&]() -> corun_status {
        HIP_TRY(launch_rmsnorm(e->x, e->p_down, dense_S, (long long)B * H, B, H, e->final_norm, c.rms_eps, e->h, st,
                               fold_of(e, mb, c.n_layers)));
        return CORUN_OK;
    }));
    ST_TRY(timed(e, CORUN_K_LM_HEAD, [&] { return launch_one(e, CORUN_K_LM_HEAD, 0); }));
    ST_TRY(timed(e, CORUN_K_ARGMAX, [&] { return launch_one(e, CORUN_K_ARGMAX, 0); }));
    ST_TRY(timed(e, OTHER, [&]() -> corun_status {
        HIP_TRY(launch_feedback(e->d_tokens, e->d_seq, e->d_valid, e->d_next, B, e->d_hist, e->d_counter,
                                e->hist_cap, st));
        return CORUN_OK;
    }));
    return CORUN_OK;
}

corun_status run_step(corun_engine *e)
{
    if (e->opt.no_graph) return enqueue_step(e);
    if (!e->exec) {
        HIP_TRY(hipStreamBeginCapture(e->st, hipStreamCaptureModeThreadLocal));
        corun_status s = enqueue_step(e);
        hipGraph_t g = nullptr;
        hipError_t ce = hipStreamEndCapture(e->st, &g);
        if (s != CORUN_OK) {
            if (g) (void)hipGraphDestroy(g);
            return s;
        }
        if (ce != hipSuccess) return fail(CORUN_E_HIP, "graph capture: %s", hipGetErrorString(ce));
        e->graph = g;
        HIP_TRY(hipGraphInstantiate(&e->exec, g, nullptr, nullptr, 0));
    }
    HIP_TRY(hipGraphLaunch(e->exec, e->st));
    return CORUN_OK;
}

corun_status enter(corun_engine *e)
{
    HIP_TRY(hipEventRecord(e->ev, e->user));
    HIP_TRY(hipStreamWaitEvent(e->st, e->ev, 0));
    return CORUN_OK;
}

// Slot `slot`'s row of the page table for the host-side checks: from the
// registered host copy, else copied from the device (one synchronous copy).
corun_status page_row(corun_engine *e, int slot, std::vector<int32_t> &row)
{
    row.resize(e->kv.max_pages_per_seq);
    const size_t off = (size_t)slot * e->kv.max_pages_per_seq;
    if (e->pt_host) {
        std::memcpy(row.data(), e->pt_host + off, row.size() * sizeof(int32_t));
        return CORUN_OK;
    }
    HIP_TRY(hipMemcpy(row.data(), e->kv.page_table + off, row.size() * sizeof(int32_t), hipMemcpyDeviceToHost));
    return CORUN_OK;
}

corun_status check_pages(corun_engine *e, const int32_t *seq_lens, const uint8_t *valid, const int32_t *tokens,
                         int n_rows, int n_steps)
{
    std::vector<int32_t> pt;
    const int32_t *pth = nullptr;
    if (e->kv.layout == CORUN_KV_PAGED) {
        if (e->pt_host) {
            pth = e->pt_host;
        } else {
            pt.resize((size_t)e->kv.n_slots * e->kv.max_pages_per_seq);
            HIP_TRY(hipMemcpy(pt.data(), e->kv.page_table, pt.size() * sizeof(int32_t), hipMemcpyDeviceToHost));
            pth = pt.data();
        }
    }
    return corun_check_batch(&e->c, &e->kv, pth, n_rows, tokens, valid, seq_lens, n_steps);
}

}  // namespace

// ---------------------------------------------------------------------------
// Engine lifetime
// ---------------------------------------------------------------------------

namespace {
// The prefill projections of n rows (a prompt, a chunk, or a batch of
// prompts' tokens): their plan is a function of n and the model alone, so a
// prompt's bits never depend on the engine's workspace size.
struct PrefillPlan {
    Proj qkv, o, gu, down, router;
};

PrefillPlan prefill_plan(const corun_model_cfg &c, int n, bool bi)
{
    const int H = c.hidden, nqkv = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim, F = c.ffn;
    PrefillPlan p;
    p.qkv = choose_proj(nqkv, H, n, 0, 0, 0, bi);
    p.o = choose_proj(H, c.n_heads * c.head_dim, n, 0, 0, 0, bi);
    if (c.n_experts == 0) {
        p.gu = choose_proj(2 * F, H, n, 0, 0, 0, bi);
        p.down = choose_proj(H, F, n, 0, 0, 0, bi);
    } else {
        p.router = choose_proj(c.n_experts, H, n, 0, 0, 0, bi);
    }
    return p;
}

// Split-K partials the prefill plans of 1 .. max_rows rows can hold at once:
// the largest S x n x N over those plans.
size_t prefill_part_elems(const corun_model_cfg &c, int max_rows, bool bi)
{
    size_t most = 1;
    for (int n = 1; n <= max_rows; ++n) {
        const PrefillPlan p = prefill_plan(c, n, bi);
        for (const Proj *pr : {&p.qkv, &p.o, &p.gu, &p.down, &p.router})
            if (pr->N > 0) most = std::max(most, proj_part_elems(*pr, n));
    }
    return most;
}
}  // namespace

extern "C" int32_t corun_describe_prefill_plan(const corun_model_cfg *c, int32_t n, const corun_options *opt,
                                               int32_t *out, int32_t cap)
{
    if (!c || !out) return fail(CORUN_E_INVAL, "null argument");
    if (n < 1) return fail(CORUN_E_INVAL, "n must be >= 1");
    corun_options o{};
    if (opt) o = *opt;
    ST_TRY(check_options(o));
    const PrefillPlan p = prefill_plan(*c, n, o.batch_invariant || o.bi_prefill);
    std::vector<int32_t> v;
    for (const Proj *pr : {&p.qkv, &p.o, &p.gu, &p.down, &p.router})
        for (int x : {pr->N, pr->K, pr->S, pr->Kc, pr->bm, pr->bn}) v.push_back(x);
    const int k = std::min<int>((int)v.size(), cap);
    for (int i = 0; i < k; ++i) out[i] = v[i];
    return k;
}

static corun_status alloc_prefill(corun_engine *e)
{
    const corun_model_cfg &c = e->c;
    const int L = e->pf_max, H = c.hidden, d = c.head_dim, nq = c.n_heads, nkv = c.n_kv_heads, F = c.ffn;
    const int Lp64 = (L + 63) / 64 * 64;
    // The partial buffer holds the split-K partials of any prefill plan of
    // up to pf_max rows (corun_prefill_batch runs the batch-invariant plans).
    const bool bi_any = e->opt.batch_invariant || e->opt.bi_prefill;
    e->pf_part_elems = prefill_part_elems(c, L, e->opt.batch_invariant != 0);
    if (bi_any) e->pf_part_elems = std::max(e->pf_part_elems, prefill_part_elems(c, L, true));
    e->pf_part_elems = std::max(e->pf_part_elems, (size_t)L * H);   // the norms' residual folds read [L][H]
    Carver cv;
    cv.take(&e->pf_x, (size_t)L * H);
    cv.take(&e->pf_part, e->pf_part_elems);
    const bool bi_pf = e->opt.batch_invariant || e->opt.bi_prefill;
    const int lrows = bi_pf ? CORUN_MAX_PREFILL_BATCH : 1;   // last positions a prefill call reports
    cv.take(&e->pf_logits, (size_t)lrows * c.vocab);
    cv.take(&e->pf_h, (size_t)Lp64 * H);
    cv.take(&e->pf_q, (size_t)L * nq * d);
    cv.take(&e->pf_o, (size_t)Lp64 * nq * d);
    cv.take(&e->pf_a, (size_t)Lp64 * F);
    cv.take(&e->pf_hlast, (size_t)64 * H);
    if (e->moe) {
        const size_t na = (size_t)L * c.top_k, Fe = c.expert_ffn;
        cv.take(&e->pf_moe_w, na);
        cv.take(&e->pf_moe_gu, na * 2 * Fe);
        cv.take(&e->pf_moe_y, na * H);
        cv.take(&e->pf_moe_sel, na);
        cv.take(&e->pf_moe_list, na);
        cv.take(&e->pf_moe_tiles, (size_t)3 * (c.n_experts + (na + 15) / 16));
        cv.take(&e->pf_moe_act, na * Fe);
        if (e->opt.record_routing) {
            cv.take(&e->rt_pf_sel, (size_t)c.n_layers * na);
            cv.take(&e->rt_pf_logit, (size_t)c.n_layers * L * c.n_experts);
        }
    }
    cv.take(&e->pf_pos, (size_t)std::max(L, kv_capacity(&e->kv)));   // positions of any chunk
    cv.take(&e->pf_tok, (size_t)L);
    cv.take(&e->pf_amax, (size_t)lrows * gemm_col_blocks(c.vocab));
    cv.take(&e->pf_rowpos, bi_pf ? (size_t)L : 1);
    cv.take(&e->pf_rowslot, bi_pf ? (size_t)L : 1);
    cv.take(&e->pf_seq, (size_t)4 * CORUN_MAX_PREFILL_BATCH);
    size_t total = cv.take(&e->pf_next, CORUN_MAX_PREFILL_BATCH);
    e->pws_bytes = total;
    HIP_TRY(hipMalloc(&e->pws, total));
    HIP_TRY(hipMemsetAsync(e->pws, 0, total, e->st));
    rebase(e->pf_x, e->pws); rebase(e->pf_part, e->pws); 
    rebase(e->pf_logits, e->pws); rebase(e->pf_h, e->pws); rebase(e->pf_q, e->pws);
    rebase(e->pf_o, e->pws); rebase(e->pf_a, e->pws); rebase(e->pf_hlast, e->pws);
    if (e->moe) {
        rebase(e->pf_moe_w, e->pws); rebase(e->pf_moe_gu, e->pws); rebase(e->pf_moe_y, e->pws);
        rebase(e->pf_moe_sel, e->pws); rebase(e->pf_moe_list, e->pws); rebase(e->pf_moe_tiles, e->pws);
        rebase(e->pf_moe_act, e->pws);
        if (e->opt.record_routing) {
            rebase(e->rt_pf_sel, e->pws);
            rebase(e->rt_pf_logit, e->pws);
        }
    }
    rebase(e->pf_pos, e->pws); rebase(e->pf_tok, e->pws); rebase(e->pf_amax, e->pws); rebase(e->pf_next, e->pws);
    rebase(e->pf_rowpos, e->pws); rebase(e->pf_rowslot, e->pws); rebase(e->pf_seq, e->pws);
    HIP_TRY(launch_iota(e->pf_pos, std::max(L, kv_capacity(&e->kv)), e->st));
    return CORUN_OK;
}

// Tile-packed copies of the projections whose decode plan takes them
// (batches of up to 64 rows), made on the engine's stream after the caller's
// stream has reached this point.  Prefill projections of up to 64 rows use
// them as well.
static corun_status pack_weights(corun_engine *e)
{
    const Plan &p = e->plan;
    const int L = e->c.n_layers;
    struct Item {
        int w;
        const Proj *pr;
        int count;
    };
    const Item items[] = {{W_QKV, &p.qkv, L},
                          {W_O, &p.o, L},
                          {W_GATE_UP, &p.gu, e->moe ? 0 : L},
                          {W_DOWN, &p.down, e->moe ? 0 : L},
                          {W_ROUTER, &p.router, e->moe ? L : 0},
                          {W_LM_HEAD, &p.lm, 1}};
    // experts (any B: an expert tile holds at most 16 assignments): gate/up
    // always (K = hidden), down when expert_ffn is a multiple of 64
    const corun_model_cfg &c = e->c;
    const int E = c.n_experts, Fe = c.expert_ffn, H = c.hidden;
    const bool pk_egu = e->moe, pk_edown = e->moe && Fe % 64 == 0;
    const size_t egu_elems = pk_egu ? (size_t)E * packed_weight_elems(2 * Fe, H) : 0;
    const size_t edown_elems = pk_edown ? (size_t)E * packed_weight_elems(H, Fe) : 0;
    size_t total = (size_t)L * (egu_elems + edown_elems) * 2;   // each copy is a whole number of 16 KB tiles
    for (const Item &it : items)
        if (it.count && takes_packed(*it.pr)) total += (size_t)it.count * packed_weight_elems(it.pr->N, it.pr->K) * 2;
    // the small-batch layer's fragment-packed copies (1 KB fragments)
    const Proj *gvp[4] = {&p.qkv, &p.o, &p.gu, &p.down};
    const int gv_mode[4] = {1, 0, 2, 0};
    const int gv_w[4] = {W_QKV, W_O, W_GATE_UP, W_DOWN};
    if (p.gv)
        for (const Proj *pr : gvp) total += (size_t)L * frag_packed_elems(pr->N, pr->K) * 2;
    if (total == 0) return CORUN_OK;
    if (hipMalloc(&e->pk_buf, total) != hipSuccess)
        return fail(CORUN_E_HIP, "packed weight copies (%zu bytes) do not fit; no_weight_pack = 1 reads the row-major "
                    "weights instead", total);
    e->pk_bytes = total;
    HIP_TRY(hipEventRecord(e->ev, e->user));
    HIP_TRY(hipStreamWaitEvent(e->st, e->ev, 0));
    // gate/up without split-K: interleave gate and up rows of the same
    // features so that the projection's epilogue can apply SwiGLU
    const bool interleave = !e->moe && takes_packed(p.gu) && p.gu.S == 1 && p.gu.N % 128 == 0;
    char *q = e->pk_buf;
    for (const Item &it : items) {
        if (!it.count || !takes_packed(*it.pr)) continue;
        const size_t bytes = packed_weight_elems(it.pr->N, it.pr->K) * 2;
        for (int l = 0; l < it.count; ++l) {
            HIP_TRY(launch_pack_weights(row_major_weight(e, it.w, l), it.pr->N, it.pr->K, (uint16_t *)q, e->st,
                                        it.w == W_GATE_UP && interleave));
            e->packed[it.w].push_back((const uint16_t *)q);
            q += bytes;
        }
    }
    e->gu_fused = interleave;
    for (int i = 0; p.gv && i < 4; ++i) {
        const size_t bytes = frag_packed_elems(gvp[i]->N, gvp[i]->K) * 2;
        for (int l = 0; l < L; ++l) {
            HIP_TRY(launch_pack_frag(row_major_weight(e, gv_w[i], l), gvp[i]->N, gvp[i]->K, gv_mode[i],
                                     e->c.head_dim, (uint16_t *)q, e->st));
            e->gvw[i].push_back((const uint16_t *)q);
            q += bytes;
        }
    }
    // expert stacks, expert by expert; gate/up interleaved when its halves
    // split into 64-row tiles
    const bool e_interleave = Fe % 64 == 0;
    for (int l = 0; pk_egu && l < L; ++l) {
        for (int x = 0; x < E; ++x)
            HIP_TRY(launch_pack_weights(e->w_egu[l] + (size_t)x * 2 * Fe * H, 2 * Fe, H,
                                        (uint16_t *)q + (size_t)x * packed_weight_elems(2 * Fe, H), e->st,
                                        e_interleave));
        e->packed[W_EXP_GATE_UP].push_back((const uint16_t *)q);
        q += egu_elems * 2;
    }
    for (int l = 0; pk_edown && l < L; ++l) {
        for (int x = 0; x < E; ++x)
            HIP_TRY(launch_pack_weights(e->w_edown[l] + (size_t)x * H * Fe, H, Fe,
                                        (uint16_t *)q + (size_t)x * packed_weight_elems(H, Fe), e->st));
        e->packed[W_EXP_DOWN].push_back((const uint16_t *)q);
        q += edown_elems * 2;
    }
    e->egu_fused = pk_egu && e_interleave;
    return CORUN_OK;
}

extern "C" corun_status corun_engine_create(const corun_model_cfg *cfg, const corun_weights *w, const corun_kv *kv,
                                            int32_t B, const corun_options *opt, void *stream, corun_engine **out)
{
    if (!out) return fail(CORUN_E_INVAL, "null out");
    *out = nullptr;
    ST_TRY(corun_check_config(cfg, kv, B));
    const bool moe = cfg->n_experts > 0;
    if (!w || !w->embed || !w->final_norm || !w->lm_head || !w->attn_norm || !w->w_qkv || !w->w_o || !w->mlp_norm)
        return fail(CORUN_E_INVAL, "missing weight pointer");
    if (moe ? (!w->w_router || !w->w_exp_gate_up || !w->w_exp_down) : (!w->w_gate_up || !w->w_down))
        return fail(CORUN_E_INVAL, moe ? "missing expert weight pointer" : "missing feed-forward weight pointer");
    if (!kv->k || !kv->v) return fail(CORUN_E_INVAL, "missing KV pointers");
    if (kv->layout == CORUN_KV_PAGED && !kv->page_table) return fail(CORUN_E_INVAL, "paged cache needs page_table");
    corun_options o{};
    if (opt) o = *opt;
    ST_TRY(check_options(o));

    corun_engine *e = new corun_engine();
    e->c = *cfg;
    e->kv = *kv;
    e->opt = o;
    e->B = B;
    e->moe = moe;
    e->user = (hipStream_t)stream;
    const int L = cfg->n_layers;
    for (int l = 0; l < L; ++l) {
        e->attn_norm.push_back((const uint16_t *)w->attn_norm[l]);
        e->w_qkv.push_back((const uint16_t *)w->w_qkv[l]);
        e->w_o.push_back((const uint16_t *)w->w_o[l]);
        e->mlp_norm.push_back((const uint16_t *)w->mlp_norm[l]);
        if (moe) {
            e->w_router.push_back((const uint16_t *)w->w_router[l]);
            e->w_egu.push_back((const uint16_t *)w->w_exp_gate_up[l]);
            e->w_edown.push_back((const uint16_t *)w->w_exp_down[l]);
        } else {
            e->w_gu.push_back((const uint16_t *)w->w_gate_up[l]);
            e->w_down.push_back((const uint16_t *)w->w_down[l]);
        }
        e->kc.push_back((uint16_t *)kv->k[l]);
        e->vc.push_back((uint16_t *)kv->v[l]);
    }
    e->embed = (const uint16_t *)w->embed;
    e->final_norm = (const uint16_t *)w->final_norm;
    e->lm_head = (const uint16_t *)w->lm_head;
    e->view.layout = kv->layout;
    e->view.max_seq_len = kv->max_seq_len;
    e->view.page_size = kv->page_size;
    e->view.max_pages_per_seq = kv->max_pages_per_seq;
    e->view.page_table = kv->page_table;
    e->plan = make_plan(cfg, kv, B, o);
    const Plan &p = e->plan;
    if (o.small_batch_layer == 1 && !p.gv) {
        delete e;
        return fail(CORUN_E_INVAL, "small_batch_layer = 1 needs a dense model, B_fixed <= 8, weight packing and no "
                    "plan overrides");
    }
    // Inside attention every block rebuilds its group's q from the split
    // partials: one launch fewer, which pays where launches dominate (B = 1:
    // about 3%) and costs where many blocks repeat the work (B = 256: the
    // attention kernel 187 -> 206 us against 7 us for the epilogue kernel).
    e->qkv_in_attn = !p.gv && (o.qkv_epilogue == 2 || (o.qkv_epilogue == 0 && B <= 8));

    auto bail = [&](corun_status s) {
        corun_engine_destroy(e);
        return s;
    };
    if (hipStreamCreateWithFlags(&e->st, hipStreamNonBlocking) != hipSuccess ||
        hipEventCreateWithFlags(&e->ev, hipEventDisableTiming) != hipSuccess)
        return bail(fail(CORUN_E_HIP, "stream/event creation failed"));

    const int H = cfg->hidden, d = cfg->head_dim, nq = cfg->n_heads, nkv = cfg->n_kv_heads, F = cfg->ffn;
    const int cap = kv_capacity(kv);
    const int rope_len = std::max(cap, o.max_prefill_len);
    e->hist_cap = 4096;
    Carver cv;
    cv.take(&e->d_tokens, B);
    cv.take(&e->d_seq, B);
    cv.take(&e->d_next, B);
    cv.take(&e->d_counter, 4);
    cv.take(&e->d_hist, (size_t)e->hist_cap * B);
    cv.take(&e->d_valid, B);
    cv.take(&e->d_order, B);
    cv.take(&e->x, (size_t)B * H);
    cv.take(&e->gss, p.gv ? (size_t)B * (H / 16) : 1);
    cv.take(&e->p_qkv, proj_part_elems(p.qkv, B));
    cv.take(&e->p_o, proj_part_elems(p.o, B));
    cv.take(&e->p_gu, proj_part_elems(p.gu, B));
    cv.take(&e->p_down, proj_part_elems(p.down, B));
    cv.take(&e->attn_ws, (size_t)B * nkv * p.max_splits * (nq / nkv) * (d + 2));
    cv.take(&e->logits, (size_t)B * cfg->vocab);
    cv.take(&e->p_lm, p.lm.S > 1 ? proj_part_elems(p.lm, B) : 1);
    cv.take(&e->amax, (size_t)B * gemm_col_blocks(cfg->vocab));
    if (moe) {
        const size_t na = (size_t)B * cfg->top_k, Fe = cfg->expert_ffn;
        cv.take(&e->p_router, proj_part_elems(p.router, B));
        cv.take(&e->moe_w, na);
        cv.take(&e->moe_gu, na * 2 * Fe);
        cv.take(&e->moe_y, na * H);
        cv.take(&e->moe_sel, na);
        cv.take(&e->moe_list, na);
        cv.take(&e->moe_tiles, (size_t)3 * p.moe_slots);
        cv.take(&e->moe_act, na * Fe);
        if (o.record_routing) {
            cv.take(&e->rt_sel, (size_t)L * na);
            cv.take(&e->rt_logit, (size_t)L * B * cfg->n_experts);
        }
    }
    cv.take(&e->d_svalid, (size_t)B);
    cv.take(&e->d_spos, (size_t)B);
    cv.take(&e->d_stok, (size_t)B);
    cv.take(&e->d_sseed, (size_t)B);
    cv.take(&e->d_stemp, (size_t)B);
    cv.take(&e->d_slp, (size_t)B);
    cv.take(&e->h, (size_t)p.Mp * H);
    cv.take(&e->q, (size_t)B * nq * d);
    cv.take(&e->o, (size_t)p.Mp * nq * d);
    cv.take(&e->a, (size_t)p.Mp * F);
    size_t total = cv.take(&e->rope, (size_t)rope_len * (d / 2));
    e->ws_bytes = total;
    if (hipMalloc(&e->ws, total) != hipSuccess) return bail(fail(CORUN_E_HIP, "workspace allocation of %zu bytes", total));
    rebase(e->d_tokens, e->ws); rebase(e->d_seq, e->ws); rebase(e->d_next, e->ws); rebase(e->d_counter, e->ws);
    rebase(e->d_hist, e->ws); rebase(e->d_valid, e->ws); rebase(e->d_order, e->ws); rebase(e->x, e->ws);
    rebase(e->gss, e->ws);
    rebase(e->p_qkv, e->ws);
    rebase(e->p_o, e->ws); rebase(e->p_gu, e->ws); rebase(e->p_down, e->ws); rebase(e->attn_ws, e->ws);
    rebase(e->logits, e->ws); rebase(e->p_lm, e->ws); rebase(e->amax, e->ws); rebase(e->h, e->ws); rebase(e->q, e->ws); rebase(e->o, e->ws); rebase(e->a, e->ws);
    rebase(e->rope, e->ws);
    rebase(e->d_svalid, e->ws); rebase(e->d_spos, e->ws); rebase(e->d_stok, e->ws); rebase(e->d_sseed, e->ws);
    rebase(e->d_stemp, e->ws); rebase(e->d_slp, e->ws);
    if (moe) {
        rebase(e->p_router, e->ws); rebase(e->moe_w, e->ws); rebase(e->moe_gu, e->ws); rebase(e->moe_y, e->ws);
        rebase(e->moe_sel, e->ws); rebase(e->moe_list, e->ws); rebase(e->moe_tiles, e->ws); rebase(e->moe_act, e->ws);
        if (o.record_routing) {
            rebase(e->rt_sel, e->ws);
            rebase(e->rt_logit, e->ws);
        }
    }
    // Rows B..Mp-1 of the MFMA A operands (h, o, a) are read but never
    // stored; start everything at zero, or at NaN when poisoning.
    const uint32_t fillv = o.poison_workspace ? 0xFFFFFFFFu : 0u;
    const size_t rope_off = (size_t)((char *)e->rope - e->ws);
    if (launch_fill_u32((uint32_t *)e->ws, (long long)(rope_off / 4), fillv, e->st) != hipSuccess ||
        launch_fill_u32((uint32_t *)e->d_counter, 1, (uint32_t)e->hist_cap, e->st) != hipSuccess ||
        launch_rope_table(e->rope, rope_len, d, (double)cfg->rope_theta, e->st) != hipSuccess ||
        launch_iota(e->d_order, B, e->st) != hipSuccess)   // a valid row order before the first upload
        return bail(fail(CORUN_E_HIP, "workspace initialisation failed"));

    if (hipHostMalloc((void **)&e->h_tok, sizeof(int32_t) * B * 5 + 64, 0) != hipSuccess ||
        hipHostMalloc((void **)&e->h_valid, B + 64, 0) != hipSuccess ||
        hipHostMalloc((void **)&e->h_hist, sizeof(int32_t) * (size_t)e->hist_cap * B, 0) != hipSuccess ||
        hipHostMalloc((void **)&e->h_samp, (size_t)B * 32 + 256, 0) != hipSuccess)
        return bail(fail(CORUN_E_HIP, "pinned staging allocation failed"));
    e->h_seq = e->h_tok + B;
    e->h_next = e->h_tok + 2 * B;
    e->h_counter = e->h_tok + 3 * B;
    e->h_order = e->h_tok + 4 * B;

    if (o.max_prefill_len > 0) {
        e->pf_max = o.max_prefill_len;
        corun_status s = alloc_prefill(e);
        if (s != CORUN_OK) return bail(s);
    }
    if (!o.no_weight_pack) {
        corun_status s = pack_weights(e);
        if (s != CORUN_OK) return bail(s);
    }
    if (hipStreamSynchronize(e->st) != hipSuccess) return bail(fail(CORUN_E_HIP, "initialisation failed"));
    *out = e;
    return CORUN_OK;
}

extern "C" void corun_engine_destroy(corun_engine *e)
{
    if (!e) return;
    if (e->st) (void)hipStreamSynchronize(e->st);
    if (e->exec) (void)hipGraphExecDestroy(e->exec);
    if (e->graph) (void)hipGraphDestroy(e->graph);
    if (e->ws) (void)hipFree(e->ws);
    if (e->pws) (void)hipFree(e->pws);
    if (e->pk_buf) (void)hipFree(e->pk_buf);
    if (e->h_tok) (void)hipHostFree(e->h_tok);
    if (e->h_valid) (void)hipHostFree(e->h_valid);
    if (e->h_hist) (void)hipHostFree(e->h_hist);
    if (e->h_samp) (void)hipHostFree(e->h_samp);
    for (hipEvent_t ev : e->rec.pool) (void)hipEventDestroy(ev);
    if (e->ev) (void)hipEventDestroy(e->ev);
    if (e->st) (void)hipStreamDestroy(e->st);
    delete e;
}

// ---------------------------------------------------------------------------
// Decode
// ---------------------------------------------------------------------------

static corun_status upload_inputs(corun_engine *e, const int32_t *tokens, const uint8_t *valid,
                                  const int32_t *seq_lens, int32_t counter)
{
    const int B = e->B;
    std::memcpy(e->h_tok, tokens, sizeof(int32_t) * B);
    std::memcpy(e->h_seq, seq_lens, sizeof(int32_t) * B);
    std::memcpy(e->h_valid, valid, B);
    *e->h_counter = counter;
    // attention dispatches live rows longest first, padding rows last; the
    // order moves only work between workgroups, never a row's arithmetic
    for (int r = 0; r < B; ++r) e->h_order[r] = r;
    std::stable_sort(e->h_order, e->h_order + B, [&](int32_t a, int32_t b) {
        const bool va = valid[a] != 0, vb = valid[b] != 0;
        if (va != vb) return va;
        return va && seq_lens[a] > seq_lens[b];
    });
    HIP_TRY(hipMemcpyAsync(e->d_order, e->h_order, sizeof(int32_t) * B, hipMemcpyHostToDevice, e->st));
    HIP_TRY(hipMemcpyAsync(e->d_tokens, e->h_tok, sizeof(int32_t) * B, hipMemcpyHostToDevice, e->st));
    HIP_TRY(hipMemcpyAsync(e->d_seq, e->h_seq, sizeof(int32_t) * B, hipMemcpyHostToDevice, e->st));
    HIP_TRY(hipMemcpyAsync(e->d_valid, e->h_valid, B, hipMemcpyHostToDevice, e->st));
    HIP_TRY(hipMemcpyAsync(e->d_counter, e->h_counter, sizeof(int32_t), hipMemcpyHostToDevice, e->st));
    e->decoded = true;
    return CORUN_OK;
}

// The last validated step inputs (still in the pinned staging) back to the
// device: the step's feedback advanced every live row's position, possibly to
// the capacity, and a kernel launched on that state would write past it.
static corun_status restore_inputs(corun_engine *e)
{
    const int B = e->B;
    HIP_TRY(hipMemcpyAsync(e->d_order, e->h_order, sizeof(int32_t) * B, hipMemcpyHostToDevice, e->st));
    HIP_TRY(hipMemcpyAsync(e->d_tokens, e->h_tok, sizeof(int32_t) * B, hipMemcpyHostToDevice, e->st));
    HIP_TRY(hipMemcpyAsync(e->d_seq, e->h_seq, sizeof(int32_t) * B, hipMemcpyHostToDevice, e->st));
    HIP_TRY(hipMemcpyAsync(e->d_valid, e->h_valid, B, hipMemcpyHostToDevice, e->st));
    return CORUN_OK;
}

extern "C" corun_status corun_decode_step(corun_engine *e, const int32_t *tokens, const uint8_t *valid,
                                          const int32_t *seq_lens, int32_t *next_tokens, float *logits)
{
    if (!e || !next_tokens) return fail(CORUN_E_INVAL, "null argument");
    ST_TRY(check_pages(e, seq_lens, valid, tokens, e->B, 1));
    ST_TRY(enter(e));
    ST_TRY(upload_inputs(e, tokens, valid, seq_lens, e->hist_cap));
    ST_TRY(run_step(e));
    const int B = e->B;
    HIP_TRY(hipMemcpyAsync(e->h_next, e->d_next, sizeof(int32_t) * B, hipMemcpyDeviceToHost, e->st));
    if (logits)
        HIP_TRY(hipMemcpyAsync(logits, e->logits, sizeof(float) * (size_t)B * e->c.vocab, hipMemcpyDeviceToDevice,
                               e->st));
    HIP_TRY(hipStreamSynchronize(e->st));
    std::memcpy(next_tokens, e->h_next, sizeof(int32_t) * B);
    return CORUN_OK;
}

extern "C" corun_status corun_decode_run(corun_engine *e, int32_t n_steps, const int32_t *tokens,
                                         const uint8_t *valid, const int32_t *seq_lens, int32_t *tokens_out)
{
    if (!e || !tokens_out) return fail(CORUN_E_INVAL, "null argument");
    if (n_steps < 1) return fail(CORUN_E_INVAL, "n_steps must be >= 1");
    ST_TRY(check_pages(e, seq_lens, valid, tokens, e->B, n_steps));
    ST_TRY(enter(e));
    const int B = e->B;
    int done = 0;
    bool first = true;
    while (done < n_steps) {
        const int n = std::min(n_steps - done, e->hist_cap);
        if (first) {
            ST_TRY(upload_inputs(e, tokens, valid, seq_lens, 0));
            first = false;
        } else {
            *e->h_counter = 0;
            HIP_TRY(hipMemcpyAsync(e->d_counter, e->h_counter, sizeof(int32_t), hipMemcpyHostToDevice, e->st));
        }
        for (int i = 0; i < n; ++i) ST_TRY(run_step(e));
        HIP_TRY(hipMemcpyAsync(e->h_hist, e->d_hist, sizeof(int32_t) * (size_t)n * B, hipMemcpyDeviceToHost, e->st));
        HIP_TRY(hipStreamSynchronize(e->st));
        std::memcpy(tokens_out + (size_t)done * B, e->h_hist, sizeof(int32_t) * (size_t)n * B);
        done += n;
    }
    // the staging now holds the inputs of the run's last step (what its
    // feedback fed it), for corun_time_kernel
    for (int b = 0; b < B && n_steps > 1; ++b) {
        if (!e->h_valid[b]) continue;
        e->h_seq[b] += n_steps - 1;
        e->h_tok[b] = tokens_out[(size_t)(n_steps - 2) * B + b];
    }
    return CORUN_OK;
}

// ---------------------------------------------------------------------------
// Isolated prefill: every launch is sized by the chunk's length and start
// alone (the whole prompt is one chunk at start 0).
// ---------------------------------------------------------------------------

extern "C" corun_status corun_prefill_chunk(corun_engine *e, const int32_t *tokens, int32_t n, int32_t start,
                                            int32_t slot, int32_t *token_out, float *last_logits)
{
    if (!e || !tokens) return fail(CORUN_E_INVAL, "null argument");
    if (e->pf_max <= 0) return fail(CORUN_E_STATE, "engine was created without a prefill workspace");
    if (n < 1) return fail(CORUN_E_INVAL, "chunk length must be >= 1");
    if (start < 0) return fail(CORUN_E_INVAL, "negative chunk start");
    if (n > e->pf_max) return fail(CORUN_E_CAPACITY, "chunk length %d exceeds the prefill workspace %d", n, e->pf_max);
    if (slot < 0 || slot >= e->kv.n_slots) return fail(CORUN_E_INVAL, "slot %d outside [0, %d)", slot, e->kv.n_slots);
    const int cap = kv_capacity(&e->kv);
    if ((int64_t)start + n > cap)
        return fail(CORUN_E_CAPACITY, "positions %d..%d exceed the cache capacity %d", start, start + n - 1, cap);
    for (int t = 0; t < n; ++t)
        if (tokens[t] < 0 || tokens[t] >= e->c.vocab)
            return fail(CORUN_E_INVAL, "token[%d] = %d outside [0, %d)", t, tokens[t], e->c.vocab);
    if (e->kv.layout == CORUN_KV_PAGED) {
        std::vector<int32_t> pt;
        ST_TRY(page_row(e, slot, pt));
        for (int j = 0; j <= (start + n - 1) / e->kv.page_size; ++j)
            if (pt[j] < 0 || pt[j] >= e->kv.num_pages)
                return fail(CORUN_E_CAPACITY, "slot %d: page %d maps to %d outside [0, %d)", slot, j, pt[j],
                            e->kv.num_pages);
    }
    ST_TRY(enter(e));
    const corun_model_cfg &c = e->c;
    const int H = c.hidden, d = c.head_dim, nq = c.n_heads, nkv = c.n_kv_heads, F = c.ffn;
    const int nqkv = (nq + 2 * nkv) * d;
    hipStream_t st = e->st;
    const int Lp = n;     // rows of every projection: the chunk's tokens
    const bool bi = e->opt.batch_invariant != 0 || e->opt.bi_prefill != 0;
    const PrefillPlan pp = prefill_plan(c, Lp, bi);   // a function of n alone
    const Proj &pq = pp.qkv, &po = pp.o, &pg = pp.gu, &pd = pp.down, &pr = pp.router;
    const Proj pl = choose_proj(c.vocab, H, 1, 1, 0, 0, bi);
    const int dense_S = e->moe ? 0 : pd.S;
    const MoeBufs pmb{nullptr,         e->pf_part,       e->pf_moe_w,   e->pf_moe_gu,
                      e->pf_moe_y,     e->pf_moe_sel,    e->pf_moe_list, e->pf_moe_tiles,
                      e->pf_moe_act,   e->moe ? c.n_experts + (Lp * c.top_k + 15) / 16 : 0,
                      e->rt_pf_sel,    e->rt_pf_logit};
    e->pf_trace_rows = Lp;

    HIP_TRY(hipMemcpyAsync(e->pf_tok, tokens, sizeof(int32_t) * Lp, hipMemcpyHostToDevice, st));
    HIP_TRY(launch_embed(e->embed, e->pf_tok, nullptr, Lp, H, e->pf_x, st));
    for (int l = 0; l < c.n_layers; ++l) {
        HIP_TRY(launch_rmsnorm(e->pf_x, l ? e->pf_part : nullptr, l ? dense_S : 0, (long long)Lp * H, Lp, H,
                               e->attn_norm[l], c.rms_eps, e->pf_h, st, fold_of(e, pmb, l)));
        HIP_TRY(proj(e, e->pf_h, H, W_QKV, l, pq, Lp, e->pf_part, (long long)Lp * nqkv, nqkv));
        HIP_TRY(launch_qkv_post(e->pf_part, pq.S, (long long)Lp * nqkv, Lp, nullptr, e->pf_pos + start, nullptr, slot,
                                nq, nkv, d, e->rope, e->pf_q, e->kc[l], e->vc[l], e->view, st));
        HIP_TRY(launch_prefill_attn(e->pf_q, Lp, start, nq, nkv, d, slot, e->kc[l], e->vc[l], e->view, e->pf_o, st));
        HIP_TRY(proj(e, e->pf_o, nq * d, W_O, l, po, Lp, e->pf_part, (long long)Lp * H, H));
        HIP_TRY(launch_rmsnorm(e->pf_x, e->pf_part, po.S, (long long)Lp * H, Lp, H, e->mlp_norm[l], c.rms_eps,
                               e->pf_h, st));
        if (e->moe) {
            const int Fe = c.expert_ffn;
            ST_TRY(moe_router(e, pmb, e->pf_h, Lp, pr, l));
            ST_TRY(moe_expert_gate_up(e, pmb, e->pf_h, l));
            if (!e->egu_fused) HIP_TRY(launch_swiglu(e->pf_moe_gu, 1, 0, Lp * c.top_k, Fe, e->pf_moe_act, Fe, st));
            ST_TRY(moe_expert_down(e, pmb, l));
        } else {
            if (gu_fuses(e, pg)) {
                HIP_TRY(gate_up_swiglu(e, e->pf_h, l, pg, Lp, e->pf_a));
            } else {
                HIP_TRY(proj(e, e->pf_h, H, W_GATE_UP, l, pg, Lp, e->pf_part, (long long)Lp * 2 * F, 2 * F));
                HIP_TRY(launch_swiglu(e->pf_part, pg.S, (long long)Lp * 2 * F, Lp, F, e->pf_a, F, st));
            }
            HIP_TRY(proj(e, e->pf_a, F, W_DOWN, l, pd, Lp, e->pf_part, (long long)Lp * H, H));
        }
    }
    if (!token_out && !last_logits) {   // an inner chunk: its KV is the product
        HIP_TRY(hipStreamSynchronize(st));
        return CORUN_OK;
    }
    // last position only: fold its down partials, final norm, lm_head, argmax
    const size_t last = (size_t)(Lp - 1) * H;
    MoeFold lf = fold_of(e, pmb, c.n_layers);
    if (lf.y) {   // the last position's assignments are rows (Lp-1) top_k ..
        lf.y += (size_t)(Lp - 1) * c.top_k * H;
        lf.w += (size_t)(Lp - 1) * c.top_k;
    }
    HIP_TRY(launch_rmsnorm(e->pf_x + last, e->pf_part + last, dense_S, (long long)Lp * H, 1, H, e->final_norm,
                           c.rms_eps, e->pf_hlast, st, lf));
    HIP_TRY(proj(e, e->pf_hlast, H, W_LM_HEAD, 0, pl, 1, e->pf_logits, 0, c.vocab, e->pf_amax));
    HIP_TRY(launch_argmax_partials(e->pf_amax, 1, gemm_col_blocks(c.vocab), nullptr, e->pf_next, st));
    HIP_TRY(hipMemcpyAsync(e->h_next, e->pf_next, sizeof(int32_t), hipMemcpyDeviceToHost, st));
    if (last_logits)
        HIP_TRY(hipMemcpyAsync(last_logits, e->pf_logits, sizeof(float) * c.vocab, hipMemcpyDeviceToDevice, st));
    HIP_TRY(hipStreamSynchronize(st));
    if (token_out) *token_out = e->h_next[0];
    return CORUN_OK;
}

extern "C" corun_status corun_prefill(corun_engine *e, const int32_t *prompt, int32_t Lp, int32_t slot,
                                      int32_t *token_out, float *last_logits)
{
    if (!token_out) return fail(CORUN_E_INVAL, "null argument");
    if (e && e->pf_max > 0 && Lp > e->pf_max)
        return fail(CORUN_E_CAPACITY, "prompt_len %d exceeds the prefill workspace %d", Lp, e->pf_max);
    if (e && Lp > kv_capacity(&e->kv)) return fail(CORUN_E_CAPACITY, "prompt_len %d exceeds the cache capacity", Lp);
    return corun_prefill_chunk(e, prompt, Lp, 0, slot, token_out, last_logits);
}

extern "C" corun_status corun_prefill_batch(corun_engine *e, const int32_t *tokens, const int32_t *lens,
                                            const int32_t *slots, int32_t n, int32_t *tokens_out, float *last_logits)
{
    if (!e || !tokens || !lens || !slots || !tokens_out) return fail(CORUN_E_INVAL, "null argument");
    if (!(e->opt.batch_invariant || e->opt.bi_prefill))
        return fail(CORUN_E_STATE, "batched prefill needs an engine created with bi_prefill or batch_invariant");
    if (e->pf_max <= 0) return fail(CORUN_E_STATE, "engine was created without a prefill workspace");
    if (n < 1 || n > CORUN_MAX_PREFILL_BATCH)
        return fail(CORUN_E_INVAL, "n = %d outside [1, %d]", n, CORUN_MAX_PREFILL_BATCH);
    const int cap = kv_capacity(&e->kv);
    long long M = 0;
    for (int i = 0; i < n; ++i) {
        if (lens[i] < 1) return fail(CORUN_E_INVAL, "lens[%d] = %d", i, lens[i]);
        if (lens[i] > cap) return fail(CORUN_E_CAPACITY, "prompt %d (%d tokens) exceeds the cache capacity", i, lens[i]);
        if (slots[i] < 0 || slots[i] >= e->kv.n_slots)
            return fail(CORUN_E_INVAL, "slots[%d] = %d outside [0, %d)", i, slots[i], e->kv.n_slots);
        for (int j = 0; j < i; ++j)
            if (slots[j] == slots[i]) return fail(CORUN_E_INVAL, "slot %d given twice", slots[i]);
        M += lens[i];
    }
    if (M > e->pf_max) return fail(CORUN_E_CAPACITY, "%lld prompt tokens exceed the prefill workspace %d", M, e->pf_max);
    for (long long t = 0; t < M; ++t)
        if (tokens[t] < 0 || tokens[t] >= e->c.vocab)
            return fail(CORUN_E_INVAL, "tokens[%lld] = %d outside [0, %d)", t, tokens[t], e->c.vocab);
    if (e->kv.layout == CORUN_KV_PAGED) {
        std::vector<int32_t> pt;
        for (int i = 0; i < n; ++i) {
            ST_TRY(page_row(e, slots[i], pt));
            for (int j = 0; j <= (lens[i] - 1) / e->kv.page_size; ++j)
                if (pt[j] < 0 || pt[j] >= e->kv.num_pages)
                    return fail(CORUN_E_CAPACITY, "slot %d: page %d maps to %d outside [0, %d)", slots[i], j, pt[j],
                                e->kv.num_pages);
        }
    }
    ST_TRY(enter(e));
    const corun_model_cfg &c = e->c;
    const int H = c.hidden, d = c.head_dim, nq = c.n_heads, nkv = c.n_kv_heads, F = c.ffn;
    const int nqkv = (nq + 2 * nkv) * d;
    const int G = nq / nkv;
    const int Lp = (int)M;   // rows of every projection: all prompts' tokens
    hipStream_t st = e->st;
    // every row's position within its prompt and its cache slot; per prompt
    // (first row, length, slot, first attention unit group)
    std::vector<int32_t> rowpos(Lp), rowslot(Lp), seq(4 * n);
    int groups = 0;
    for (int i = 0, r0 = 0; i < n; r0 += lens[i], ++i) {
        for (int t = 0; t < lens[i]; ++t) {
            rowpos[r0 + t] = t;
            rowslot[r0 + t] = slots[i];
        }
        seq[4 * i] = r0;
        seq[4 * i + 1] = lens[i];
        seq[4 * i + 2] = slots[i];
        seq[4 * i + 3] = groups;
        groups += (((lens[i] + 31) / 32) * G + 7) / 8;
    }
    const PrefillPlan pp = prefill_plan(c, Lp, true);   // batch-invariant: no split-K for any Lp
    const Proj &pq = pp.qkv, &po = pp.o, &pg = pp.gu, &pd = pp.down, &pr = pp.router;
    const Proj pl = choose_proj(c.vocab, H, n, 1, 0, 0, true);
    const int dense_S = e->moe ? 0 : pd.S;
    const MoeBufs pmb{nullptr,         e->pf_part,       e->pf_moe_w,   e->pf_moe_gu,
                      e->pf_moe_y,     e->pf_moe_sel,    e->pf_moe_list, e->pf_moe_tiles,
                      e->pf_moe_act,   e->moe ? c.n_experts + (Lp * c.top_k + 15) / 16 : 0,
                      e->rt_pf_sel,    e->rt_pf_logit};
    e->pf_trace_rows = Lp;

    HIP_TRY(hipMemcpyAsync(e->pf_tok, tokens, sizeof(int32_t) * Lp, hipMemcpyHostToDevice, st));
    HIP_TRY(hipMemcpyAsync(e->pf_rowpos, rowpos.data(), sizeof(int32_t) * Lp, hipMemcpyHostToDevice, st));
    HIP_TRY(hipMemcpyAsync(e->pf_rowslot, rowslot.data(), sizeof(int32_t) * Lp, hipMemcpyHostToDevice, st));
    HIP_TRY(hipMemcpyAsync(e->pf_seq, seq.data(), sizeof(int32_t) * 4 * n, hipMemcpyHostToDevice, st));
    HIP_TRY(launch_embed(e->embed, e->pf_tok, nullptr, Lp, H, e->pf_x, st));
    for (int l = 0; l < c.n_layers; ++l) {
        HIP_TRY(launch_rmsnorm(e->pf_x, l ? e->pf_part : nullptr, l ? dense_S : 0, (long long)Lp * H, Lp, H,
                               e->attn_norm[l], c.rms_eps, e->pf_h, st, fold_of(e, pmb, l)));
        HIP_TRY(proj(e, e->pf_h, H, W_QKV, l, pq, Lp, e->pf_part, (long long)Lp * nqkv, nqkv));
        HIP_TRY(launch_qkv_post(e->pf_part, pq.S, (long long)Lp * nqkv, Lp, nullptr, e->pf_rowpos, e->pf_rowslot, -1,
                                nq, nkv, d, e->rope, e->pf_q, e->kc[l], e->vc[l], e->view, st));
        HIP_TRY(launch_prefill_attn_multi(e->pf_q, e->pf_seq, n, groups, nq, nkv, d, e->kc[l], e->vc[l], e->view,
                                          e->pf_o, st));
        HIP_TRY(proj(e, e->pf_o, nq * d, W_O, l, po, Lp, e->pf_part, (long long)Lp * H, H));
        HIP_TRY(launch_rmsnorm(e->pf_x, e->pf_part, po.S, (long long)Lp * H, Lp, H, e->mlp_norm[l], c.rms_eps,
                               e->pf_h, st));
        if (e->moe) {
            const int Fe = c.expert_ffn;
            ST_TRY(moe_router(e, pmb, e->pf_h, Lp, pr, l));
            ST_TRY(moe_expert_gate_up(e, pmb, e->pf_h, l));
            if (!e->egu_fused) HIP_TRY(launch_swiglu(e->pf_moe_gu, 1, 0, Lp * c.top_k, Fe, e->pf_moe_act, Fe, st));
            ST_TRY(moe_expert_down(e, pmb, l));
        } else {
            if (gu_fuses(e, pg)) {
                HIP_TRY(gate_up_swiglu(e, e->pf_h, l, pg, Lp, e->pf_a));
            } else {
                HIP_TRY(proj(e, e->pf_h, H, W_GATE_UP, l, pg, Lp, e->pf_part, (long long)Lp * 2 * F, 2 * F));
                HIP_TRY(launch_swiglu(e->pf_part, pg.S, (long long)Lp * 2 * F, Lp, F, e->pf_a, F, st));
            }
            HIP_TRY(proj(e, e->pf_a, F, W_DOWN, l, pd, Lp, e->pf_part, (long long)Lp * H, H));
        }
    }
    // final norm of every row (the same row-wise arithmetic as one prompt's
    // last row), then the prompts' last rows through lm_head and argmax
    HIP_TRY(launch_rmsnorm(e->pf_x, e->pf_part, dense_S, (long long)Lp * H, Lp, H, e->final_norm, c.rms_eps, e->pf_h,
                           st, fold_of(e, pmb, c.n_layers)));
    HIP_TRY(launch_gather_last_rows(e->pf_h, e->pf_seq, n, H, e->pf_hlast, st));
    HIP_TRY(proj(e, e->pf_hlast, H, W_LM_HEAD, 0, pl, n, e->pf_logits, 0, c.vocab, e->pf_amax));
    HIP_TRY(launch_argmax_partials(e->pf_amax, n, gemm_col_blocks(c.vocab), nullptr, e->pf_next, st));
    HIP_TRY(hipMemcpyAsync(tokens_out, e->pf_next, sizeof(int32_t) * n, hipMemcpyDeviceToHost, st));
    if (last_logits)
        HIP_TRY(hipMemcpyAsync(last_logits, e->pf_logits, sizeof(float) * (size_t)n * c.vocab,
                               hipMemcpyDeviceToDevice, st));
    HIP_TRY(hipStreamSynchronize(st));
    return CORUN_OK;
}

extern "C" corun_status corun_engine_set_page_table_host(corun_engine *e, const int32_t *pt_host)
{
    if (!e) return fail(CORUN_E_INVAL, "null engine");
    if (pt_host && e->kv.layout != CORUN_KV_PAGED) return fail(CORUN_E_STATE, "the engine's cache is not paged");
    e->pt_host = pt_host;
    return CORUN_OK;
}

extern "C" corun_status corun_engine_info(const corun_engine *e, int32_t *B_fixed, corun_model_cfg *cfg, corun_kv *kv)
{
    if (!e) return fail(CORUN_E_INVAL, "null engine");
    if (B_fixed) *B_fixed = e->B;
    if (cfg) *cfg = e->c;
    if (kv) *kv = e->kv;
    return CORUN_OK;
}

extern "C" corun_status corun_routing_trace(corun_engine *e, int32_t source, int32_t *sel, float *logits,
                                            int32_t *rows_out)
{
    if (!e || !rows_out) return fail(CORUN_E_INVAL, "null argument");
    if (!e->moe || !e->opt.record_routing)
        return fail(CORUN_E_STATE, "no routing record: a mixture-of-experts engine created with record_routing");
    if (source != 0 && source != 1) return fail(CORUN_E_INVAL, "source must be 0 (decode) or 1 (prefill)");
    if (source == 1 && e->pf_max <= 0) return fail(CORUN_E_STATE, "engine was created without a prefill workspace");
    const int rows = source == 0 ? e->B : e->pf_trace_rows;
    *rows_out = rows;
    const size_t L = (size_t)e->c.n_layers;
    HIP_TRY(hipStreamSynchronize(e->st));
    if (sel && rows > 0)
        HIP_TRY(hipMemcpy(sel, source == 0 ? e->rt_sel : e->rt_pf_sel, sizeof(int32_t) * L * rows * e->c.top_k,
                          hipMemcpyDeviceToHost));
    if (logits && rows > 0)
        HIP_TRY(hipMemcpy(logits, source == 0 ? e->rt_logit : e->rt_pf_logit,
                          sizeof(float) * L * rows * e->c.n_experts, hipMemcpyDeviceToHost));
    return CORUN_OK;
}

// ---------------------------------------------------------------------------
// Seeded sampling
// ---------------------------------------------------------------------------

extern "C" corun_status corun_sample(corun_engine *e, const float *logits_dev, int64_t ld, int32_t rows,
                                     const uint8_t *valid, const int32_t *positions, const uint64_t *seeds,
                                     const float *temperature, int32_t *tokens_out, float *logprobs_out)
{
    if (!e || !logits_dev || !valid || !positions || !seeds || !temperature || !tokens_out)
        return fail(CORUN_E_INVAL, "null argument");
    if (rows < 1 || rows > e->B) return fail(CORUN_E_SHAPE, "rows %d outside [1, B = %d]", rows, e->B);
    if (ld < e->c.vocab) return fail(CORUN_E_SHAPE, "row stride %lld below the vocabulary %d", (long long)ld, e->c.vocab);
    for (int r = 0; r < rows; ++r) {
        if (!valid[r]) continue;
        if (positions[r] < 0) return fail(CORUN_E_INVAL, "row %d: negative position %d", r, positions[r]);
        if (std::isnan(temperature[r]) || std::isinf(temperature[r]))
            return fail(CORUN_E_INVAL, "row %d: temperature is not finite", r);
    }
    ST_TRY(enter(e));
    // pinned staging: seeds [B] u64, positions [B], temperatures [B], tokens [B], logprobs [B], valid [B]
    char *hs = e->h_samp;
    uint64_t *hseed = reinterpret_cast<uint64_t *>(hs);
    int32_t *hpos = reinterpret_cast<int32_t *>(hs + 8 * (size_t)e->B);
    float *htemp = reinterpret_cast<float *>(hs + 12 * (size_t)e->B);
    int32_t *htok = reinterpret_cast<int32_t *>(hs + 16 * (size_t)e->B);
    float *hlp = reinterpret_cast<float *>(hs + 20 * (size_t)e->B);
    uint8_t *hval = reinterpret_cast<uint8_t *>(hs + 24 * (size_t)e->B);
    std::memcpy(hseed, seeds, sizeof(uint64_t) * rows);
    std::memcpy(hpos, positions, sizeof(int32_t) * rows);
    std::memcpy(htemp, temperature, sizeof(float) * rows);
    std::memcpy(hval, valid, rows);
    hipStream_t st = e->st;
    HIP_TRY(hipMemcpyAsync(e->d_sseed, hseed, sizeof(uint64_t) * rows, hipMemcpyHostToDevice, st));
    HIP_TRY(hipMemcpyAsync(e->d_spos, hpos, sizeof(int32_t) * rows, hipMemcpyHostToDevice, st));
    HIP_TRY(hipMemcpyAsync(e->d_stemp, htemp, sizeof(float) * rows, hipMemcpyHostToDevice, st));
    HIP_TRY(hipMemcpyAsync(e->d_svalid, hval, rows, hipMemcpyHostToDevice, st));
    HIP_TRY(launch_sample(logits_dev, ld, rows, e->c.vocab, e->d_svalid, e->d_spos, e->d_sseed, e->d_stemp,
                          e->d_stok, e->d_slp, st));
    HIP_TRY(hipMemcpyAsync(htok, e->d_stok, sizeof(int32_t) * rows, hipMemcpyDeviceToHost, st));
    HIP_TRY(hipMemcpyAsync(hlp, e->d_slp, sizeof(float) * rows, hipMemcpyDeviceToHost, st));
    HIP_TRY(hipStreamSynchronize(st));
    std::memcpy(tokens_out, htok, sizeof(int32_t) * rows);
    if (logprobs_out) std::memcpy(logprobs_out, hlp, sizeof(float) * rows);
    return CORUN_OK;
}

extern "C" corun_status corun_time_kernel(corun_engine *e, int32_t kernel, int32_t layer, int32_t n_iters,
                                          float *avg_us)
{
    if (!e || !avg_us) return fail(CORUN_E_INVAL, "null argument");
    if (kernel < 0 || kernel >= CORUN_K_COUNT) return fail(CORUN_E_INVAL, "unknown kernel id %d", kernel);
    if (layer < 0 || layer >= e->c.n_layers) return fail(CORUN_E_INVAL, "layer %d out of range", layer);
    if (n_iters < 1) return fail(CORUN_E_INVAL, "n_iters must be >= 1");
    if (!e->decoded) return fail(CORUN_E_STATE, "no decode step has run: the kernels have no validated inputs");
    ST_TRY(enter(e));
    // every timed launch runs on the last step's own (validated) inputs
    ST_TRY(restore_inputs(e));
    hipEvent_t t0, t1;
    HIP_TRY(hipEventCreate(&t0));
    HIP_TRY(hipEventCreate(&t1));
    corun_status s = launch_one(e, kernel, layer);   // warm-up
    if (s == CORUN_OK && hipEventRecord(t0, e->st) != hipSuccess) s = fail(CORUN_E_HIP, "event record failed");
    // cycle through the layers so every launch streams its own weights and
    // cache from HBM, as in the step (one layer's weights fit the 256 MB
    // last-level cache, all of them do not)
    for (int i = 0; s == CORUN_OK && i < n_iters; ++i) s = launch_one(e, kernel, (layer + i) % e->c.n_layers);
    float ms = 0.f;
    if (s == CORUN_OK) {
        if (hipEventRecord(t1, e->st) != hipSuccess || hipEventSynchronize(t1) != hipSuccess ||
            hipEventElapsedTime(&ms, t0, t1) != hipSuccess)
            s = fail(CORUN_E_HIP, "event timing failed");
    }
    (void)hipEventDestroy(t0);
    (void)hipEventDestroy(t1);
    if (s == CORUN_OK) *avg_us = 1000.f * ms / n_iters;
    return s;
}

extern "C" corun_status corun_profile_step(corun_engine *e, int32_t n_steps, float *avg_us, int32_t *launches_out)
{
    if (!e || !avg_us) return fail(CORUN_E_INVAL, "null argument");
    if (n_steps < 1) return fail(CORUN_E_INVAL, "n_steps must be >= 1");
    if (!e->decoded) return fail(CORUN_E_STATE, "no decode step has run: the kernels have no validated inputs");
    ST_TRY(enter(e));
    double sum[CORUN_K_COUNT + 1] = {};
    int cnt[CORUN_K_COUNT + 1] = {};
    corun_status s = CORUN_OK;
    for (int i = 0; i < n_steps && s == CORUN_OK; ++i) {
        s = restore_inputs(e);   // every step at the last step's own validated inputs
        if (s != CORUN_OK) break;
        e->prof.clear();
        e->rec.used = 0;
        e->rec.launches.clear();
        e->profiling = true;
        s = enqueue_step(e);
        e->profiling = false;
        if (s != CORUN_OK) break;
        if (hipStreamSynchronize(e->st) != hipSuccess) {
            s = fail(CORUN_E_HIP, "profiled step failed");
            break;
        }
        for (const auto &r : e->prof) {
            double us = 0.0;   // the class's kernels, each from its own start to its own end
            for (size_t j = r.first; j < r.end && s == CORUN_OK; ++j) {
                float ms = 0.f;
                if (hipEventElapsedTime(&ms, e->rec.launches[j].first, e->rec.launches[j].second) != hipSuccess)
                    s = fail(CORUN_E_HIP, "event timing failed");
                us += 1000.0 * ms;
            }
            if (s != CORUN_OK) break;
            sum[r.kind] += us;
            cnt[r.kind] += 1;
        }
    }
    e->profiling = false;
    if (s != CORUN_OK) return s;
    for (int k = 0; k < CORUN_K_COUNT; ++k) {
        avg_us[k] = cnt[k] ? (float)(sum[k] / cnt[k]) : 0.f;
        if (launches_out) launches_out[k] = cnt[k] / n_steps;
    }
    return CORUN_OK;
}
