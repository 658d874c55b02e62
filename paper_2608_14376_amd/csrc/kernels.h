// kernels.h -- launchers of the gfx950 kernels, called by the host engine.
// Every launcher enqueues on `st` and returns the launch error code.  The
// launch geometry of each is a function of its size arguments only; no kernel
// reads the number of live rows.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <hip/hip_ext.h>

#include <utility>
#include <vector>

namespace corun {

// While set on the calling thread (nullptr: off), every kernel launch of the
// launchers below records a pair of events around the kernel's own execution
// and appends it to `launches`; events come from `pool` (grown as needed,
// owned by the caller), `used` of them taken so far.
struct LaunchRecorder {
    std::vector<hipEvent_t> pool;
    size_t used = 0;
    std::vector<std::pair<hipEvent_t, hipEvent_t>> launches;
};
void set_launch_recorder(LaunchRecorder *r);

// Per-row token selection and fp32 residual init: x[b] = float(E[tok_b]),
// tok_b = valid[b] ? tokens[b] : 0; with ss, also the sums of squares of x[b]
// over 16-column groups, ss[b][H / 16] (launch_gemv's norm input).
hipError_t launch_embed(const uint16_t *E, const int32_t *tokens, const uint8_t *valid, int rows,
                        int H, float *x, hipStream_t st, float *ss = nullptr);

// Mixture-of-experts combine folded into the next RMSNorm:
// x[b] += sum_{r < top_k} w[b][r] y[b top_k + r] (rank order) for valid rows.
struct MoeFold {
    const float *y = nullptr;       // [rows * top_k][H] expert outputs, fp32
    const float *w = nullptr;       // [rows][top_k] routing weights
    const uint8_t *valid = nullptr;
    int top_k = 0;
};

// x[b] += sum_{s<S} part[s][b] (fixed order s = 0..S-1) [+ the MoE combine],
// then h[b] = bf16(x[b] * rsqrt(mean(x[b]^2) + eps) * g).
hipError_t launch_rmsnorm(float *x, const float *part, int S, long long part_stride, int rows, int H,
                          const uint16_t *g, float eps, uint16_t *h, hipStream_t st, MoeFold mf = MoeFold{});

// Mixture-of-experts routing: per valid row, top_k experts of the router
// logits (sum of S split partials [S][rows][E]), ties to the lower id, with
// renormalised softmax weights; padding rows get sel = -1.  Optionally the
// choice and the summed router logits are copied to sel_trace [rows][top_k]
// and logit_trace [rows][E] (valid rows' logits only).
hipError_t launch_moe_route(const float *part, int S, long long part_stride, int rows, int E, int top_k,
                            const uint8_t *valid, int32_t *sel, float *wsel, hipStream_t st,
                            int32_t *sel_trace = nullptr, float *logit_trace = nullptr);
// Deterministic dispatch of the n_assign = rows * top_k assignments into the
// fixed pool of n_slots 16-row tiles: list (expert-major, increasing
// assignment) and tiles[slot] = {expert, first list index, count}.
hipError_t launch_moe_dispatch(const int32_t *sel, int n_assign, int E, int n_slots, int32_t *list, int32_t *tiles,
                               hipStream_t st);
// out[a][n] = sum_k A[a / row_div][k] W_e[n][k] for every listed assignment a
// of expert e (W_e = W + e * w_expert_stride), one launch over all tile slots.
hipError_t launch_moe_gemm(const uint16_t *A, int lda, int row_div, const uint16_t *W, long long w_expert_stride, int N,
                           int K, const int32_t *list, const int32_t *tiles, int n_slots, float *out, int ldo,
                           hipStream_t st);
// The same product on the pipelined kernel (K % 64 == 0): one 32 x 128 tile
// per (128 columns, tile slot), weights row-major per expert or tile-packed
// per expert (packed; w_expert_stride in elements of the packed copy).
// With act (packed gate/up-interleaved copies, N % 128 == 0) the epilogue
// writes act[a][j] = SwiGLU of feature j (bf16, ld ldo) instead of out.
hipError_t launch_moe_gemm_dma(const uint16_t *A, int lda, int row_div, const uint16_t *W, long long w_expert_stride,
                               bool packed, int N, int K, const int32_t *list, const int32_t *tiles, int n_slots,
                               float *out, uint16_t *act, int ldo, hipStream_t st);

// Projection partials: out[s][m][n] = sum_{k in chunk s} A[m][k] W[n][k]
// for m < M_store (bf16 MFMA, fp32 accumulate).  A has lda columns and at
// least roundup(M, 64) readable rows.  K % 8 == 0, N % 16 == 0.
// Best (value, column) of one row over one wavefront's column block.
struct ArgBest {
    float v;
    int i;
};

// The QKV projection's split partials for an attention kernel that applies
// the QKV epilogue itself (launch_attn_split): part [S][rows][(nq + 2 nkv) d]
// with split stride `stride`, and the RoPE table.
struct QkvIn {
    const float *part = nullptr;
    int S = 0;
    long long stride = 0;
    const float2 *rope = nullptr;
};

// Expert tiles of a mixture-of-experts projection (launch_moe_dispatch):
// slot s holds tiles[3 s + 2] assignments list[tiles[3 s + 1] ..] of expert
// tiles[3 s]; an assignment's A row is assignment / row_div; expert e's
// weight starts at W + e w_stride.
struct ExpertTiles {
    const int32_t *list = nullptr, *tiles = nullptr;
    int row_div = 1;
    long long w_stride = 0;
};

struct GemmShape {
    int M, N, K;
    int S;          // split-K count
    int Kc;         // K elements per split (multiple of 32)
    int mt;         // skinny kernel: 16-row M tiles per wave: 1, 2 or 4
    int bm;         // 0 = skinny kernel; 64, 128, 256 = LDS-tiled kernel with this M tile
    int bn;         // > 0: pipelined kernel with bm x bn tiles (128 x 128, 256 x 128, 256 x 256)
    int pk;         // 1: W is the tile-packed copy (launch_pack_weights); bm 32 or 64, bn 128 only
};
// Dispatch on g.bm.
hipError_t launch_proj(const uint16_t *A, int lda, const uint16_t *W, const GemmShape &g, float *out,
                       long long split_stride, int ldo, hipStream_t st, ArgBest *amax = nullptr);
// With amax != nullptr (S == 1 only) the epilogue also writes, per row m and
// column block cb of 64 columns, amax[m * ceil(N / 64) + cb].
hipError_t launch_gemm(const uint16_t *A, int lda, const uint16_t *W, const GemmShape &g, float *out,
                       long long split_stride, int ldo, hipStream_t st, ArgBest *amax = nullptr);
// LDS-tiled variant for large M: tiles of bm (64, 128 or 256) x 128, split-K
// over grid.y, same output contract as launch_gemm (no argmax epilogue).
hipError_t launch_gemm_tiled(const uint16_t *A, int lda, const uint16_t *W, const GemmShape &g, int bm, float *out,
                             long long split_stride, int ldo, hipStream_t st, ArgBest *amax = nullptr);
// Pipelined large-M variant (direct global -> LDS loads, 32x32 MFMA tiles):
// K and Kc multiples of 64 (32 for bn == 256).
// With act != nullptr (g.pk, S == 1, N % 128 == 0): W is the gate/up-
// interleaved packed copy of a [2F, K] gate/up weight (launch_pack_weights
// with interleave) and the kernel writes act[m * ldo + j] = SwiGLU of
// feature j (bf16) instead of fp32 outputs; out and amax are unused.
hipError_t launch_gemm_dma(const uint16_t *A, int lda, const uint16_t *W, const GemmShape &g, float *out,
                           long long split_stride, int ldo, hipStream_t st, ArgBest *amax = nullptr,
                           uint16_t *act = nullptr);
inline int gemm_col_blocks(int N) { return (N + 63) / 64; }
// next[r] = best index over the np column-block partials of row r (-1 for padding rows).
hipError_t launch_argmax_partials(const ArgBest *part, int rows, int np, const uint8_t *valid, int32_t *next,
                                  hipStream_t st);

// Reduce QKV partials, round to bf16, rotate q and k by their position,
// round again, write q (bf16 [rows][nq*d]) and append k, v to the cache.
struct KvView {
    int layout;                 // 0 contiguous, 1 paged
    int max_seq_len;            // contiguous
    int page_size, max_pages_per_seq;
    const int32_t *page_table;  // device
};
hipError_t launch_qkv_post(const float *part, int S, long long part_stride, int rows,
                           const uint8_t *valid, const int32_t *pos, const int32_t *slot_of_row,
                           int slot_const, int nq, int nkv, int d, const float2 *rope_tab,
                           uint16_t *q, uint16_t *kc, uint16_t *vc, KvView kv, hipStream_t st);

// Split-KV decode attention.  Row r (slot slot_of_row[r] or slot_const,
// attending keys 0..pos[r]) is cut into chunks of `chunk` tokens; block
// (split, kvh, r) writes the chunk's (max, sum, unnormalised acc) for the G
// query heads of kv head kvh.  Merge combines the splits in index order.
// With qi.part set, q is not read: every block applies the QKV epilogue of
// launch_qkv_post to its group's q from the split partials, and the block
// holding the new token (position pos[r]) also makes its k and v, appends
// them to the cache and uses them -- the same bits launch_qkv_post writes.
hipError_t launch_attn_split(const uint16_t *q, int rows, const uint8_t *valid, const int32_t *pos,
                             const int32_t *slot_of_row, int slot_const, int nq, int nkv, int d,
                             uint16_t *kc, uint16_t *vc, KvView kv, int chunk,
                             int max_splits, float *ws, hipStream_t st, QkvIn qi = QkvIn{},
                             const int32_t *row_order = nullptr);
hipError_t launch_attn_merge(const float *ws, int rows, const uint8_t *valid, const int32_t *pos,
                             int nq, int nkv, int d, int chunk, int max_splits, uint16_t *o,
                             hipStream_t st);

// Seeded sampling of rows of fp32 logits (row stride ld): token[r] =
// argmax_v (l_v / temp[r] + g_v) with g_v from Philox4x32-10 keyed by seed[r],
// counter (pos[r], v, 0, 0); greedy where temp[r] <= 0; logprob[r] of the
// chosen token; padding rows get -1 / 0.
hipError_t launch_sample(const float *logits, long long ld, int rows, int V, const uint8_t *valid, const int32_t *pos,
                         const uint64_t *seed, const float *temp, int32_t *token, float *logprob, hipStream_t st);

// Causal attention of the isolated prefill: q (bf16 [n][nq d], row i = query
// position p0 + i) against keys 0..t of `slot` for query position t, o (bf16
// [n][nq d]).  Keys before p0 are read from the cache (earlier chunks of the
// prompt).  Sized by (n, p0) only.
hipError_t launch_prefill_attn(const uint16_t *q, int n, int p0, int nq, int nkv, int d, int slot, const uint16_t *kc,
                               const uint16_t *vc, KvView kv, uint16_t *o, hipStream_t st);

// The same attention for several prompts in one launch: seq (device int32
// [nseq][4]) = (first row in q/o, length, cache slot, first unit group),
// total_groups = the sum over prompts of ceil(ceil(len / 32) G / 8).  Each
// prompt's results are bit-identical to its own launch with p0 = 0.
// dst row i (bf16 [n][H]) = src row seq[i][0] + seq[i][1] - 1.
hipError_t launch_gather_last_rows(const uint16_t *src, const int32_t *seq, int n, int H, uint16_t *dst, hipStream_t st);

hipError_t launch_prefill_attn_multi(const uint16_t *q, const int32_t *seq, int nseq, int total_groups, int nq,
                                     int nkv, int d, const uint16_t *kc, const uint16_t *vc, KvView kv, uint16_t *o,
                                     hipStream_t st);

// a[m][j] = bf16(silu(bf16(sum_s gate)) * bf16(sum_s up)) over the partials
// of the [2F] gate/up projection (gate columns first).
hipError_t launch_swiglu(const float *part, int S, long long part_stride, int rows, int F,
                         uint16_t *a, int lda, hipStream_t st);

// out[i] = sum_{s<S} part[s * stride + i], s in order, for i < n.
hipError_t launch_reduce_splits(const float *part, int S, long long stride, long long n, float *out,
                                hipStream_t st);

// next[b] = first index of the maximum of logits[b] (valid rows), -1 otherwise.
hipError_t launch_argmax(const float *logits, int rows, int V, const uint8_t *valid, int32_t *next,
                         hipStream_t st);

// Device-side feedback between replayed steps: live rows take their next
// token and advance their position; the step's tokens are appended to the
// history at step index *counter, which then increments.
hipError_t launch_feedback(int32_t *tokens, int32_t *seq_lens, const uint8_t *valid,
                           const int32_t *next, int B, int32_t *history, int32_t *counter,
                           int max_hist, hipStream_t st);

// cos / sin table of the rotary embedding: tab[p][i] = (cos, sin)(p * theta^(-2i/d))
// evaluated in fp64 and rounded to fp32.
hipError_t launch_rope_table(float2 *tab, int max_pos, int d, double theta, hipStream_t st);

// fill n bytes with the byte value v (graph-safe replacement for memset)
hipError_t launch_fill_u32(uint32_t *p, long long n_words, uint32_t v, hipStream_t st);
// Tile-packed copy of a row-major [N, K] bf16 weight (K % 64 == 0) for the
// pipelined kernel's 128 x 64 weight tiles: [ceil(N / 128)][K / 64][128][64],
// rows past N zero; packed_weight_elems(N, K) elements.
// With interleave (N % 128 == 0), tile nt holds rows 64 nt .. 64 nt + 63 of
// each half of W: a gate/up weight's gate and up rows of the same features.
size_t packed_weight_elems(int N, int K);
hipError_t launch_pack_weights(const uint16_t *W, int N, int K, uint16_t *P, hipStream_t st, bool interleave = false);

// prefill helpers: pos[t] = t for t < n
// Fragment-packed copy of a row-major [N, K] weight for launch_gemv (layout
// and row orders at k_pack_frag): mode 0 rows in order, 1 rotation pairs of
// head_dim d (qkv), 2 gate/up feature pairs ([2F, K], gate rows first).
// N % 16 == 0, K % 8 == 0; P holds frag_packed_elems(N, K) bf16.
size_t frag_packed_elems(int N, int K);
hipError_t launch_pack_frag(const uint16_t *W, int N, int K, int mode, int d, uint16_t *P, hipStream_t st);

enum { GV_RESID = 0, GV_QKV = 1, GV_SWIGLU = 2 };
// A operand of launch_gemv: bf16 activations a [M][lda], or (a == nullptr)
// the RMSNorm of the fp32 residual x [M][K] with gain g and eps, its 1 / rms
// from ss [M][K / 16], the sums of squares of 16-column groups of x.
struct GemvIn {
    const uint16_t *a = nullptr;
    int lda = 0;
    const float *x = nullptr;
    const float *ss = nullptr;
    const uint16_t *g = nullptr;
    float eps = 0.f;
};
// Outputs per epilogue: GV_RESID x [M][N] (added into) and ss [M][N / 16];
// GV_SWIGLU act [M][N / 2]; GV_QKV q [M][nq d] and the cache (row = slot,
// position pos[row], rows with valid[row] == 0 skipped), rotation table rope.
struct GemvOut {
    float *x = nullptr;
    float *ss = nullptr;
    uint16_t *act = nullptr;
    uint16_t *q = nullptr, *kc = nullptr, *vc = nullptr;
    KvView kv{};
    const float2 *rope = nullptr;
    const uint8_t *valid = nullptr;
    const int32_t *pos = nullptr;
    int nq = 0, nkv = 0, d = 0;
};
// y = A W^T over M <= 16 rows from the fragment-packed W, one workgroup per
// 16 output columns; supported: (GV_RESID, activations), (GV_QKV, norm),
// (GV_SWIGLU, norm).
hipError_t launch_gemv(const uint16_t *Wp, int M, int N, int K, int epi, const GemvIn &in, const GemvOut &out,
                       hipStream_t st);

hipError_t launch_iota(int32_t *p, int n, hipStream_t st);

}  // namespace corun
