/*
 * corun.h -- C ABI of the MI355X (gfx950) CoRun decode/prefill library.
 *
 * CoRun (arXiv 2608.14376) makes LLM inference deterministic without
 * batch-invariant kernels: every decode iteration is padded to one fixed batch
 * size and replayed as one captured graph (Sec. IV, "Fixed-Shape Batched
 * Decode"), every prompt is prefilled alone at its own length (Sec. IV,
 * "Isolated Prefill"), and the kernels only need to be position-invariant:
 * F_n(PX) = P F_n(X) for every permutation P at the fixed shape n (Sec. III,
 * Definition 2).  The determinism argument (Sec. IV, "Determinism Argument")
 * then gives, for a request at slot p of the padded step D_N,
 *     pi_p D_N(X) = d(z)
 * -- its logits, next token and KV append depend only on its own state z.
 *
 * This library provides D_N for a pre-norm grouped-query decoder (dense or
 * mixture-of-experts), the isolated prefill, and the greedy sampler S(l)
 * (Sec. IV, "Shape-Aligned Sampling" with no random variate).  Each live row's
 * outputs are bitwise independent of which other requests or padding rows
 * share the step and of the slot it occupies.
 *
 * Conventions (all entry points):
 *  - Pointers marked "device" are HIP device pointers; "host" are ordinary
 *    host memory.  The caller owns every buffer it passes.  The engine borrows
 *    the weight, KV-cache and page-table buffers for its whole lifetime (the
 *    captured graph bakes their addresses in) and owns only its workspace.
 *  - Every call returns a corun_status; no call aborts or throws.  On failure
 *    corun_last_error() returns a message for the calling thread.
 *  - Host-side validation happens before anything is enqueued: a call that
 *    fails validation has no side effect on device memory.
 *  - One engine is used from one host thread at a time; calls are ordered
 *    after prior work on the `stream` given at creation and complete before
 *    they return (the outputs they return are host values).
 *  - bf16 tensors are raw IEEE bfloat16 bit patterns; matrices use the
 *    PyTorch Linear layout [out_features, in_features], row-major.
 */
#ifndef CORUN_H
#define CORUN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct corun_engine corun_engine;

typedef enum {
    CORUN_OK = 0,
    CORUN_E_INVAL = -1,     /* null pointer, out-of-range token, slot or length */
    CORUN_E_SHAPE = -2,     /* model or batch shape the kernels do not support */
    CORUN_E_CAPACITY = -3,  /* KV cache (or prefill workspace) too small */
    CORUN_E_HIP = -4,       /* HIP runtime failure; message has hipGetErrorString */
    CORUN_E_STATE = -5      /* call not valid for this engine (e.g. no prefill workspace) */
} corun_status;

enum { CORUN_KV_CONTIGUOUS = 0, CORUN_KV_PAGED = 1 };

/* Model shape.  n_experts = top_k = expert_ffn = 0 selects a dense SwiGLU
 * MLP of width `ffn`; otherwise every layer routes each token to top_k of
 * n_experts SwiGLU experts of width expert_ffn (softmax over all experts,
 * top_k, renormalised).  Requirements: hidden, ffn, expert_ffn multiples of
 * 16 (a K dimension may have a tail of 8, e.g. ffn = 688); head_dim 64 or
 * 128; n_heads a multiple of n_kv_heads with n_heads / n_kv_heads <= 16;
 * vocab a multiple of 16. */
typedef struct {
    int32_t n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn, vocab;
    int32_t n_experts, top_k, expert_ffn;
    float rms_eps, rope_theta;
} corun_model_cfg;

/* Weights: device bf16 buffers, caller-owned, borrowed for the engine's
 * lifetime and not to be changed during it (the engine may keep packed
 * copies: corun_options.no_weight_pack).  Per-layer fields are HOST arrays
 * of n_layers DEVICE pointers (copied at creation).  Dense models leave the
 * three expert fields NULL; MoE models leave w_gate_up / w_down NULL. */
typedef struct {
    const void *embed;                 /* [vocab, hidden] */
    const void *final_norm;            /* [hidden] */
    const void *lm_head;               /* [vocab, hidden] */
    const void *const *attn_norm;      /* [L] -> [hidden] */
    const void *const *w_qkv;          /* [L] -> [(nq + 2 nkv) d, hidden]: q rows, then k, then v, head-major */
    const void *const *w_o;            /* [L] -> [hidden, nq d] */
    const void *const *mlp_norm;       /* [L] -> [hidden] */
    const void *const *w_gate_up;      /* [L] -> [2 ffn, hidden], gate rows first */
    const void *const *w_down;         /* [L] -> [hidden, ffn] */
    const void *const *w_router;       /* [L] -> [n_experts, hidden] */
    const void *const *w_exp_gate_up;  /* [L] -> [n_experts, 2 expert_ffn, hidden] */
    const void *const *w_exp_down;     /* [L] -> [n_experts, hidden, expert_ffn] */
} corun_weights;

/* KV cache: device bf16, caller-owned, borrowed.  k and v are HOST arrays of
 * n_layers DEVICE pointers.  Keys and values are stored by token (each
 * token's head_dim elements contiguous):
 *  contiguous: K and V layers [n_slots, n_kv_heads, max_seq_len, head_dim];
 *              max_seq_len a multiple of 16;
 *  paged:      K and V layers [num_pages, n_kv_heads, page_size, head_dim];
 *              page_table (DEVICE int32 [n_slots, max_pages_per_seq]) maps a
 *              slot's token t to page page_table[slot][t / page_size] at
 *              position t % page_size; page_size a multiple of 16; capacity
 *              per slot is max_pages_per_seq * page_size tokens.
 * Slot b of the decode step reads and appends the cache of slot b. */
typedef struct {
    int32_t layout;                    /* CORUN_KV_CONTIGUOUS | CORUN_KV_PAGED */
    int32_t n_slots;                   /* >= B_fixed */
    int32_t max_seq_len;               /* contiguous capacity per slot (tokens) */
    int32_t page_size, num_pages, max_pages_per_seq;   /* paged only */
    void *const *k;
    void *const *v;
    const int32_t *page_table;
} corun_kv;

/* Creation options; pass NULL for defaults (all fields 0). */
typedef struct {
    int32_t attn_chunk;        /* split-KV chunk in tokens (multiple of 64); 0 = chosen from (model, B, capacity);
                                  a chunk >= the capacity turns split-KV off (one split per row) */
    int32_t max_prefill_len;   /* prefill workspace in tokens; 0 = none (corun_prefill returns CORUN_E_STATE) */
    int32_t no_graph;          /* 1 = launch the step's kernels eagerly instead of replaying the captured graph */
    int32_t poison_workspace;  /* 1 = fill the workspace with NaN bit patterns at creation (test aid) */
    int32_t split_k_override;  /* >0: force this split-K factor on every projection (test aid; changes the plan) */
    int32_t gemm_bm;           /* 0 = automatic; 64/128/256 = force the LDS-tiled projection kernel with this
                                  M tile (tuning aid; changes the plan) */
    int32_t batch_invariant;   /* 1 = batch-invariant kernels, the baseline CoRun is measured against (Sec. III,
                                  "Batch-Dependent GPU Reductions", Fig. 3b, and Definition 1): every projection, in
                                  decode and prefill, runs without split-K on one kernel whatever B or the prompt
                                  length (each output element one MFMA chain over K in order; the tile, which
                                  changes no element's arithmetic, still follows M), and decode attention runs
                                  with split-KV off (one split covers the whole cache), so a row's results depend
                                  on neither its position nor B.  Requires attn_chunk, split_k_override and
                                  gemm_bm = 0. */
    int32_t bi_prefill;        /* 1 = batch-invariant prefill only (Sec. VIII, "Batch-Invariant Kernels for
                                  Prefill": the hybrid of batch-invariant prefill and position-invariant
                                  fixed-shape decode): every prefill uses the plan of batch_invariant, and
                                  corun_prefill_batch is enabled; decode keeps its fixed-B plan. */
    int32_t no_weight_pack;    /* 0 (default) = at creation the engine copies every projection weight whose
                                  decode plan streams it with the small-M kernel (B_fixed <= 64) into a layout of
                                  contiguous 128 x 64 tiles, in memory it owns (one more copy of those weights),
                                  and reads that copy from then on, in decode and in prefill projections of up to
                                  64 rows; results are bit-identical either way.  With the small-batch layer
                                  (small_batch_layer) the four layer projections are copied into its fragment
                                  layout instead.  The weights must not change after creation.  1 = no copies:
                                  read the caller's row-major weights (and no small-batch layer). */
    int32_t qkv_epilogue;      /* where the decode step applies the QKV epilogue (RoPE, KV append): 0 = chosen
                                  from B (inside the attention kernel for B_fixed <= 8, where it saves a launch;
                                  its own kernel above, where recomputing q in every attention block costs
                                  more); 1 = its own kernel; 2 = inside attention.  Bit-identical results. */
    int32_t record_routing;    /* 1 = mixture-of-experts engines keep, for every layer, each row's chosen experts
                                  and the router logits they were chosen from, for the last decode step and the
                                  last prefill call (corun_routing_trace).  Extra workspace of
                                  n_layers x rows x (top_k + n_experts) x 4 bytes; results are unchanged. */
    int32_t small_batch_layer; /* the decode layer for the smallest batches: every layer projection streams a
                                  fragment-packed weight copy (16 output columns x 32 K elements per 1 KB MFMA
                                  operand, made at creation in memory the engine owns) over the whole of K, with no
                                  split-K; O and down add straight into the fp32 residual, QKV and gate/up
                                  normalise their input on the fly, RoPE + KV append and SwiGLU run in their
                                  epilogues, and a layer launches no RMSNorm.  Results differ in rounding from the
                                  split-K plan (a different fixed K order), not in position invariance.
                                  0 = automatic: dense models at B_fixed = 1 (unless no_weight_pack,
                                  batch_invariant, qkv_epilogue, split_k_override or gemm_bm is set);
                                  1 = on for a dense model with B_fixed <= 8 (CORUN_E_INVAL otherwise);
                                  2 = off. */
} corun_options;

/* Create an engine for one fixed padded batch size B_fixed (Sec. IV,
 * "Fixed-Shape Batched Decode": the capture size).  Every plan choice --
 * GEMM tiles, split-K factors, the attention chunk -- is a function of
 * (cfg, B_fixed, kv capacity, options) only and never of how many rows are
 * live.  `stream` is a hipStream_t (NULL = the null stream) that calls are
 * ordered against.  On success *out owns a workspace and, unless no_graph,
 * the decode step is captured as one hipGraph on the first step. */
corun_status corun_engine_create(const corun_model_cfg *cfg, const corun_weights *w,
                                 const corun_kv *kv, int32_t B_fixed,
                                 const corun_options *opt, void *stream, corun_engine **out);

void corun_engine_destroy(corun_engine *e);

/* One padded decode step D_N over B_fixed slots (Sec. IV, "Fixed-Shape
 * Batched Decode" and "Determinism Argument").
 *  tokens     host int32 [B]: the token to feed each slot
 *  valid_mask host uint8 [B]: 1 = live request, 0 = padding (its token and
 *             seq_len are ignored; any values are allowed)
 *  seq_lens   host int32 [B]: tokens already cached for the slot, which is
 *             also the new token's 0-based position; a live row needs
 *             0 <= seq_len < capacity
 *  next_tokens host int32 [B] out: greedy next token (first index of the
 *             maximum fp32 logit), -1 for padding rows
 *  logits     device fp32 [B, vocab] out, or NULL: the step's logits
 *             (padding rows hold unspecified values)
 * Live rows append their k, v at position seq_len of their slot's cache in
 * every layer; padding rows write nothing.  Errors: CORUN_E_INVAL (token out
 * of range for a live row, negative seq_len), CORUN_E_CAPACITY (seq_len or
 * a page beyond the cache). */
corun_status corun_decode_step(corun_engine *e, const int32_t *tokens, const uint8_t *valid_mask,
                               const int32_t *seq_lens, int32_t *next_tokens, float *logits);

/* n_steps greedy decode steps with the live set fixed: step i+1 feeds each
 * live row the token step i produced and advances its seq_len by one, all on
 * the device (the same captured step, replayed n_steps times with no host
 * round trip).  tokens_out: host int32 [n_steps, B] (row i = step i's
 * next_tokens).  Requires seq_len + n_steps <= capacity for every live row. */
corun_status corun_decode_run(corun_engine *e, int32_t n_steps, const int32_t *tokens,
                              const uint8_t *valid_mask, const int32_t *seq_lens,
                              int32_t *tokens_out);

/* Isolated prefill of one prompt into `slot` (Sec. IV, "Isolated Prefill";
 * the base case of the determinism argument): the prompt runs alone, with a
 * launch plan that depends only on prompt_len (not on the engine's max_prefill_len;
 * corun_describe_prefill_plan), writes k, v for positions
 * 0..prompt_len-1 of the slot in every layer, and samples the first token
 * greedily from the last position's logits (Sec. IV, "Shape-Aligned
 * Sampling": one sampling row).
 *  prompt      host int32 [prompt_len], each in [0, vocab)
 *  token_out   host int32 out
 *  last_logits device fp32 [vocab] out, or NULL
 * Errors: CORUN_E_STATE without a prefill workspace, CORUN_E_CAPACITY if
 * prompt_len exceeds it or the slot's cache, CORUN_E_INVAL otherwise. */
corun_status corun_prefill(corun_engine *e, const int32_t *prompt, int32_t prompt_len, int32_t slot,
                           int32_t *token_out, float *last_logits);

/* One chunk of a chunked isolated prefill (Sec. IV, "Isolated Prefill": a
 * long prompt divided into fixed-size chunks that run alone, one iteration
 * each, in order; Algorithm 1 continues them before admitting other work).
 * Runs prompt positions start .. start+n-1 alone: their k, v are appended
 * at those positions of `slot` in every layer, and their queries attend to
 * positions 0 .. t of the slot's cache, the first `start` of which the
 * caller must already have written (the prompt's earlier chunks, in order).
 * The launch plan depends on n only (corun_describe_prefill_plan), so with a
 * chunk size fixed per deployment a prompt always runs as the same sequence
 * of shapes, on any engine of the model.
 *  tokens      host int32 [n]: the prompt's tokens at those positions
 *  token_out   host int32 out, or NULL: greedy token from position
 *              start+n-1 (the first generated token if this is the last chunk)
 *  last_logits device fp32 [vocab] out, or NULL: that position's logits
 * With token_out and last_logits both NULL the final norm and lm_head are
 * skipped (an inner chunk).  corun_prefill is the single chunk at start 0.
 * Errors: CORUN_E_STATE without a prefill workspace, CORUN_E_CAPACITY if n
 * exceeds it or start+n the slot's cache, CORUN_E_INVAL otherwise. */
corun_status corun_prefill_chunk(corun_engine *e, const int32_t *tokens, int32_t n, int32_t start, int32_t slot,
                                 int32_t *token_out, float *last_logits);

/* Most prompts one corun_prefill_batch call takes. */
#define CORUN_MAX_PREFILL_BATCH 64

/* Batched prefill of several whole prompts in one pass (Sec. VIII,
 * "Batch-Invariant Kernels for Prefill"): the prompts' tokens run as one
 * batch of rows through batch-invariant kernels -- one projection tile and
 * no split-K for any number of rows, row-wise norms, per-prompt causal
 * attention with each prompt's own plan -- so every prompt's k, v and
 * last-position logits are bit-identical to its own corun_prefill on the
 * same engine, whatever the other prompts are.  Requires an engine created
 * with bi_prefill or batch_invariant (else CORUN_E_STATE).
 *  tokens      host int32 [sum of lens]: the prompts back to back
 *  lens        host int32 [n], each >= 1; their sum at most max_prefill_len
 *  slots       host int32 [n]: distinct cache slots
 *  n           1 .. CORUN_MAX_PREFILL_BATCH
 *  tokens_out  host int32 [n] out: each prompt's greedy first token
 *  last_logits device fp32 [n, vocab] out, or NULL
 * Errors: CORUN_E_CAPACITY (sum of lens beyond the workspace, a prompt
 * beyond its slot's cache), CORUN_E_INVAL (bad sizes, slots, tokens). */
corun_status corun_prefill_batch(corun_engine *e, const int32_t *tokens, const int32_t *lens, const int32_t *slots,
                                 int32_t n, int32_t *tokens_out, float *last_logits);

/* The engine's fixed batch size, model configuration and KV description
 * (copies; the k/v/page-table pointers are the caller's borrowed ones).
 * Any out pointer may be NULL. */
corun_status corun_engine_info(const corun_engine *e, int32_t *B_fixed, corun_model_cfg *cfg, corun_kv *kv);

/* Routing record of a mixture-of-experts engine created with record_routing
 * (Sec. VII names the router as the fragile point of a mixture of experts: a
 * top-k choice is a comparison of floating-point logits).  source 0 = the
 * last decode step (rows = B_fixed), 1 = the last prefill call (rows = its
 * row count: prompt_len, the chunk length, or the batch's total tokens).
 *  sel     host int32 [n_layers][rows][top_k] out, or NULL: the experts each
 *          row was routed to in rank order (-1 for decode padding rows)
 *  logits  host fp32 [n_layers][rows][n_experts] out, or NULL: the router
 *          logits the choice was made from (unspecified for padding rows)
 *  rows_out host int32 out
 * Waits for the engine's stream.  Errors: CORUN_E_STATE (dense model, no
 * record_routing, or source 1 without a prefill workspace), CORUN_E_INVAL. */
corun_status corun_routing_trace(corun_engine *e, int32_t source, int32_t *sel, float *logits, int32_t *rows_out);

/* Request-bound seeded multinomial sampling (Sec. IV, "Shape-Aligned
 * Sampling"; y_t = S(l_t, R(s, t)) in Sec. IV, "Determinism Argument"), run on
 * logits that corun_decode_step (rows = B, the fixed shape) or corun_prefill
 * (rows = 1) wrote to a caller buffer.  The random variate of row r is a
 * function of (seeds[r], positions[r], column) only: u_v from Philox4x32-10
 * (Salmon et al., SC 2011) keyed by the 64-bit seed with counter
 * (positions[r], v, 0, 0), u = ((w0 >> 6) 2^26 + (w1 >> 6) + 1/2) 2^-52 from
 * its first two words, so no RNG state exists to be consumed, and
 * padding rows and co-runners cannot move a request's stream.
 *  token[r]   = argmax_v ( l[r][v] / T_r + g_v ), g_v = -ln(-ln u_v)
 *               (the Gumbel-max rule: an exact draw from softmax(l / T));
 *               greedy (argmax l, lowest index) where T_r <= 0;
 *  logprob[r] = log softmax(l[r] / T_r)[token[r]] (softmax(l[r]) if greedy),
 * decided and summed in fp64 with a fixed reduction order.
 *  logits_dev   device fp32 [rows][ld], ld >= vocab (caller-owned)
 *  valid        host uint8 [rows]; invalid rows get token -1, logprob 0
 *  positions    host int32 [rows]: position of the token being sampled
 *               (seq_len + 1 after a decode step, prompt_len after prefill)
 *  seeds        host uint64 [rows]; temperature host float [rows]
 *  tokens_out   host int32 [rows]; logprobs_out host float [rows] or NULL
 * Errors: CORUN_E_SHAPE for rows outside [1, B] or ld < vocab; CORUN_E_INVAL
 * for a null pointer, a negative position or a non-finite temperature of a
 * valid row.  Runs on the engine's stream after the caller's stream. */
corun_status corun_sample(corun_engine *e, const float *logits_dev, int64_t ld, int32_t rows,
                          const uint8_t *valid, const int32_t *positions, const uint64_t *seeds,
                          const float *temperature, int32_t *tokens_out, float *logprobs_out);

/* Most rows one corun_sample_noalloc call takes (the size of its static
 * staging). */
#define CORUN_SAMPLE_NOALLOC_MAX_ROWS 1024

/* corun_sample without an engine and without allocating, for callers that
 * cannot allocate device memory: code that must not call hipMalloc (a tight
 * serving loop, a harness that forbids it).  The same sampler and result
 * bits as corun_sample on the same logits and arguments; the per-row inputs
 * and outputs are staged in a fixed static device array of 25 KiB that each
 * GPU holds for the life of the process (rows at most
 * CORUN_SAMPLE_NOALLOC_MAX_ROWS).  Runs on `stream` (a hipStream_t; NULL =
 * the null stream) on the current device and waits for it before returning.
 * Every call on a GPU shares that GPU's staging: calls that overlap on one
 * device (from two threads, or on two streams at once) race; calls made one
 * after another do not.
 *  logits_dev   device fp32 [rows][ld], ld >= vocab (caller-owned)
 *  vocab        columns sampled per row, >= 1
 *  valid, positions, seeds, temperature, tokens_out, logprobs_out: as for
 *               corun_sample (host arrays of `rows` entries; logprobs_out may
 *               be NULL)
 * Errors: CORUN_E_SHAPE for rows outside [1, CORUN_SAMPLE_NOALLOC_MAX_ROWS],
 * vocab < 1 or ld < vocab; CORUN_E_INVAL as for corun_sample; CORUN_E_HIP. */
corun_status corun_sample_noalloc(const float *logits_dev, int64_t ld, int32_t rows, int32_t vocab,
                                  const uint8_t *valid, const int32_t *positions, const uint64_t *seeds,
                                  const float *temperature, int32_t *tokens_out, float *logprobs_out,
                                  void *stream);

/* ---------------------------------------------------------------------------
 * Host scheduler (Sec. IV, "Isolated Prefill", Algorithms 1 and 2, around the
 * fixed-shape batched decode and the request-bound sampler): a
 * continuous-batching loop with slot reuse, a concurrency limit and
 * full-sequence KV admission, driving corun_prefill, corun_decode_step and
 * corun_sample.  Each corun_sched_step() runs one iteration: the isolated
 * prefill of the request Algorithm 1 selects (the head of `running` whose
 * prefill is unfinished, else the head of `waiting` if fewer than
 * max_num_reqs are running and its prompt plus max_new_tokens fit the KV
 * cache now), else one decode step of every running request padded to B.
 * Requests leave at max_new_tokens, returning their slot (the lowest free one
 * is reused) and pages.  With a paged cache the scheduler owns the page-table
 * rows of the slots: all pages of the full sequence are taken at admission;
 * it keeps a host copy of the table, registered with the engine
 * (corun_engine_set_page_table_host) from creation until
 * corun_sched_destroy, so decode steps validate pages without a device copy.
 * The engine is borrowed and must outlive the scheduler.  engine NULL is a
 * dry run: the same scheduling, no model, tokens 0.  Not thread-safe; one
 * scheduler per engine.
 * ------------------------------------------------------------------------- */
typedef struct corun_sched corun_sched;
typedef struct {
    int32_t max_num_reqs;       /* concurrency limit, <= B (0 = B) */
    /* dry run only (engine NULL): the slots and cache; page_size 0 = contiguous */
    int32_t n_slots, max_seq_len, page_size, num_pages, max_pages_per_seq;
    int32_t prefill_chunk;      /* > 0: prefill prompts in chunks of this many tokens (the last one shorter),
                                   one isolated iteration each (corun_prefill_chunk); 0 = whole prompts */
    int32_t prefill_batch_tokens; /* > 0: batched prefill (Sec. VIII, batch-invariant prefill): a prefill
                                   iteration takes the request Algorithm 1 selects and the waiting requests
                                   behind it, in order, while each passes admission and the prompts total at
                                   most this many tokens, through one corun_prefill_batch (the engine needs
                                   bi_prefill; keep this within its max_prefill_len).  Excludes
                                   prefill_chunk.  0 = one prompt per prefill iteration. */
} corun_sched_cfg;

corun_status corun_sched_create(corun_engine *e, const corun_sched_cfg *cfg, corun_sched **out);
void corun_sched_destroy(corun_sched *s);
/* Queue one request (FIFO).  prompt: host int32 [prompt_len], copied.
 * temperature <= 0 is greedy.  CORUN_E_CAPACITY if prompt + max_new_tokens
 * can never fit one slot; CORUN_E_INVAL for a reused id or bad sizes. */
corun_status corun_sched_add_request(corun_sched *s, int64_t id, const int32_t *prompt, int32_t prompt_len,
                                     int32_t max_new_tokens, uint64_t seed, float temperature);
/* One iteration; event: 0 idle, 1 isolated prefill (a whole prompt or one
 * chunk of it), 2 decode step. */
corun_status corun_sched_step(corun_sched *s, int32_t *event);
/* A request's generated tokens and their log-probabilities so far (up to
 * cap), their count and whether it finished. */
corun_status corun_sched_output(const corun_sched *s, int64_t id, int32_t *tokens, float *logprobs, int32_t cap,
                                int32_t *n_generated, int32_t *finished);
/* Queue lengths, free slots and pages, and slot_owner [B] (request id, -1
 * free).  Any out pointer may be NULL. */
corun_status corun_sched_state(const corun_sched *s, int32_t *n_running, int32_t *n_waiting, int32_t *free_slots,
                               int32_t *free_pages, int64_t *slot_owner);
/* Message of the last failed scheduler call (engine failures included). */
const char *corun_sched_last_error(void);

/* Kernels that corun_time_kernel can time. */
enum {
    CORUN_K_QKV_GEMM = 0,     /* QKV projection (split-K partials) */
    CORUN_K_O_GEMM = 1,       /* attention output projection */
    CORUN_K_GATE_UP_GEMM = 2, /* gate/up projection */
    CORUN_K_DOWN_GEMM = 3,    /* down projection */
    CORUN_K_LM_HEAD = 4,      /* lm_head projection */
    CORUN_K_ATTN_SPLIT = 5,   /* split-KV decode attention */
    CORUN_K_ATTN_MERGE = 6,   /* fixed-order split merge */
    CORUN_K_RMSNORM = 7,      /* residual fold + RMSNorm */
    CORUN_K_QKV_POST = 8,     /* QKV epilogue: RoPE + KV append (no kernel where the attention kernel
                                 applies it: corun_options.qkv_epilogue) */
    CORUN_K_SWIGLU = 9,       /* SwiGLU epilogue (no kernel where the gate/up projection's epilogue applies it:
                                 packed weights without split-K) */
    CORUN_K_ARGMAX = 10,      /* greedy argmax */
    CORUN_K_MOE_ROUTER = 11,  /* MoE: router projection, top-k routing and dispatch (3 kernels) */
    CORUN_K_COUNT = 12
};
/* For mixture-of-experts models CORUN_K_GATE_UP_GEMM / CORUN_K_SWIGLU /
 * CORUN_K_DOWN_GEMM time the grouped expert kernels. */

/* Measurement aid: launch one kernel of the decode step n_iters times back
 * to back on the engine's stream, launch i using layer (layer + i) mod
 * n_layers (so weights and cache stream from HBM as in the step) and the
 * engine's current workspace (as left by the last step), and return the mean
 * duration per launch in microseconds, measured with HIP events around the
 * launches.  The launches run on the inputs of the last decode step (tokens,
 * valid mask, positions as validated by the call that ran it, uploaded again
 * first: the step itself advanced the positions), so a kernel that appends
 * to the cache rewrites the value that step wrote at that position.  Re-running a kernel rewrites the workspace
 * values it wrote in the step (the residual-folding RMSNorm adds its
 * partials again; the next step recomputes the residual from the
 * embedding).  CORUN_E_STATE before the engine's first decode step. */
corun_status corun_time_kernel(corun_engine *e, int32_t kernel, int32_t layer, int32_t n_iters, float *avg_us);

/* Measurement aid: n_steps decode steps, each on the inputs of the last
 * decode step (uploaded again first, as for corun_time_kernel), with the
 * step's kernels launched eagerly in the step's order, each with a pair of
 * HIP events recorded around its own execution (hipExtLaunchKernel).
 * avg_us[k] receives the mean duration of kernel class k's launches inside
 * those steps (a class that runs several kernels, such as the MoE router,
 * counts their sum; each launch runs after the kernels that precede it in
 * the step, as in the captured graph), launches[k] (or NULL) their count
 * per step; classes
 * that do not launch get 0.  Arrays of CORUN_K_COUNT entries.  The steps
 * rewrite the cache positions the last step wrote, with the same values.
 * CORUN_E_STATE before the engine's first decode step. */
corun_status corun_profile_step(corun_engine *e, int32_t n_steps, float *avg_us, int32_t *launches);

/* Host-only checks, usable without a GPU: the shape rules of
 * corun_model_cfg / corun_kv, and the per-row checks of corun_decode_step
 * for a batch of B rows (n_steps further tokens of capacity are required). */
corun_status corun_check_config(const corun_model_cfg *cfg, const corun_kv *kv, int32_t B_fixed);
corun_status corun_check_batch(const corun_model_cfg *cfg, const corun_kv *kv, const int32_t *page_table_host,
                               int32_t B, const int32_t *tokens, const uint8_t *valid_mask,
                               const int32_t *seq_lens, int32_t n_steps);

/* Paged caches: register a host copy of the page table (HOST int32
 * [n_slots, max_pages_per_seq], caller-owned, borrowed until replaced or
 * the engine is destroyed; NULL unregisters).  The host-side checks of
 * corun_decode_step / corun_decode_run / corun_prefill* then read it instead
 * of copying the device table back (a synchronous copy of the whole table on
 * every decode call).  The caller keeps it equal to the device table
 * whenever it calls into the engine: the kernels read the device table, the
 * checks the copy.  CORUN_E_STATE for an engine with a contiguous cache. */
corun_status corun_engine_set_page_table_host(corun_engine *e, const int32_t *page_table_host);

/* The launch plan an engine would use (host-only, no GPU): fills `out` with
 * up to `cap` int32 values -- B, padded M, then (N, K, split_k, k_chunk,
 * m_tile, n_tile) for the qkv, o, gate_up, down and lm_head projections
 * (m_tile 0 = the skinny kernel; n_tile 0 = the LDS-tiled kernel; m_tile =
 * n_tile = 16 the small-batch layer's fragment-packed kernel, k_chunk = K
 * rounded up to 32; else the pipelined kernel's N tile), then the attention
 * chunk and its maximum split count (32 values).  Returns the count written
 * or a negative corun_status (CORUN_E_INVAL for small_batch_layer = 1 where
 * the layer cannot run). */
int32_t corun_describe_plan(const corun_model_cfg *cfg, const corun_kv *kv, int32_t B_fixed,
                            const corun_options *opt, int32_t *out, int32_t cap);

/* The projection plan of a prefill call over n rows (host-only, no GPU):
 * (N, K, split_k, k_chunk, m_tile, n_tile) for the qkv, o, gate_up, down and
 * router projections (zeros where the model has none), 30 values.  It is a
 * function of (cfg, n, batch_invariant or bi_prefill) only -- not of the
 * engine's max_prefill_len, whose workspace holds the partials of any plan
 * up to that length (Sec. IV, "Isolated Prefill": a prompt's prefill shape
 * is fixed by the prompt).  Returns the count written or a negative
 * corun_status. */
int32_t corun_describe_prefill_plan(const corun_model_cfg *cfg, int32_t n, const corun_options *opt, int32_t *out,
                                    int32_t cap);

/* Message for the calling thread's last non-OK status ("" if none). */
const char *corun_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CORUN_H */
