// Host scheduler of CoRun (arXiv 2608.14376): isolated prefill (Sec. IV,
// "Isolated Prefill", Algorithms 1 and 2) around a fixed-shape batched decode
// (Sec. IV, "Fixed-Shape Batched Decode") with request-bound sampling (Sec.
// IV, "Shape-Aligned Sampling"), as a continuous-batching loop with slot
// reuse, a concurrency limit and full-sequence KV admission.
//
// The scheduler is a client of the engine's C ABI: corun_prefill_chunk,
// corun_decode_step and corun_sample.  Each schedule() call runs one
// iteration, either the isolated prefill of one request or one decode step
// of every running request, padded to the engine's fixed B.
//
// Without an engine (a dry run) every iteration is scheduled exactly the same
// way but runs no model: the generated tokens are 0.  That exposes the
// admission and slot logic to host-only tests.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <deque>
#include <string>
#include <unordered_map>
#include <vector>

#include "corun.h"

namespace {

thread_local std::string s_error;

// an engine call failed: its message becomes the scheduler's
corun_status from_engine(corun_status s)
{
    s_error = corun_last_error();
    return s;
}

corun_status sfail(corun_status s, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    s_error = buf;
    return s;
}

struct Request {
    int64_t id = 0;
    std::vector<int32_t> prompt;
    int32_t max_new = 0;
    uint64_t seed = 0;
    float temperature = 0.f;
    int32_t num_computed = 0;           // prompt tokens whose KV is cached (chunks done so far)
    int32_t slot = -1;
    std::vector<int32_t> pages;
    std::vector<int32_t> tokens;        // generated
    std::vector<float> logprobs;
    bool finished = false;
};

}  // namespace

struct corun_sched {
    corun_engine *e = nullptr;          // null: dry run
    int B = 0, max_num_reqs = 0, vocab = 0;
    int32_t chunk = 0;                  // prefill chunk (0 = whole prompts)
    int32_t batch_tokens = 0;           // batched prefill: most prompt tokens per prefill iteration (0 = one prompt)
    float *blogits = nullptr;           // device [n][vocab]: a batched prefill's last-position logits
    corun_kv kv{};
    bool paged = false;
    std::unordered_map<int64_t, Request> reqs;
    std::deque<int64_t> running, waiting;
    std::vector<int64_t> slot_owner;    // [B], -1 = free
    std::vector<int32_t> free_pages;    // stack, lowest id on top
    // paged: the host copy of the page table this scheduler keeps equal to
    // the device table and registers with the engine for its checks
    std::vector<int32_t> pt_host;
    float *logits = nullptr;            // device [B][vocab]
    float *last = nullptr;              // device [vocab]
    int64_t n_prefill = 0, n_decode = 0;
};

namespace {

int32_t pages_for(const corun_sched *s, const Request &r)
{
    const int64_t total = (int64_t)r.prompt.size() + r.max_new;
    return (int32_t)((total + s->kv.page_size - 1) / s->kv.page_size);
}

// The request's whole configured sequence (prompt + max_new tokens) fits the
// KV cache now, so no later decode step can run out of room (Sec. IV,
// "Isolated Prefill": full-sequence admission).
bool can_fit_full_sequence(const corun_sched *s, const Request &r)
{
    if (std::find(s->slot_owner.begin(), s->slot_owner.end(), (int64_t)-1) == s->slot_owner.end()) return false;
    const int64_t total = (int64_t)r.prompt.size() + r.max_new;
    if (!s->paged) return total <= s->kv.max_seq_len;
    const int32_t need = pages_for(s, r);
    return need <= s->kv.max_pages_per_seq && need <= (int32_t)s->free_pages.size();
}

// Algorithm 1: the request needing prefill, or none (-1).  A running head
// whose prompt is not fully computed continues first (chunked prefill); a
// waiting request starts only below the concurrency limit and when its full
// sequence fits.
int64_t find_prefill_request(corun_sched *s)
{
    if (!s->running.empty()) {
        const Request &head = s->reqs.at(s->running.front());
        if (head.num_computed < (int32_t)head.prompt.size()) return head.id;
    }
    if (!s->waiting.empty() && (int)s->running.size() < s->max_num_reqs) {
        const Request &head = s->reqs.at(s->waiting.front());
        if (can_fit_full_sequence(s, head)) return head.id;
    }
    return -1;
}

corun_status write_page_row(corun_sched *s, const Request &r)
{
    std::vector<int32_t> row(s->kv.max_pages_per_seq, r.pages.empty() ? 0 : r.pages[0]);
    std::copy(r.pages.begin(), r.pages.end(), row.begin());
    if (!s->e) return CORUN_OK;
    const size_t off = (size_t)r.slot * s->kv.max_pages_per_seq;
    int32_t *dst = const_cast<int32_t *>(s->kv.page_table) + off;
    if (hipMemcpy(dst, row.data(), row.size() * sizeof(int32_t), hipMemcpyHostToDevice) != hipSuccess)
        return sfail(CORUN_E_HIP, "page table update failed");
    std::copy(row.begin(), row.end(), s->pt_host.begin() + off);
    return CORUN_OK;
}

corun_status admit(corun_sched *s, Request &r)
{
    int slot = -1;
    for (int i = 0; i < s->B; ++i)
        if (s->slot_owner[i] < 0) {
            slot = i;                       // the lowest free slot
            break;
        }
    if (slot < 0) return sfail(CORUN_E_STATE, "no free slot");
    r.slot = slot;
    s->slot_owner[slot] = r.id;
    if (s->paged) {
        const int32_t need = pages_for(s, r);
        for (int i = 0; i < need; ++i) {
            r.pages.push_back(s->free_pages.back());
            s->free_pages.pop_back();
        }
        return write_page_row(s, r);
    }
    return CORUN_OK;
}

void release(corun_sched *s, Request &r)
{
    r.finished = true;
    if (r.slot >= 0) s->slot_owner[r.slot] = -1;
    r.slot = -1;
    for (auto it = r.pages.rbegin(); it != r.pages.rend(); ++it) s->free_pages.push_back(*it);
    r.pages.clear();
}

corun_status append(corun_sched *s, Request &r, int32_t tok, float lp)
{
    r.tokens.push_back(tok);
    r.logprobs.push_back(lp);
    (void)s;
    return CORUN_OK;
}

// Prefill of one request alone (its own shape): the whole prompt, or its next
// fixed-size chunk.  After the prompt's last position its first token is
// sampled from that position's logits (one sampling row).
corun_status run_prefill(corun_sched *s, Request &r)
{
    const int32_t L = (int32_t)r.prompt.size(), start = r.num_computed;
    const int32_t n = s->chunk > 0 ? std::min(s->chunk, L - start) : L - start;
    const bool last = start + n == L;
    int32_t tok = 0;
    float lp = 0.f;
    if (s->e) {
        corun_status st = corun_prefill_chunk(s->e, r.prompt.data() + start, n, start, r.slot,
                                              last ? &tok : nullptr, last ? s->last : nullptr);
        if (st != CORUN_OK) return from_engine(st);
        if (last) {
            const uint8_t one = 1;
            const int32_t pos = L;
            st = corun_sample(s->e, s->last, s->vocab, 1, &one, &pos, &r.seed, &r.temperature, &tok, &lp);
            if (st != CORUN_OK) return from_engine(st);
        }
    }
    r.num_computed = start + n;
    ++s->n_prefill;
    return last ? append(s, r, tok, lp) : CORUN_OK;
}

// One fixed-shape decode step of every running request, padded to B, then
// request-bound sampling of every live row.
corun_status run_decode(corun_sched *s)
{
    const int B = s->B;
    std::vector<int32_t> tokens(B, 0), seq(B, 0), pos(B, 0), next(B, -1);
    std::vector<uint8_t> valid(B, 0);
    std::vector<uint64_t> seeds(B, 0);
    std::vector<float> temp(B, 0.f), lps(B, 0.f);
    for (int64_t id : s->running) {
        const Request &r = s->reqs.at(id);
        if (r.tokens.empty()) continue;   // prefill unfinished (Algorithm 1 runs it first): not in this step
        tokens[r.slot] = r.tokens.back();
        seq[r.slot] = (int32_t)r.prompt.size() + (int32_t)r.tokens.size() - 1;   // cached tokens
        pos[r.slot] = seq[r.slot] + 1;                                           // the sampled token's position
        valid[r.slot] = 1;
        seeds[r.slot] = r.seed;
        temp[r.slot] = r.temperature;
    }
    if (s->e) {
        corun_status st = corun_decode_step(s->e, tokens.data(), valid.data(), seq.data(), next.data(), s->logits);
        if (st != CORUN_OK) return from_engine(st);
        st = corun_sample(s->e, s->logits, s->vocab, B, valid.data(), pos.data(), seeds.data(), temp.data(),
                          next.data(), lps.data());
        if (st != CORUN_OK) return from_engine(st);
    } else {
        std::fill(next.begin(), next.end(), 0);
    }
    ++s->n_decode;
    for (int64_t id : s->running) {
        Request &r = s->reqs.at(id);
        if (r.tokens.empty()) continue;
        corun_status st = append(s, r, next[r.slot], lps[r.slot]);
        if (st != CORUN_OK) return st;
    }
    return CORUN_OK;
}

// Requests that reached their output length leave `running` (in order) and
// give back their slot and pages.
void retire(corun_sched *s)
{
    std::deque<int64_t> keep;
    for (int64_t id : s->running) {
        Request &r = s->reqs.at(id);
        if ((int32_t)r.tokens.size() >= r.max_new) release(s, r);
        else keep.push_back(id);
    }
    s->running.swap(keep);
}

// The engine's own scheduling iteration (the role of the wrapped scheduler):
// admit and prefill the head of `waiting` if the concurrency limit and the
// KV cache allow it, else continue a running head's prefill, else decode
// every running request.  Inside Algorithm 2 only the selected request is
// visible, so this admits exactly it; called directly (nothing to prefill)
// the same checks keep it to a decode iteration.
corun_status schedule_origin(corun_sched *s, int32_t *event)
{
    if (!s->waiting.empty() && (int)s->running.size() < s->max_num_reqs &&
        can_fit_full_sequence(s, s->reqs.at(s->waiting.front()))) {
        const int64_t id = s->waiting.front();
        s->waiting.pop_front();
        Request &r = s->reqs.at(id);
        corun_status st = admit(s, r);
        if (st != CORUN_OK) return st;
        s->running.push_back(id);
        st = run_prefill(s, r);
        if (st != CORUN_OK) return st;
        *event = 1;
        return CORUN_OK;
    }
    if (!s->running.empty()) {
        Request &head = s->reqs.at(s->running.front());
        if (head.num_computed < (int32_t)head.prompt.size()) {
            corun_status st = run_prefill(s, head);
            if (st != CORUN_OK) return st;
            *event = 1;
            return CORUN_OK;
        }
        corun_status st = run_decode(s);
        if (st != CORUN_OK) return st;
        *event = 2;
        return CORUN_OK;
    }
    *event = 0;
    return CORUN_OK;
}

void remove_id(std::deque<int64_t> &q, int64_t id)
{
    q.erase(std::remove(q.begin(), q.end(), id), q.end());
}

// Batched prefill iteration (batch-invariant prefill, Sec. VIII): the
// request Algorithm 1 selected from `waiting` and the requests behind it, in
// order, while each passes the same admission checks (concurrency limit, a
// free slot, its full sequence in the cache after its batch-mates') and the
// batch's prompt tokens stay within batch_tokens.  They are admitted, run
// through one corun_prefill_batch -- each prompt's result bit-identical to
// its own prefill -- and each samples its first token; the batch then heads
// `running` in order, as Algorithm 2 puts an isolated request there.
corun_status run_prefill_batch(corun_sched *s, int64_t det, int32_t *event)
{
    std::vector<int64_t> batch = {det};
    int64_t tokens = (int64_t)s->reqs.at(det).prompt.size();
    int free_slots = (int)std::count(s->slot_owner.begin(), s->slot_owner.end(), (int64_t)-1) - 1;
    int64_t free_pages = s->paged ? (int64_t)s->free_pages.size() - pages_for(s, s->reqs.at(det)) : 0;
    auto it = std::find(s->waiting.begin(), s->waiting.end(), det);
    for (++it; it != s->waiting.end(); ++it) {
        const Request &r = s->reqs.at(*it);
        if ((int)batch.size() >= CORUN_MAX_PREFILL_BATCH) break;
        if ((int)(s->running.size() + batch.size()) >= s->max_num_reqs) break;
        if (tokens + (int64_t)r.prompt.size() > s->batch_tokens) break;
        if (free_slots < 1) break;
        if (!s->paged && (int64_t)r.prompt.size() + r.max_new > s->kv.max_seq_len) break;
        if (s->paged && (pages_for(s, r) > s->kv.max_pages_per_seq || pages_for(s, r) > free_pages)) break;
        batch.push_back(r.id);
        tokens += (int64_t)r.prompt.size();
        --free_slots;
        if (s->paged) free_pages -= pages_for(s, r);
    }
    std::vector<int32_t> toks, lens, slots;
    for (int64_t id : batch) {
        remove_id(s->waiting, id);
        Request &r = s->reqs.at(id);
        corun_status st = admit(s, r);
        if (st != CORUN_OK) return st;
        toks.insert(toks.end(), r.prompt.begin(), r.prompt.end());
        lens.push_back((int32_t)r.prompt.size());
        slots.push_back(r.slot);
    }
    const int n = (int)batch.size();
    std::vector<int32_t> first(n, 0), pos(n);
    std::vector<float> lps(n, 0.f);
    std::vector<uint64_t> seeds(n);
    std::vector<float> temps(n);
    std::vector<uint8_t> valid(n, 1);
    for (int i = 0; i < n; ++i) {
        const Request &r = s->reqs.at(batch[i]);
        pos[i] = (int32_t)r.prompt.size();
        seeds[i] = r.seed;
        temps[i] = r.temperature;
    }
    if (s->e) {
        corun_status st = corun_prefill_batch(s->e, toks.data(), lens.data(), slots.data(), n, first.data(), s->blogits);
        if (st != CORUN_OK) return from_engine(st);
        st = corun_sample(s->e, s->blogits, s->vocab, n, valid.data(), pos.data(), seeds.data(), temps.data(),
                          first.data(), lps.data());
        if (st != CORUN_OK) return from_engine(st);
    }
    std::deque<int64_t> running(batch.begin(), batch.end());
    for (int64_t id : s->running) running.push_back(id);
    s->running.swap(running);
    for (int i = 0; i < n; ++i) {
        Request &r = s->reqs.at(batch[i]);
        r.num_computed = (int32_t)r.prompt.size();
        corun_status st = append(s, r, first[i], lps[i]);
        if (st != CORUN_OK) return st;
    }
    ++s->n_prefill;
    *event = 1;
    return CORUN_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------

extern "C" corun_status corun_sched_create(corun_engine *e, const corun_sched_cfg *cfg, corun_sched **out)
{
    if (!out || !cfg) return sfail(CORUN_E_INVAL, "null argument");
    *out = nullptr;
    corun_sched *s = new corun_sched();
    s->e = e;
    if (e) {
        corun_model_cfg mc{};
        if (corun_engine_info(e, &s->B, &mc, &s->kv) != CORUN_OK) {
            delete s;
            return from_engine(CORUN_E_INVAL);
        }
        s->vocab = mc.vocab;
    } else {
        s->B = cfg->n_slots;
        s->vocab = 1;
        s->kv.layout = cfg->page_size > 0 ? CORUN_KV_PAGED : CORUN_KV_CONTIGUOUS;
        s->kv.n_slots = cfg->n_slots;
        s->kv.max_seq_len = cfg->max_seq_len;
        s->kv.page_size = cfg->page_size;
        s->kv.num_pages = cfg->num_pages;
        s->kv.max_pages_per_seq = cfg->max_pages_per_seq;
    }
    s->paged = s->kv.layout == CORUN_KV_PAGED;
    s->max_num_reqs = cfg->max_num_reqs > 0 ? std::min(cfg->max_num_reqs, s->B) : s->B;
    if (cfg->prefill_chunk < 0) {
        delete s;
        return sfail(CORUN_E_INVAL, "negative prefill_chunk");
    }
    s->chunk = cfg->prefill_chunk;
    if (cfg->prefill_batch_tokens < 0 || (cfg->prefill_batch_tokens > 0 && cfg->prefill_chunk > 0)) {
        delete s;
        return sfail(CORUN_E_INVAL, "prefill_batch_tokens must be >= 0 and excludes prefill_chunk");
    }
    s->batch_tokens = cfg->prefill_batch_tokens;
    if (s->B <= 0 || (!s->paged && s->kv.max_seq_len <= 0) ||
        (s->paged && (s->kv.page_size <= 0 || s->kv.num_pages <= 0 || s->kv.max_pages_per_seq <= 0))) {
        delete s;
        return sfail(CORUN_E_INVAL, "bad slot or cache description");
    }
    s->slot_owner.assign(s->B, -1);
    if (s->paged)
        for (int32_t p = s->kv.num_pages - 1; p >= 0; --p) s->free_pages.push_back(p);
    if (e && s->paged) {
        // one copy of the device table now; from here on this scheduler
        // writes both, and the engine's checks read the host copy
        s->pt_host.resize((size_t)s->kv.n_slots * s->kv.max_pages_per_seq);
        if (hipMemcpy(s->pt_host.data(), s->kv.page_table, s->pt_host.size() * sizeof(int32_t),
                      hipMemcpyDeviceToHost) != hipSuccess ||
            corun_engine_set_page_table_host(e, s->pt_host.data()) != CORUN_OK) {
            delete s;
            return sfail(CORUN_E_HIP, "page table copy");
        }
    }
    if (e) {
        const size_t brows = s->batch_tokens > 0 ? (size_t)std::min(s->B, CORUN_MAX_PREFILL_BATCH) : 1;
        if (hipMalloc(&s->logits, sizeof(float) * (size_t)s->B * s->vocab) != hipSuccess ||
            hipMalloc(&s->last, sizeof(float) * (size_t)s->vocab) != hipSuccess ||
            hipMalloc(&s->blogits, sizeof(float) * brows * s->vocab) != hipSuccess) {
            corun_sched_destroy(s);
            return sfail(CORUN_E_HIP, "logits buffers");
        }
    }
    *out = s;
    return CORUN_OK;
}

extern "C" void corun_sched_destroy(corun_sched *s)
{
    if (!s) return;
    if (s->e && !s->pt_host.empty()) (void)corun_engine_set_page_table_host(s->e, nullptr);   // the engine may outlive it
    if (s->logits) (void)hipFree(s->logits);
    if (s->last) (void)hipFree(s->last);
    if (s->blogits) (void)hipFree(s->blogits);
    delete s;
}

extern "C" corun_status corun_sched_add_request(corun_sched *s, int64_t id, const int32_t *prompt, int32_t prompt_len,
                                                int32_t max_new_tokens, uint64_t seed, float temperature)
{
    if (!s || !prompt) return sfail(CORUN_E_INVAL, "null argument");
    if (prompt_len < 1 || max_new_tokens < 1) return sfail(CORUN_E_INVAL, "empty prompt or output");
    if (s->reqs.count(id)) return sfail(CORUN_E_INVAL, "request id %lld already used", (long long)id);
    if (std::isnan(temperature) || std::isinf(temperature)) return sfail(CORUN_E_INVAL, "temperature not finite");
    Request r;
    r.id = id;
    r.prompt.assign(prompt, prompt + prompt_len);
    r.max_new = max_new_tokens;
    r.seed = seed;
    r.temperature = temperature;
    // a request that could never fit would block the waiting queue's head forever
    const int64_t total = (int64_t)prompt_len + max_new_tokens;
    if (!s->paged && total > s->kv.max_seq_len)
        return sfail(CORUN_E_CAPACITY, "prompt + output %lld exceeds the slot capacity %d", (long long)total,
                     s->kv.max_seq_len);
    if (s->paged && pages_for(s, r) > std::min(s->kv.max_pages_per_seq, s->kv.num_pages))
        return sfail(CORUN_E_CAPACITY, "prompt + output needs %d pages", pages_for(s, r));
    s->reqs.emplace(id, std::move(r));
    s->waiting.push_back(id);
    return CORUN_OK;
}

// Algorithm 2: isolate the request Algorithm 1 selects, else an ordinary
// decode iteration.
extern "C" corun_status corun_sched_step(corun_sched *s, int32_t *event)
{
    if (!s || !event) return sfail(CORUN_E_INVAL, "null argument");
    const int64_t det = find_prefill_request(s);
    corun_status st;
    if (det < 0) {
        st = schedule_origin(s, event);
    } else if (s->batch_tokens > 0 && std::find(s->waiting.begin(), s->waiting.end(), det) != s->waiting.end()) {
        st = run_prefill_batch(s, det, event);
    } else {
        std::deque<int64_t> stashed_running = s->running, stashed_waiting = s->waiting;
        s->waiting.clear();
        if (std::find(s->running.begin(), s->running.end(), det) != s->running.end()) {
            s->running.assign(1, det);
            remove_id(stashed_running, det);
        } else {
            s->running.clear();
            s->waiting.push_back(det);
            remove_id(stashed_waiting, det);
        }
        st = schedule_origin(s, event);
        for (int64_t id : stashed_running) s->running.push_back(id);
        for (int64_t id : stashed_waiting) s->waiting.push_back(id);
    }
    if (st != CORUN_OK) return st;
    retire(s);
    return CORUN_OK;
}

extern "C" corun_status corun_sched_output(const corun_sched *s, int64_t id, int32_t *tokens, float *logprobs,
                                           int32_t cap, int32_t *n_generated, int32_t *finished)
{
    if (!s) return sfail(CORUN_E_INVAL, "null argument");
    auto it = s->reqs.find(id);
    if (it == s->reqs.end()) return sfail(CORUN_E_INVAL, "unknown request %lld", (long long)id);
    const Request &r = it->second;
    const int n = std::min<int>((int)r.tokens.size(), std::max(cap, 0));
    if (tokens) std::copy(r.tokens.begin(), r.tokens.begin() + n, tokens);
    if (logprobs) std::copy(r.logprobs.begin(), r.logprobs.begin() + n, logprobs);
    if (n_generated) *n_generated = (int32_t)r.tokens.size();
    if (finished) *finished = r.finished ? 1 : 0;
    return CORUN_OK;
}

extern "C" corun_status corun_sched_state(const corun_sched *s, int32_t *n_running, int32_t *n_waiting,
                                          int32_t *free_slots, int32_t *free_pages, int64_t *slot_owner)
{
    if (!s) return sfail(CORUN_E_INVAL, "null argument");
    if (n_running) *n_running = (int32_t)s->running.size();
    if (n_waiting) *n_waiting = (int32_t)s->waiting.size();
    if (free_slots) *free_slots = (int32_t)std::count(s->slot_owner.begin(), s->slot_owner.end(), (int64_t)-1);
    if (free_pages) *free_pages = (int32_t)s->free_pages.size();
    if (slot_owner) std::copy(s->slot_owner.begin(), s->slot_owner.end(), slot_owner);
    return CORUN_OK;
}

extern "C" const char *corun_sched_last_error(void) { return s_error.c_str(); }
