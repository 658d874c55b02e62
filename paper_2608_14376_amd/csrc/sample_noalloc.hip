// sample_noalloc.hip -- corun_sample_noalloc: the request-bound seeded
// sampler of corun_sample without an engine and without allocating.
//
// corun_sample stages its per-row inputs (seeds, positions, temperatures,
// valid flags) and outputs (tokens, log-probabilities) in device memory the
// engine allocated at creation.  This variant stages them in `scratch`, a
// fixed array of device memory that the code object carries: each GPU the
// library runs on holds one copy for the life of the process.  The entry
// point makes no hipMalloc / hipFree call and calls nothing that allocates,
// so a caller that must not allocate device memory (a tight serving loop, a
// harness that forbids it) can sample from its own logits buffer.
//
// Every call on a GPU shares that GPU's scratch: calls that overlap on one
// device (two host threads, or two streams in flight at once) race.  A call
// is complete when it returns (it waits for its stream), so calls made one
// after another from one thread never overlap.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "corun.h"
#include "kernels.h"

namespace corun {
corun_status set_error(corun_status s, const char *msg);
}

namespace {

// Staging layout for up to CORUN_SAMPLE_NOALLOC_MAX_ROWS rows, each array
// 256-byte aligned: seeds u64, positions i32, temperatures f32, tokens i32,
// log-probabilities f32, valid flags u8.
constexpr int kRows = CORUN_SAMPLE_NOALLOC_MAX_ROWS;
constexpr size_t kSeedOff = 0;
constexpr size_t kPosOff = kSeedOff + 8 * (size_t)kRows;
constexpr size_t kTempOff = kPosOff + 4 * (size_t)kRows;
constexpr size_t kTokOff = kTempOff + 4 * (size_t)kRows;
constexpr size_t kLpOff = kTokOff + 4 * (size_t)kRows;
constexpr size_t kValidOff = kLpOff + 4 * (size_t)kRows;
constexpr size_t kScratchBytes = (kValidOff + (size_t)kRows + 255) / 256 * 256;
static_assert(kRows % 64 == 0, "each staging array stays 256-byte aligned");

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// The device address of `scratch` on each GPU, looked up once per device
// with that device current.  In host code the array's own name is only a
// host-side handle; every use below goes through these addresses.
constexpr int kMaxDevices = 64;
std::mutex g_mu;
unsigned char *g_scratch[kMaxDevices] = {};

corun_status scratch_of_current_device(unsigned char **out)
{
    int dev = -1;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) {
        char buf[160];
        snprintf(buf, sizeof buf, "hipGetDevice: %s", hipGetErrorString(err));
        return corun::set_error(CORUN_E_HIP, buf);
    }
    if (dev < 0 || dev >= kMaxDevices) return corun::set_error(CORUN_E_HIP, "device index beyond 64");
    std::lock_guard<std::mutex> lock(g_mu);
    if (g_scratch[dev] == nullptr) {
        void *p = nullptr;
        err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (err != hipSuccess || p == nullptr) {
            char buf[160];
            snprintf(buf, sizeof buf, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(err));
            return corun::set_error(CORUN_E_HIP, buf);
        }
        g_scratch[dev] = static_cast<unsigned char *>(p);
    }
    *out = g_scratch[dev];
    return CORUN_OK;
}

}  // namespace

#define NA_HIP(expr)                                                                         \
    do {                                                                                     \
        hipError_t e_ = (expr);                                                              \
        if (e_ != hipSuccess) {                                                              \
            char buf_[256];                                                                  \
            snprintf(buf_, sizeof buf_, "%s: %s", #expr, hipGetErrorString(e_));             \
            return corun::set_error(CORUN_E_HIP, buf_);                                      \
        }                                                                                    \
    } while (0)

extern "C" corun_status corun_sample_noalloc(const float *logits_dev, int64_t ld, int32_t rows, int32_t vocab,
                                             const uint8_t *valid, const int32_t *positions, const uint64_t *seeds,
                                             const float *temperature, int32_t *tokens_out, float *logprobs_out,
                                             void *stream)
{
    if (!logits_dev || !valid || !positions || !seeds || !temperature || !tokens_out)
        return corun::set_error(CORUN_E_INVAL, "null argument");
    if (rows < 1 || rows > kRows) {
        char buf[128];
        snprintf(buf, sizeof buf, "rows %d outside [1, %d] (the static staging's size)", rows, kRows);
        return corun::set_error(CORUN_E_SHAPE, buf);
    }
    if (vocab < 1) return corun::set_error(CORUN_E_SHAPE, "vocab must be >= 1");
    if (ld < vocab) return corun::set_error(CORUN_E_SHAPE, "row stride below the vocabulary");
    for (int r = 0; r < rows; ++r) {
        if (!valid[r]) continue;
        if (positions[r] < 0) return corun::set_error(CORUN_E_INVAL, "negative position of a valid row");
        if (std::isnan(temperature[r]) || std::isinf(temperature[r]))
            return corun::set_error(CORUN_E_INVAL, "temperature of a valid row is not finite");
    }
    unsigned char *s = nullptr;
    corun_status st = scratch_of_current_device(&s);
    if (st != CORUN_OK) return st;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    uint64_t *d_seed = reinterpret_cast<uint64_t *>(s + kSeedOff);
    int32_t *d_pos = reinterpret_cast<int32_t *>(s + kPosOff);
    float *d_temp = reinterpret_cast<float *>(s + kTempOff);
    int32_t *d_tok = reinterpret_cast<int32_t *>(s + kTokOff);
    float *d_lp = reinterpret_cast<float *>(s + kLpOff);
    uint8_t *d_valid = s + kValidOff;
    // every array the kernel reads is written here for all `rows` rows, so
    // nothing a previous call left in the scratch is read
    NA_HIP(hipMemcpyAsync(d_seed, seeds, sizeof(uint64_t) * rows, hipMemcpyHostToDevice, hs));
    NA_HIP(hipMemcpyAsync(d_pos, positions, sizeof(int32_t) * rows, hipMemcpyHostToDevice, hs));
    NA_HIP(hipMemcpyAsync(d_temp, temperature, sizeof(float) * rows, hipMemcpyHostToDevice, hs));
    NA_HIP(hipMemcpyAsync(d_valid, valid, rows, hipMemcpyHostToDevice, hs));
    NA_HIP(corun::launch_sample(logits_dev, ld, rows, vocab, d_valid, d_pos, d_seed, d_temp, d_tok, d_lp, hs));
    NA_HIP(hipMemcpyAsync(tokens_out, d_tok, sizeof(int32_t) * rows, hipMemcpyDeviceToHost, hs));
    if (logprobs_out) NA_HIP(hipMemcpyAsync(logprobs_out, d_lp, sizeof(float) * rows, hipMemcpyDeviceToHost, hs));
    NA_HIP(hipStreamSynchronize(hs));
    return CORUN_OK;
}
