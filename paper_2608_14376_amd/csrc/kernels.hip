// kernels.hip -- gfx950 (CDNA4) kernels of the padded, position-invariant
// decode step and the isolated prefill.
//
// Position invariance (Sec. III, Definition 2) is the only property the
// method needs from a kernel: at a fixed launch shape, a row's arithmetic --
// which values are combined, in which order, in which precision -- may not
// depend on the row's index or on any other row's data.  Every kernel here
// gets it the same way:
//   * the launch geometry and every loop bound derive from sizes fixed when
//     the engine is created (B, model shape, cache capacity), never from the
//     number of live rows;
//   * each row's reductions run in one fixed order: sequential loops,
//     a fixed butterfly across the 64 lanes of one wavefront, and split
//     partials combined in split-index order -- no floating-point atomics;
//   * request-local metadata (a row's own length and pages) may change how
//     much work that row does (Sec. III: metadata belongs to the row), but
//     never how another row is computed.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>

#include "kernels.h"

namespace corun {

// Launch timing (corun_profile_step): while a recorder is set on the calling
// thread, every launch below records a pair of events around the kernel's
// own execution (hipExtLaunchKernel) and lists them in the recorder.
namespace {
thread_local LaunchRecorder *t_rec = nullptr;

void launch_events(hipEvent_t *start, hipEvent_t *stop)
{
    *start = *stop = nullptr;
    LaunchRecorder *r = t_rec;
    if (r == nullptr) return;
    while (r->used + 2 > r->pool.size()) {
        hipEvent_t ev;
        if (hipEventCreate(&ev) != hipSuccess) return;   // untimed launch; the recorder notes nothing
        r->pool.push_back(ev);
    }
    *start = r->pool[r->used];
    *stop = r->pool[r->used + 1];
    r->used += 2;
    r->launches.push_back({*start, *stop});
}
}  // namespace

void set_launch_recorder(LaunchRecorder *r) { t_rec = r; }

#define KLAUNCH(kernel, grid, block, shmem, stream, ...)                                                   \
    do {                                                                                                    \
        hipEvent_t ks_, ke_;                                                                                \
        launch_events(&ks_, &ke_);                                                                          \
        if (ks_ != nullptr)                                                                                 \
            hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, ks_, ke_, 0, __VA_ARGS__);            \
        else                                                                                                \
            hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);                            \
    } while (0)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 -> bf16, round to nearest even, NaN quieted: gfx950's v_cvt_pk_bf16_f32
// (bit-identical, over all 2^32 inputs, to adding 0x7fff + lsb and truncating,
// with (u >> 16) | 0x40 for NaN)
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
// two values in one instruction: a in the low half, b in the high half
__device__ __forceinline__ uint32_t f2bf2(float a, float b)
{
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

// SwiGLU of one feature from its fp32 gate and up sums: both rounded to
// bf16 (the projection's output precision), silu(g) u rounded to bf16.  The
// SwiGLU kernel and the gate/up projection's fused epilogue share it, so the
// two paths agree bit for bit.
__device__ __forceinline__ uint16_t swiglu_bf16(float gs, float us)
{
    const float g = bf2f(f2bf(gs));
    const float u = bf2f(f2bf(us));
    const float silu = g / (1.0f + __expf(-g));
    return f2bf(silu * u);
}

__device__ __forceinline__ float wave_max(float v)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    return v;
}

__device__ __forceinline__ size_t kv_offset(const KvView &kv, int nkv, int d, int slot, int kvh, int t)
{
    if (kv.layout == 1) {
        int page = kv.page_table[(size_t)slot * kv.max_pages_per_seq + t / kv.page_size];
        return (((size_t)page * nkv + kvh) * kv.page_size + (t % kv.page_size)) * d;
    }
    return (((size_t)slot * nkv + kvh) * kv.max_seq_len + t) * d;
}

// Values are stored like keys, by token: element e of token t of a kv head
// is element e of that token's value row.
__device__ __forceinline__ size_t v_offset(const KvView &kv, int nkv, int d, int slot, int kvh, int t, int e)
{
    return kv_offset(kv, nkv, d, slot, kvh, t) + e;
}

// Transposed LDS read (gfx950 ds_read_b64_tr_b16).  Within each group of 16
// lanes, lane a + 4 q supplies the address of four 16-bit values (row q,
// elements 4 a .. 4 a + 3 of some column block); lane i of the group then
// receives element i of the block from rows 0..3.  Two such reads give a
// lane eight consecutive rows of one column: the B (or A) operand of a bf16
// MFMA whose K runs along the rows, read from row-major tiles.
typedef short s16x4_tr __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint2 lds_read_tr16(const void *lds_ptr)
{
    typedef __attribute__((address_space(3))) s16x4_tr lds_s16x4;
    const s16x4_tr v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_s16x4 *)(const __attribute__((address_space(3))) void *)lds_ptr);
    return __builtin_bit_cast(uint2, v);
}

// Value tiles in LDS are token-major, 16-byte chunk c of token t (KCH
// chunks per token) at t KCH + (c ^ vtile_swz<KCH>(t)).  A transposed read
// of the attention kernels takes, per 16-lane group, 32 bytes (two chunks)
// of four consecutive tokens 4 r + 0..3, and the two groups of a half
// wavefront read either the next two chunks of the same tokens or the same
// chunks of the tokens 8 further on.  The swizzle moves the four tokens to
// four distinct 16-bank ranges (bits 2-3 of the chunk, with the token's
// parity for 128-byte rows) and those 8 tokens further to the other half of
// each range (bit 1), so the 64 lanes of a half wavefront pair touch each
// of the 64 banks once.
template <int KCH>
__device__ __forceinline__ int vtile_swz(int t)
{
    static_assert(KCH == 8 || KCH == 16, "128- or 256-byte value rows");
    if constexpr (KCH == 16) return (4 * (t & 3)) ^ (2 * ((t >> 3) & 1));
    else return (4 * ((t >> 1) & 1)) ^ (2 * ((t >> 3) & 1));
}

__device__ __forceinline__ int row_slot(const int32_t *slot_of_row, int slot_const, int r)
{
    return slot_of_row ? slot_of_row[r] : (slot_const >= 0 ? slot_const : r);
}

// (value, index) under "larger value, then smaller index" is a total order:
// any tree of these comparisons selects the first index of the maximum.
__device__ __forceinline__ void better(float &v, int &i, float v2, int i2)
{
    if (v2 > v || (v2 == v && i2 < i)) {
        v = v2;
        i = i2;
    }
}

// ---------------------------------------------------------------------------
// Fixed reduction trees on the cross-lane hardware.
//
// dpp_f<CTRL>: lane i takes the value of the lane CTRL selects (a DPP move).
// row16_sum: the sum over the 16 lanes of a DPP row -- pairs i ^ 1, then
// i ^ 2 (quad permutes), then i and 7 - i within eight lanes (half-row
// mirror), then i and 15 - i (row mirror).  wave_sum_dpp: row16_sum, then
// the two rows of each 32-lane half (ds_swizzle, i ^ 16), then lane 0 plus
// lane 32.  At every stage a lane and its partner add the same two values
// (addition commutes), so every lane ends with the same bits.
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ float row16_sum(float v)
{
    v += dpp_f<0xB1>(v);    // quad_perm [1, 0, 3, 2]: lane i ^ 1
    v += dpp_f<0x4E>(v);    // quad_perm [2, 3, 0, 1]: lane i ^ 2
    v += dpp_f<0x141>(v);   // row_half_mirror: lane 7 - i of its eight
    v += dpp_f<0x140>(v);   // row_mirror: lane 15 - i of its sixteen
    return v;
}

__device__ __forceinline__ float wave_sum_dpp(float v)
{
    v = row16_sum(v);
    // bit-mask swizzle within 32 lanes: and 0x1f, or 0, xor 0x10
    v += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x401F));
    const float lo = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
    const float hi = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
    return lo + hi;
}

// ---------------------------------------------------------------------------
// Embedding gather
// ---------------------------------------------------------------------------
// Grid: rows x ceil(H / 256) blocks, flattened into x (rows may exceed the
// 65535 limit of the other grid dimensions in a long prefill).  With ss
// (H a multiple of 256) it also writes each row's sums of squares over
// 16-column groups, ss[b][i / 16], for the small-batch projections' norm.
__global__ void k_embed(const uint16_t *__restrict__ E, const int32_t *__restrict__ tokens,
                        const uint8_t *__restrict__ valid, int H, float *__restrict__ x, float *__restrict__ ss)
{
    const int nb = (H + 255) / 256;
    const int b = blockIdx.x / nb;
    const int i = (blockIdx.x % nb) * 256 + threadIdx.x;
    const int tok = (valid == nullptr || valid[b]) ? tokens[b] : 0;
    const float v = i < H ? bf2f(E[(size_t)tok * H + i]) : 0.f;
    if (i < H) x[(size_t)b * H + i] = v;
    if (ss != nullptr) {
        const float sq = row16_sum(v * v);            // lanes 16 k .. 16 k + 15: one 16-column group
        if ((threadIdx.x & 15) == 0 && i < H) ss[(size_t)b * (H / 16) + i / 16] = sq;
    }
}

hipError_t launch_embed(const uint16_t *E, const int32_t *tokens, const uint8_t *valid, int rows, int H,
                        float *x, hipStream_t st, float *ss)
{
    if (ss != nullptr && H % 256 != 0) return hipErrorInvalidValue;
    const long long blocks = (long long)rows * ((H + 255) / 256);
    KLAUNCH(k_embed, dim3((unsigned)blocks), dim3(256), 0, st, E, tokens, valid, H, x, ss);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// RMSNorm with the residual add of the previous projection's split partials
// folded in.  One workgroup of min(H/4, 1024) threads per row; thread j owns
// the float4 groups 4 (j + nth i), kept in registers (H <= 8192).  Each
// element adds its partials in split order; the sum of squares runs
// sequentially per thread, then through a fixed tree: each wavefront's DPP /
// ds_swizzle tree (wave_sum_dpp), then the wavefront sums in wavefront order.
// A row spans up to 16 wavefronts because the fold reads the split-K
// partials too ((S + 2) x 16 KB per row of 4096): one wavefront per row,
// built and measured, took 16.3 against 6.2 us at B = 256 (64 workgroups of
// four single-row wavefronts), too few loads in flight per row.
// ---------------------------------------------------------------------------
// Fixed-order sum over a block of nw wavefronts: each wavefront's DPP tree,
// then the wavefront sums added in wavefront order.
__device__ __forceinline__ float block_sum(float v, float *red, int nw)
{
    v = wave_sum_dpp(v);
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[w] = v;
    __syncthreads();
    float t = red[0];
    for (int i = 1; i < nw; ++i) t += red[i];
    return t;
}

template <int NG>
__global__ __launch_bounds__(1024) void k_rmsnorm(float *__restrict__ x, const float *__restrict__ part,
                                                  int S, long long part_stride, int rows, int H,
                                                  const uint16_t *__restrict__ g, float eps,
                                                  uint16_t *__restrict__ h, MoeFold mf)
{
    __shared__ float red[16];
    const int row = blockIdx.x;
    const int nth = blockDim.x;
    float *xr = x + (size_t)row * H;
    const float *pr = part + (size_t)row * H;
    float4 v[NG];
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < NG; ++j) {
        const int i = 4 * (threadIdx.x + nth * j);
        if (i < H) {
            v[j] = *(const float4 *)(xr + i);
            // partials are added in split order; their loads are issued in
            // batches of 8 ahead of the adds
            int s = 0;
            for (; s + 8 <= S; s += 8) {
                float4 p[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) p[u] = *(const float4 *)(pr + (s + u) * part_stride + i);
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    v[j].x += p[u].x; v[j].y += p[u].y; v[j].z += p[u].z; v[j].w += p[u].w;
                }
            }
            for (; s < S; ++s) {
                const float4 p = *(const float4 *)(pr + s * part_stride + i);
                v[j].x += p.x; v[j].y += p.y; v[j].z += p.z; v[j].w += p.w;
            }
            if (mf.y != nullptr && (mf.valid == nullptr || mf.valid[row])) {
                // mixture-of-experts combine: sum_r w_r y_r in rank order, then added
                float4 c = {0.f, 0.f, 0.f, 0.f};
                for (int rk = 0; rk < mf.top_k; ++rk) {
                    const float w = mf.w[(size_t)row * mf.top_k + rk];
                    const float4 y = *(const float4 *)(mf.y + ((size_t)row * mf.top_k + rk) * H + i);
                    c.x += w * y.x; c.y += w * y.y; c.z += w * y.z; c.w += w * y.w;
                }
                v[j].x += c.x; v[j].y += c.y; v[j].z += c.z; v[j].w += c.w;
            }
            if (S > 0 || mf.y != nullptr) *(float4 *)(xr + i) = v[j];
            ss += v[j].x * v[j].x;
            ss += v[j].y * v[j].y;
            ss += v[j].z * v[j].z;
            ss += v[j].w * v[j].w;
        }
    }
    ss = block_sum(ss, red, nth >> 6);
    const float rstd = 1.0f / sqrtf(ss / (float)H + eps);
    uint16_t *hr = h + (size_t)row * H;
#pragma unroll
    for (int j = 0; j < NG; ++j) {
        const int i = 4 * (threadIdx.x + nth * j);
        if (i < H) {
            const ushort4 gg = *(const ushort4 *)(g + i);
            ushort4 o;
            o.x = f2bf(v[j].x * rstd * bf2f(gg.x));
            o.y = f2bf(v[j].y * rstd * bf2f(gg.y));
            o.z = f2bf(v[j].z * rstd * bf2f(gg.z));
            o.w = f2bf(v[j].w * rstd * bf2f(gg.w));
            *(ushort4 *)(hr + i) = o;
        }
    }
}

hipError_t launch_rmsnorm(float *x, const float *part, int S, long long part_stride, int rows, int H,
                          const uint16_t *g, float eps, uint16_t *h, hipStream_t st, MoeFold mf)
{
    if (H % 256 || H > 8192) return hipErrorInvalidValue;
    const int groups = H / 4;
    const int nth = groups >= 1024 ? 1024 : groups;        // multiple of 64
    if (groups <= nth)
        KLAUNCH((k_rmsnorm<1>), dim3(rows), dim3(nth), 0, st, x, part, S, part_stride, rows, H, g, eps, h,
                           mf);
    else
        KLAUNCH((k_rmsnorm<2>), dim3(rows), dim3(nth), 0, st, x, part, S, part_stride, rows, H, g, eps, h,
                           mf);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Projection y = A W^T on bf16 MFMA (v_mfma_f32_16x16x32_bf16), fp32
// accumulate, split-K partials.
//
// A wavefront owns MT row tiles x NT column tiles of 16x16 and one K chunk.
// Lane l supplies row (l % 16) of each operand tile and the 8 consecutive K
// elements 8 (l / 16) .. +7 of every 32-wide K step; A and W use the same
// lane -> K assignment, so each MFMA adds the full 32-term dot product.
// Weights stream straight from HBM into registers (16 bytes per lane per
// load, KU K-steps in flight); activations are small and hit in L1/L2.
// Output lane l holds rows 4 (l / 16) + i, column l % 16 of each tile.
// ---------------------------------------------------------------------------
template <int MT, int NT, int KU>
struct GemmFrags {
    bf16x8 w[NT][KU];
    bf16x8 a[MT][KU];
};

template <int MT, int NT, int KU>
__device__ __forceinline__ void gemm_load(GemmFrags<MT, NT, KU> &f, const uint16_t *const (&wp)[NT],
                                          const uint16_t *const (&ap)[MT], const bool (&arow)[MT], int k)
{
    const uint4 z = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int u = 0; u < KU; ++u) f.w[nt][u] = __builtin_bit_cast(bf16x8, *(const uint4 *)(wp[nt] + k + 32 * u));
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int u = 0; u < KU; ++u)
        {
            uint4 v = z;
            if (arow[mt]) v = *(const uint4 *)(ap[mt] + k + 32 * u);
            f.a[mt][u] = __builtin_bit_cast(bf16x8, v);
        }
}

template <int MT, int NT, int KU>
__device__ __forceinline__ void gemm_mma(const GemmFrags<MT, NT, KU> &f, f32x4 (&acc)[MT][NT])
{
#pragma unroll
    for (int u = 0; u < KU; ++u)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.a[mt][u], f.w[nt][u], acc[mt][nt], 0, 0, 0);
}

template <int MT, int NT, int KU>
__global__ __launch_bounds__(256) void k_gemm(const uint16_t *__restrict__ A, int lda,
                                              const uint16_t *__restrict__ W, int M, int N, int K, int Kc,
                                              float *__restrict__ out, long long split_stride, int ldo,
                                              ArgBest *__restrict__ amax)
{
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int r = lane & 15, kg = lane >> 4;
    const int ncb = (N + 16 * NT - 1) / (16 * NT);
    const int cb = blockIdx.x * 4 + wave;
    if (cb >= ncb) return;
    const int s = blockIdx.y;
    const int m0 = blockIdx.z * 16 * MT;
    const int kbeg = s * Kc;
    const int kend = min(K, kbeg + Kc);
    const int n0 = cb * 16 * NT;
    const int nvalid = min(NT, (N - n0) / 16);

    const uint16_t *wp[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
        wp[nt] = W + (size_t)(n0 + 16 * min(nt, nvalid - 1) + r) * K + kg * 8;
    const uint16_t *ap[MT];
    bool arow[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        ap[mt] = A + (size_t)(m0 + 16 * mt + r) * lda + kg * 8;
        arow[mt] = (m0 + 16 * mt + r) < M;   // rows past M contribute zeros and are never stored
    }

    f32x4 acc[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = (f32x4){0.f, 0.f, 0.f, 0.f};

    // Main loop, software-pipelined two deep: the next batch of KU K-steps is
    // in flight while the current one feeds the MFMAs.
    constexpr int STEP = 32 * KU;
    const int nfull = (kend - kbeg) / STEP;
    int k = kbeg;
    GemmFrags<MT, NT, KU> f0, f1;
    if (nfull > 0) gemm_load(f0, wp, ap, arow, k);
    for (int it = 0; it < nfull; it += 2) {
        if (it + 1 < nfull) gemm_load(f1, wp, ap, arow, k + STEP);
        gemm_mma(f0, acc);
        if (it + 2 < nfull) gemm_load(f0, wp, ap, arow, k + 2 * STEP);
        if (it + 1 < nfull) gemm_mma(f1, acc);
        k += 2 * STEP;
    }
    k = kbeg + nfull * STEP;
    for (; k < kend; k += 32) {   // K tail, one 32-step at a time; K % 8 == 0
        const bool in = (k + kg * 8) < kend;
        const uint4 z = {0u, 0u, 0u, 0u};
        bf16x8 wf[NT], af[MT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
        {
            uint4 v = z;
            if (in) v = *(const uint4 *)(wp[nt] + k);
            wf[nt] = __builtin_bit_cast(bf16x8, v);
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
        {
            uint4 v = z;
            if (in && arow[mt]) v = *(const uint4 *)(ap[mt] + k);
            af[mt] = __builtin_bit_cast(bf16x8, v);
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[mt], wf[nt], acc[mt][nt], 0, 0, 0);
    }

    float *o = out + (size_t)s * split_stride;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            if (nt >= nvalid) continue;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = m0 + 16 * mt + kg * 4 + i;
                if (row < M) o[(size_t)row * ldo + n0 + 16 * nt + r] = acc[mt][nt][i];
            }
        }
    if (amax != nullptr) {
        // per row: best (value, column) over this wavefront's columns -- an
        // exact selection under the "larger value, then smaller index" order
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float bv = -INFINITY;
                int bi = 0x7fffffff;
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
                    if (nt < nvalid) better(bv, bi, acc[mt][nt][i], n0 + 16 * nt + r);
#pragma unroll
                for (int off = 1; off < 16; off <<= 1) {
                    const float v2 = __shfl_xor(bv, off, 64);
                    const int i2 = __shfl_xor(bi, off, 64);
                    better(bv, bi, v2, i2);
                }
                const int row = m0 + 16 * mt + kg * 4 + i;
                if (r == 0 && row < M) amax[(size_t)row * ncb + cb] = ArgBest{bv, bi};
            }
    }
}

// ---------------------------------------------------------------------------
// Large-M projection (decode at B >= 64, prefill): LDS-tiled bf16 MFMA.
//
// Workgroup tile BM x BN, K in steps of 64, four wavefronts in a
// WAVES_M x WAVES_N grid, each owning (BM/WAVES_M) x (BN/WAVES_N) of the tile
// as 16x16 MFMA tiles.  Each K step stages A[BM][64] and W[BN][64] in LDS
// (two stages: the next step's global loads are in flight while the current
// stage feeds the MFMAs).  LDS rows are padded to 72 elements (144 bytes) so
// the 16 rows read by one 16-lane group fall on disjoint banks.  Each weight
// element is read from HBM once per M tile; at BM >= M (decode), exactly
// once.  Every output element's K reduction runs in the same order: K steps
// in order, each the MFMA's fixed 32-term dot product chained in order.
// ---------------------------------------------------------------------------
template <int BM, int BN, int WAVES_M>
__global__ __launch_bounds__(256) void k_gemm_tiled(const uint16_t *__restrict__ A, int lda,
                                                    const uint16_t *__restrict__ W, int M, int N, int K, int Kc,
                                                    float *__restrict__ out, long long split_stride, int ldo,
                                                    ArgBest *__restrict__ amax)
{
    constexpr int BK = 64, LDR = 72;
    constexpr int WAVES_N = 4 / WAVES_M;
    constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    constexpr int FM = WM / 16, FN = WN / 16;
    constexpr int A_LD = BM / 32, W_LD = BN / 32;     // 16-byte loads per thread per stage
    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDR];
    __shared__ __attribute__((aligned(16))) uint16_t Ws[2][BN * LDR];

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int num_m = (M + BM - 1) / BM;
    const int mt = blockIdx.x % num_m, ntile = blockIdx.x / num_m;
    const int m0 = mt * BM, n0 = ntile * BN;
    const int s = blockIdx.y;
    const int kbeg = s * Kc, kend = min(K, kbeg + Kc);
    const int wm0 = (wave / WAVES_N) * WM, wn0 = (wave % WAVES_N) * WN;
    const int r16 = lane & 15, kg = lane >> 4;

    // global -> register staging: thread t covers rows t/8 + 32 i, 16 bytes at column (t % 8) * 8
    const int lrow = tid >> 3, lcol = (tid & 7) * 8;
    // staging held in vector values (not arrays), so it stays in VGPRs
    typedef unsigned int stageA_t __attribute__((ext_vector_type(4 * A_LD)));
    typedef unsigned int stageW_t __attribute__((ext_vector_type(4 * W_LD)));
    stageA_t ra;
    stageW_t rw;
#define CORUN_TILED_GLOAD(k0_)                                                                  \
    do {                                                                                        \
        const uint4 z_ = {0u, 0u, 0u, 0u};                                                      \
        const bool kin_ = ((k0_) + lcol) < kend;                                                \
        _Pragma("unroll") for (int i_ = 0; i_ < A_LD; ++i_) {                                   \
            const int row_ = m0 + lrow + 32 * i_;                                               \
            uint4 v_ = z_;                                                                      \
            if (kin_ && row_ < M) v_ = *(const uint4 *)(A + (size_t)row_ * lda + (k0_) + lcol); \
            ra[4 * i_ + 0] = v_.x; ra[4 * i_ + 1] = v_.y; ra[4 * i_ + 2] = v_.z; ra[4 * i_ + 3] = v_.w; \
        }                                                                                       \
        _Pragma("unroll") for (int i_ = 0; i_ < W_LD; ++i_) {                                   \
            const int row_ = n0 + lrow + 32 * i_;                                               \
            uint4 v_ = z_;                                                                      \
            if (kin_ && row_ < N) v_ = *(const uint4 *)(W + (size_t)row_ * K + (k0_) + lcol);  \
            rw[4 * i_ + 0] = v_.x; rw[4 * i_ + 1] = v_.y; rw[4 * i_ + 2] = v_.z; rw[4 * i_ + 3] = v_.w; \
        }                                                                                       \
    } while (0)
#define CORUN_TILED_SSTORE(st_)                                                                 \
    do {                                                                                        \
        _Pragma("unroll") for (int i_ = 0; i_ < A_LD; ++i_)                                     \
            *(uint4 *)(&As[st_][(lrow + 32 * i_) * LDR + lcol]) =                               \
                (uint4){ra[4 * i_], ra[4 * i_ + 1], ra[4 * i_ + 2], ra[4 * i_ + 3]};            \
        _Pragma("unroll") for (int i_ = 0; i_ < W_LD; ++i_)                                     \
            *(uint4 *)(&Ws[st_][(lrow + 32 * i_) * LDR + lcol]) =                               \
                (uint4){rw[4 * i_], rw[4 * i_ + 1], rw[4 * i_ + 2], rw[4 * i_ + 3]};            \
    } while (0)

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = (f32x4){0.f, 0.f, 0.f, 0.f};

    int cur = 0;
    if (kbeg < kend) {
        CORUN_TILED_GLOAD(kbeg);
        CORUN_TILED_SSTORE(0);
    }
    __syncthreads();
    for (int k0 = kbeg; k0 < kend; k0 += BK) {
        const bool has_next = k0 + BK < kend;
        if (has_next) CORUN_TILED_GLOAD(k0 + BK);
#pragma unroll
        for (int kk = 0; kk < BK / 32; ++kk) {
            bf16x8 af[FM], wf[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i)
                af[i] = *(const bf16x8 *)(&As[cur][(wm0 + 16 * i + r16) * LDR + kk * 32 + kg * 8]);
#pragma unroll
            for (int j = 0; j < FN; ++j)
                wf[j] = *(const bf16x8 *)(&Ws[cur][(wn0 + 16 * j + r16) * LDR + kk * 32 + kg * 8]);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], wf[j], acc[i][j], 0, 0, 0);
        }
        if (has_next) {
            if (cur) CORUN_TILED_SSTORE(0);
            else CORUN_TILED_SSTORE(1);
        }
        __syncthreads();
        cur ^= 1;
    }
#undef CORUN_TILED_GLOAD
#undef CORUN_TILED_SSTORE

    float *o = out + (size_t)s * split_stride;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int col = n0 + wn0 + 16 * j + r16;
            if (col >= N) continue;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int row = m0 + wm0 + 16 * i + kg * 4 + q;
                if (row < M) o[(size_t)row * ldo + col] = acc[i][j][q];
            }
        }
    if constexpr (WN == 64) {
        if (amax != nullptr) {   // per row: best over this wavefront's 64 columns (one 64-column block)
            const int ncb = (N + 63) / 64;
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float bv = -INFINITY;
                    int bi = 0x7fffffff;
#pragma unroll
                    for (int j = 0; j < FN; ++j) {
                        const int col = n0 + wn0 + 16 * j + r16;
                        if (col < N) better(bv, bi, acc[i][j][q], col);
                    }
#pragma unroll
                    for (int off = 1; off < 16; off <<= 1) {
                        const float v2 = __shfl_xor(bv, off, 64);
                        const int i2 = __shfl_xor(bi, off, 64);
                        better(bv, bi, v2, i2);
                    }
                    const int row = m0 + wm0 + 16 * i + kg * 4 + q;
                    if (r16 == 0 && row < M && n0 + wn0 < N) amax[(size_t)row * ncb + (n0 + wn0) / 64] = ArgBest{bv, bi};
                }
        }
    }
}

// ---------------------------------------------------------------------------
// Large-M projection, pipelined: both operands stream global -> LDS with the
// direct 16-byte LDS loads of gfx950 (no register staging) through a ring of
// NST stages of BK (32 or 64) K elements: while the matrix cores run stage i
// from registers, stage i + 1 is read from LDS and NST - 1 stages are in
// flight.  The loads of a stage are the only vector-memory
// operations of the loop, so "stage i has landed" is a fixed vmcnt: the
// number of loads issued after it.
//
// Stage layout: A rows [BM][BK] then W rows [BN][BK], each row as BK / 8
// 16-byte chunks, chunk c of row r stored at c ^ f(r) (f(r) = (r / 4) % 4 for
// 64-byte rows, (r / 2) % 8 for 128-byte rows), which puts the 16 rows read
// by one 16-lane group of a fragment read on 16 distinct bank groups.  One
// load instruction of a wavefront fills 1 KB of the stage: 16 rows x 64
// bytes or 8 rows x 128 bytes.  Whole 128-byte lines per row and instruction
// matter: the 64-byte form roughly halves what one CU can pull while its
// activation and weight loads share the path.
//
// NW wavefronts in a WGM x (NW / WGM) grid; wavefront tile (BM / WGM) x
// (BN / (NW / WGM)) as 32x32 tiles of v_mfma_f32_32x32x16_bf16.  Every output
// element's K reduction runs in one order (K steps in order, each the
// instruction's fixed 16-term product) whatever its row, so rows stay
// position-invariant.  Rows >= M and columns >= N load clamped (real) rows
// and are never stored; K and the split chunk are multiples of BK, so no
// stage is partial.
//
// Packed weights (PKW, 128 x 64 tiles only): W is the tile-packed copy that
// launch_pack_weights writes, [ceil(N / 128)][K / 64][128][64], each 16 KB
// tile contiguous and rows past N zero.  A workgroup then streams one
// contiguous run of K / 64 tiles instead of 128 rows 2 K bytes apart; the
// same elements meet the same instructions in the same order, so the results
// are bit-identical to the row-major layout.  At small M, where the kernel
// streams weights, this is 5-20% faster.
//
// Tile order: with several M tiles, workgroups are handed to the eight XCDs
// in turn, so each XCD gets a contiguous run of tiles, walked in groups of
// eight M tiles per N tile: the workgroups sharing a weight tile or an
// activation tile run together on one L2.
// ---------------------------------------------------------------------------
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ constexpr int vmcnt_imm(int n)
{
    return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8);   // vmcnt(n), expcnt and lgkmcnt not waited
}

// wait until at most `stages` stages of OPS loads each are outstanding
// (s_waitcnt takes an immediate: dispatch the uniform stage count)
template <int OPS, int S_>
__device__ __forceinline__ void wait_stages(int stages)
{
    if constexpr (S_ >= 0) {
        if (stages == S_) __builtin_amdgcn_s_waitcnt(vmcnt_imm(S_ * OPS));
        else wait_stages<OPS, S_ - 1>(stages);
    }
}

__device__ __forceinline__ void lds_barrier()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <int C>
__device__ __forceinline__ int dma_swz(int r, int c)
{
    static_assert(C == 4 || C == 8, "64- or 128-byte rows");
    if constexpr (C == 4) return r * 4 + (c ^ ((r >> 2) & 3));
    else return r * 8 + (c ^ ((r >> 1) & 7));
}

template <int BM, int BN, int BK, int NST, int WGM, int NW = 4, bool PKW = false, bool SWIGLU = false,
          bool MOE = false>
__global__ __launch_bounds__(64 * NW) void k_gemm_dma(const uint16_t *__restrict__ A, int lda,
                                                  const uint16_t *__restrict__ W, int M, int N, int K, int Kc,
                                                  float *__restrict__ out, long long split_stride, int ldo,
                                                  ArgBest *__restrict__ amax, uint16_t *__restrict__ act,
                                                  ExpertTiles et)
{
    constexpr int C = BK / 8;                         // 16-byte chunks per row
    constexpr int NT = 64 * NW;                       // threads
    constexpr int WGN = NW / WGM;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int FM = WM / 32, FN = WN / 32;
    constexpr int A_OPS = BM * C / NT, W_OPS = BN * C / NT;
    static_assert(A_OPS * NT == BM * C && W_OPS * NT == BN * C, "loads cover the tile");
    constexpr int OPS = A_OPS + W_OPS, P = NST;       // every slot of the ring is a stage in flight
    constexpr int STAGE = (BM + BN) * C;             // 16-byte units
    static_assert(P * OPS <= 63, "vmcnt range");
    static_assert(!PKW || (BN == 128 && BK == 64), "packed weights come in 128 x 64 tiles");
    static_assert(!SWIGLU || (PKW && NW == 2 && WGM == 1), "SwiGLU pairs the two wavefronts' 64 columns");
    static_assert(!MOE || BM >= 16, "an expert tile holds up to 16 assignments");
    __shared__ __attribute__((aligned(16))) uint4 ring[NST * STAGE];

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int num_m = (M + BM - 1) / BM, num_n = (N + BN - 1) / BN;
    int t = blockIdx.x, mt, nt;
    // expert tiles: grid.y walks the tile slots; rows are the slot's
    // assignments, A row = assignment / row_div, output row = assignment
    int row_end = M, slot_start = 0;
    if constexpr (MOE) {
        const int sl = blockIdx.y;
        row_end = et.tiles[3 * sl + 2];
        if (row_end == 0) return;                    // an unused slot (uniform over the workgroup)
        slot_start = et.tiles[3 * sl + 1];
        W += (size_t)et.tiles[3 * sl] * et.w_stride;
        mt = 0;
        nt = t;
    } else if (num_m == 1) {
        mt = 0;
        nt = t;
    } else {
        const int T = num_m * num_n;
        if (T >= 8 && gridDim.y == 1) {
            const int x = t & 7, j = t >> 3, per = T >> 3, rem = T & 7;
            t = x * per + min(x, rem) + j;
        }
        constexpr int GM = 8;
        const int group = t / (GM * num_n), first = group * GM, gs = min(num_m - first, GM);
        const int in = t - group * GM * num_n;
        mt = first + in % gs;
        nt = in / gs;
    }
    const int m0 = mt * BM, n0 = nt * BN;
    const int s = MOE ? 0 : blockIdx.y;
    const int kbeg = s * Kc, kend = min(K, kbeg + Kc);
    const int nk = kend > kbeg ? (kend - kbeg) / BK : 0;
    auto out_row = [&](int row) -> size_t {
        if constexpr (MOE) return (size_t)et.list[slot_start + row];
        else return (size_t)row;
    };

    // per load op j: source row and logical chunk of this thread's 16 bytes
    const uint16_t *asrc[A_OPS];
    const uint16_t *wsrc[W_OPS];
#pragma unroll
    for (int j = 0; j < A_OPS; ++j) {
        const int g = j * NT + tid, r = g / C, c = dma_swz<C>(r, g % C) - r * C;   // the swizzle is an involution
        size_t arow;
        if constexpr (MOE) arow = (size_t)(et.list[slot_start + min(r, row_end - 1)] / et.row_div);
        else arow = (size_t)min(m0 + r, M - 1);
        asrc[j] = A + arow * lda + kbeg + 8 * c;
    }
#pragma unroll
    for (int j = 0; j < W_OPS; ++j) {
        const int g = j * NT + tid, r = g / C, c = dma_swz<C>(r, g % C) - r * C;
        if constexpr (PKW) wsrc[j] = W + ((size_t)nt * (K / BK) + kbeg / BK) * (BN * BK) + r * BK + 8 * c;
        else wsrc[j] = W + (size_t)min(n0 + r, N - 1) * K + kbeg + 8 * c;
    }
    // a stage kofs K elements in: kofs further along a row, or kofs / BK tiles on
    constexpr int WSTEP = PKW ? BN : 1;
    typedef __attribute__((address_space(3))) void lds_void;
    auto issue = [&](int slot, int kofs) {
        uint4 *base = ring + slot * STAGE + wave * 64;
#pragma unroll
        for (int j = 0; j < A_OPS; ++j)
            __builtin_amdgcn_global_load_lds((const void *)(asrc[j] + kofs), (lds_void *)(base + j * NT), 16, 0, 0);
#pragma unroll
        for (int j = 0; j < W_OPS; ++j)
            __builtin_amdgcn_global_load_lds((const void *)(wsrc[j] + (size_t)kofs * WSTEP),
                                             (lds_void *)(base + BM * C + j * NT), 16, 0, 0);
    };

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

    const int wm0 = (wave / WGN) * WM, wn0 = (wave % WGN) * WN;
    const int r32 = lane & 31, h = lane >> 5;
    // a stage's fragments: per 16-wide K step, FM activation and FN weight tiles
    struct Frags {
        bf16x8 a[BK / 16][FM], w[BK / 16][FN];
    };
    auto read = [&](Frags &f, int slot) {
        const uint4 *As = ring + slot * STAGE;
        const uint4 *Ws = As + BM * C;
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
#pragma unroll
            for (int i = 0; i < FM; ++i) f.a[ks][i] = __builtin_bit_cast(bf16x8, As[dma_swz<C>(wm0 + 32 * i + r32, 2 * ks + h)]);
#pragma unroll
            for (int j = 0; j < FN; ++j) f.w[ks][j] = __builtin_bit_cast(bf16x8, Ws[dma_swz<C>(wn0 + 32 * j + r32, 2 * ks + h)]);
        }
    };
    auto mma = [&](const Frags &f) {
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks)
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[ks][i], f.w[ks][j], acc[i][j], 0, 0, 0);
    };
    // Stage i: make stage i + 1 visible, refill stage i's slot with stage
    // i + P, read stage i + 1's fragments into `nxt`, then run stage i's
    // products from `cur` while those reads and P - 1 stages of loads are in
    // flight.  Stage i's fragments were read into registers during step
    // i - 1; each wavefront waits for its LDS reads (lgkmcnt 0) before the
    // barrier, so no read of the slot is pending when its refill is issued.
    auto step = [&](int i, const Frags &cur, Frags &nxt) {
        if (i + 1 < nk) {
            wait_stages<OPS, P - 1>(min(P - 2, nk - 2 - i));
            __builtin_amdgcn_s_waitcnt(0xC07F);       // lgkmcnt(0): this wavefront's LDS reads are done
            lds_barrier();
            if (i + P < nk) issue((i + P) % NST, (i + P) * BK);
            read(nxt, (i + 1) % NST);
        }
        mma(cur);
    };
    // The same step where stage i + 1 exists and stage i + P is still to be
    // issued: no branch, a constant wait.  With the conditional form alone
    // the loop body joins a path on which the previous step's fragment reads
    // were never waited for, so the compiler waited for every LDS read
    // (including the ones just issued for the next stage) before each
    // second step's products.
    auto step_full = [&](int i, const Frags &cur, Frags &nxt) {
        __builtin_amdgcn_s_waitcnt(vmcnt_imm((P - 2) * OPS));
        __builtin_amdgcn_s_waitcnt(0xC07F);
        lds_barrier();
        issue((i + P) % NST, (i + P) * BK);
        read(nxt, (i + 1) % NST);
        mma(cur);
        // Issue order for one wavefront per SIMD (four wavefronts): the stage
        // loads, then one fragment read between consecutive products, so the
        // reads drain while the matrix cores run (lm_head at M = 256: 451 ->
        // 423 us).  With two wavefronts per SIMD the compiler's own order was
        // faster (the 256 x 256 tile: 70 against 73 us at M = 256).
        if constexpr (NW == 4) {
            constexpr int NRD = (BK / 16) * (FM + FN), NMM = (BK / 16) * FM * FN;
            __builtin_amdgcn_sched_group_barrier(0x020, OPS, 0);
#pragma unroll
            for (int k = 0; k < NRD && k < NMM; ++k) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
            if constexpr (NMM > NRD) __builtin_amdgcn_sched_group_barrier(0x008, NMM - NRD, 0);
        }
    };
#pragma unroll
    for (int i = 0; i < P; ++i)
        if (i < nk) issue(i, i * BK);
    Frags f0, f1;
    if (nk > 0) {
        wait_stages<OPS, P - 1>(min(P - 1, nk - 1));
        lds_barrier();
        read(f0, 0);
    }
    int i = 0;
    for (; i + 1 + P < nk; i += 2) {
        step_full(i, f0, f1);
        step_full(i + 1, f1, f0);
    }
    for (; i + 1 < nk; i += 2) {
        step(i, f0, f1);
        step(i + 1, f1, f0);
    }
    if (i < nk) step(i, f0, f1);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));   // nothing may land in LDS after the workgroup ends

    if constexpr (SWIGLU) {
        // Tile nt of the interleaved copy: wavefront 0 holds gate features
        // 64 nt .. 64 nt + 63, wavefront 1 the matching up features.  Up goes
        // through the idle ring; wavefront 0 writes act[row][64 nt + j].
        constexpr int TP = 68;
        static_assert(BM * TP * 4 <= NST * STAGE * 16, "SwiGLU staging fits the ring");
        float *T = reinterpret_cast<float *>(ring);
        __syncthreads();                              // every wavefront is done reading the ring
        if (wave == 1)
#pragma unroll
            for (int a = 0; a < FM; ++a)
#pragma unroll
                for (int b = 0; b < FN; ++b)
#pragma unroll
                    for (int q = 0; q < 16; ++q)
                        T[(32 * a + 8 * (q >> 2) + 4 * h + (q & 3)) * TP + 32 * b + r32] = acc[a][b][q];
        __syncthreads();
        if (wave == 0) {
            const int F = N / 2;
#pragma unroll
            for (int a = 0; a < FM; ++a)
#pragma unroll
                for (int b = 0; b < FN; ++b) {
                    const int j = nt * 64 + 32 * b + r32;
#pragma unroll
                    for (int q = 0; q < 16; ++q) {
                        const int rl = 32 * a + 8 * (q >> 2) + 4 * h + (q & 3), row = m0 + rl;
                        if (row < row_end && j < F)
                            act[out_row(row) * ldo + j] = swiglu_bf16(0.f + acc[a][b][q], 0.f + T[rl * TP + 32 * b + r32]);
                    }
                }
        }
        return;
    }

    // lane holds, per 32x32 tile, column r32 and rows 8 (q / 4) + 4 h + q % 4
    float *o = out + (size_t)s * split_stride;
#pragma unroll
    for (int a = 0; a < FM; ++a)
#pragma unroll
        for (int b = 0; b < FN; ++b) {
            const int col = n0 + wn0 + 32 * b + r32;
            if (col >= N) continue;
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const int row = m0 + wm0 + 32 * a + 8 * (q >> 2) + 4 * h + (q & 3);
                if (row < row_end) o[out_row(row) * ldo + col] = acc[a][b][q];
            }
        }
    // every configuration the launcher uses has 64-column wavefront tiles
    if (WN == 64 && amax != nullptr) {
        // per row: best (value, column) over this wavefront's 64 columns (one
        // 64-column block).  Each 32-row fragment goes through the wavefront's
        // own padded 32 x 68 float tile in the (now idle) ring; lane l scans
        // half a row, columns in increasing order, then the two halves meet.
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
        lds_barrier();                                // every wavefront is done reading the ring
        constexpr int TP = 68;
        static_assert(NW * 32 * TP * 4 <= NST * STAGE * 16, "argmax staging fits the ring");
        float *T = reinterpret_cast<float *>(ring) + wave * 32 * TP;
        const int ncb = (N + 63) / 64;
        const int rr = lane >> 1, hf = lane & 1;
#pragma unroll
        for (int a = 0; a < FM; ++a) {
#pragma unroll
            for (int b = 0; b < FN; ++b)
#pragma unroll
                for (int q = 0; q < 16; ++q) T[(8 * (q >> 2) + 4 * h + (q & 3)) * TP + 32 * b + r32] = acc[a][b][q];
            float bv = -INFINITY;
            int bi = 0x7fffffff;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const float4 v = *reinterpret_cast<const float4 *>(T + rr * TP + 32 * hf + 4 * i);
                const int col = n0 + wn0 + 32 * hf + 4 * i;
                if (col + 0 < N) better(bv, bi, v.x, col + 0);
                if (col + 1 < N) better(bv, bi, v.y, col + 1);
                if (col + 2 < N) better(bv, bi, v.z, col + 2);
                if (col + 3 < N) better(bv, bi, v.w, col + 3);
            }
            const float v2 = __shfl_xor(bv, 1, 64);
            const int i2 = __shfl_xor(bi, 1, 64);
            better(bv, bi, v2, i2);
            const int row = m0 + wm0 + 32 * a + rr;
            if (hf == 0 && row < M && n0 + wn0 < N) amax[(size_t)row * ncb + (n0 + wn0) / 64] = ArgBest{bv, bi};
        }
    }
}

hipError_t launch_gemm_dma(const uint16_t *A, int lda, const uint16_t *W, const GemmShape &g, float *out,
                           long long split_stride, int ldo, hipStream_t st, ArgBest *amax, uint16_t *act)
{
    // 32 or 64 x 128 (small batches): two wavefronts side by side (32- or
    // 64-row, 64-column wavefront tiles); 128-column tiles: four wavefronts
    // (2 x 2, 64-row and 64-column wavefront tiles), 64-element stages;
    // 256 x 256: eight wavefronts (2 x 4, 128 x 64), two per SIMD, 32-element
    // stages, three in the ring (96 KB): from M = 256 to 32768 it measured
    // 1-5% faster than four (gate/up at M = 8192: 1307 against 1378 us).
    // Every configuration has 64-column wavefront tiles, as the argmax
    // epilogue needs.
    const int bk = g.bn == 256 ? 32 : 64;
    if (g.K % bk != 0 || g.Kc % bk != 0 || g.M <= 0) return hipErrorInvalidValue;
    const int num_n = (g.N + g.bn - 1) / g.bn;
    const int num_m = (g.M + g.bm - 1) / g.bm;
    dim3 grid(num_m * num_n, g.S);
    if (g.pk) {   // tile-packed weights: the small-M configurations only
        if (act != nullptr) {   // gate/up-interleaved copy, SwiGLU epilogue, no split-K
            if (g.S != 1 || g.N % 128 != 0) return hipErrorInvalidValue;
            if (g.bm == 32 && g.bn == 128)
                KLAUNCH((k_gemm_dma<32, 128, 64, 4, 1, 2, true, true>), grid, dim3(128), 0, st, A, lda, W,
                                   g.M, g.N, g.K, g.Kc, nullptr, 0, ldo, nullptr, act, ExpertTiles{});
            else if (g.bm == 64 && g.bn == 128)
                KLAUNCH((k_gemm_dma<64, 128, 64, 4, 1, 2, true, true>), grid, dim3(128), 0, st, A, lda, W,
                                   g.M, g.N, g.K, g.Kc, nullptr, 0, ldo, nullptr, act, ExpertTiles{});
            else
                return hipErrorInvalidValue;
            return hipGetLastError();
        }
        if (g.bm == 32 && g.bn == 128)
            KLAUNCH((k_gemm_dma<32, 128, 64, 4, 1, 2, true>), grid, dim3(128), 0, st, A, lda, W, g.M, g.N,
                               g.K, g.Kc, out, split_stride, ldo, amax, nullptr, ExpertTiles{});
        else if (g.bm == 64 && g.bn == 128)
            KLAUNCH((k_gemm_dma<64, 128, 64, 4, 1, 2, true>), grid, dim3(128), 0, st, A, lda, W, g.M, g.N,
                               g.K, g.Kc, out, split_stride, ldo, amax, nullptr, ExpertTiles{});
        else
            return hipErrorInvalidValue;
        return hipGetLastError();
    }
    if (g.bm == 32 && g.bn == 128)
        KLAUNCH((k_gemm_dma<32, 128, 64, 4, 1, 2>), grid, dim3(128), 0, st, A, lda, W, g.M, g.N, g.K, g.Kc,
                           out, split_stride, ldo, amax, nullptr, ExpertTiles{});
    else if (g.bm == 64 && g.bn == 128)
        KLAUNCH((k_gemm_dma<64, 128, 64, 4, 1, 2>), grid, dim3(128), 0, st, A, lda, W, g.M, g.N, g.K, g.Kc,
                           out, split_stride, ldo, amax, nullptr, ExpertTiles{});
    else if (g.bm == 128 && g.bn == 128)
        KLAUNCH((k_gemm_dma<128, 128, 64, 4, 2, 4>), grid, dim3(256), 0, st, A, lda, W, g.M, g.N, g.K, g.Kc,
                           out, split_stride, ldo, amax, nullptr, ExpertTiles{});
    else if (g.bm == 256 && g.bn == 128)
        KLAUNCH((k_gemm_dma<256, 128, 64, 3, 2, 4>), grid, dim3(256), 0, st, A, lda, W, g.M, g.N, g.K, g.Kc,
                           out, split_stride, ldo, amax, nullptr, ExpertTiles{});
    else if (g.bm == 256 && g.bn == 256)
        KLAUNCH((k_gemm_dma<256, 256, 32, 3, 2, 8>), grid, dim3(512), 0, st, A, lda, W, g.M, g.N, g.K, g.Kc,
                           out, split_stride, ldo, amax, nullptr, ExpertTiles{});
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_gemm_tiled(const uint16_t *A, int lda, const uint16_t *W, const GemmShape &g, int bm, float *out,
                             long long split_stride, int ldo, hipStream_t st, ArgBest *amax)
{
    if (amax != nullptr && bm == 64) return hipErrorInvalidValue;   // argmax epilogue needs 64-column wavefront tiles
    const int num_n = (g.N + 127) / 128;
    const int num_m = (g.M + bm - 1) / bm;
    dim3 grid(num_m * num_n, g.S);
    switch (bm) {
    case 64:
        KLAUNCH((k_gemm_tiled<64, 128, 1>), grid, dim3(256), 0, st, A, lda, W, g.M, g.N, g.K, g.Kc, out,
                           split_stride, ldo, amax);
        break;
    case 128:
        KLAUNCH((k_gemm_tiled<128, 128, 2>), grid, dim3(256), 0, st, A, lda, W, g.M, g.N, g.K, g.Kc, out,
                           split_stride, ldo, amax);
        break;
    case 256:
        KLAUNCH((k_gemm_tiled<256, 128, 2>), grid, dim3(256), 0, st, A, lda, W, g.M, g.N, g.K, g.Kc, out,
                           split_stride, ldo, amax);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_gemm(const uint16_t *A, int lda, const uint16_t *W, const GemmShape &g, float *out,
                       long long split_stride, int ldo, hipStream_t st, ArgBest *amax)
{
    constexpr int NT = 4;
    const int ncb = (g.N + 16 * NT - 1) / (16 * NT);
    const int rows_per_tile = 16 * g.mt;
    dim3 grid((ncb + 3) / 4, g.S, (g.M + rows_per_tile - 1) / rows_per_tile);
    switch (g.mt) {
    case 1:
        KLAUNCH((k_gemm<1, NT, 4>), grid, dim3(256), 0, st, A, lda, W, g.M, g.N, g.K, g.Kc, out,
                           split_stride, ldo, amax);
        break;
    case 2:
        KLAUNCH((k_gemm<2, NT, 4>), grid, dim3(256), 0, st, A, lda, W, g.M, g.N, g.K, g.Kc, out,
                           split_stride, ldo, amax);
        break;
    case 4:
        KLAUNCH((k_gemm<4, NT, 2>), grid, dim3(256), 0, st, A, lda, W, g.M, g.N, g.K, g.Kc, out,
                           split_stride, ldo, amax);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// QKV epilogue: split reduction, bf16 rounding, rotary embedding at the
// row's own position, bf16 rounding, KV append.  Block (head, row); thread i
// owns the rotation pair (i, i + d/2).
// ---------------------------------------------------------------------------
// The QKV epilogue of one rotation pair (elements i and i + d/2 of a head):
// the split partials at columns c0 and c0 + half folded in split order (loads
// of up to eight splits issued together), both sums rounded to bf16, rotated
// by (cos, sin) when rot, rounded again.  k_qkv_post and the attention
// kernel's fused epilogue both run this, so they write the same bits.
__device__ __forceinline__ void qkv_pair(const float *__restrict__ pb, long long stride, int S, int c0, int half,
                                         bool rot, float2 cs, uint16_t &b0, uint16_t &b1)
{
    float x0 = 0.f, x1 = 0.f;
    if (S == 1) {
        x0 += pb[c0];
        x1 += pb[c0 + half];
    } else for (int s = 0; s < S; s += 8) {
        float a0[8], a1[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (s + u < S) {
                a0[u] = pb[(s + u) * stride + c0];
                a1[u] = pb[(s + u) * stride + c0 + half];
            }
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (s + u < S) {
                x0 += a0[u];
                x1 += a1[u];
            }
    }
    x0 = bf2f(f2bf(x0));
    x1 = bf2f(f2bf(x1));
    if (rot) {
        const float y0 = __builtin_fmaf(x0, cs.x, -(x1 * cs.y));
        const float y1 = __builtin_fmaf(x1, cs.x, x0 * cs.y);
        x0 = y0;
        x1 = y1;
    }
    b0 = f2bf(x0);
    b1 = f2bf(x1);
}

__global__ void k_qkv_post(const float *__restrict__ part, int S, long long part_stride,
                           const uint8_t *__restrict__ valid, const int32_t *__restrict__ pos,
                           const int32_t *__restrict__ slot_of_row, int slot_const, int nq, int nkv, int d,
                           const float2 *__restrict__ rope_tab, uint16_t *__restrict__ q,
                           uint16_t *__restrict__ kc, uint16_t *__restrict__ vc, KvView kv)
{
    const int nh = nq + 2 * nkv;
    const int hd = blockIdx.x % nh, r = blockIdx.x / nh, i = threadIdx.x;
    const int half = d >> 1;
    if (i >= half) return;
    if (valid != nullptr && !valid[r]) return;
    const int p = pos[r];
    const int ncols = (nq + 2 * nkv) * d;
    const bool rot = hd < nq + nkv;
    float2 cs = {1.f, 0.f};
    if (rot) cs = rope_tab[(size_t)p * half + i];    // issued with the partial loads
    uint16_t b0, b1;
    qkv_pair(part + (size_t)r * ncols, part_stride, S, hd * d + i, half, rot, cs, b0, b1);
    const int c0 = hd * d + i, c1 = c0 + half;
    if (hd < nq) {
        q[(size_t)r * nq * d + c0] = b0;
        q[(size_t)r * nq * d + c1] = b1;
    } else {
        const int slot = row_slot(slot_of_row, slot_const, r);
        if (hd < nq + nkv) {
            uint16_t *dst = kc + kv_offset(kv, nkv, d, slot, hd - nq, p);
            dst[i] = b0;
            dst[i + half] = b1;
        } else {
            const int kvh = hd - nq - nkv;
            vc[v_offset(kv, nkv, d, slot, kvh, p, i)] = b0;
            vc[v_offset(kv, nkv, d, slot, kvh, p, i + half)] = b1;
        }
    }
}

hipError_t launch_qkv_post(const float *part, int S, long long part_stride, int rows, const uint8_t *valid,
                           const int32_t *pos, const int32_t *slot_of_row, int slot_const, int nq, int nkv,
                           int d, const float2 *rope_tab, uint16_t *q, uint16_t *kc, uint16_t *vc, KvView kv,
                           hipStream_t st)
{
    const long long blocks = (long long)rows * (nq + 2 * nkv);
    KLAUNCH(k_qkv_post, dim3((unsigned)blocks), dim3(64), 0, st, part, S, part_stride, valid, pos,
                       slot_of_row, slot_const, nq, nkv, d, rope_tab, q, kc, vc, kv);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Split-KV decode attention.  The split count of a row is
// ceil((pos + 1) / chunk): a function of the row's own length only, so the
// split is request-local and the merge order (split index) is fixed.
//
// Block (kvh, split, row), four wavefronts.  The chunk is walked in steps of
// 128 tokens: the step's key rows and value rows ([token][d], as cached) are
// loaded global -> LDS by direct 16-byte loads in which every instruction
// covers whole 128-byte lines (4 rows of 256 bytes); a load form of 16 rows
// x 64 bytes per
// instruction, which the matrix-core operand layout would give if loaded
// straight into registers, caps the read rate near 4.7 TB/s against 6.2 TB/s
// for whole lines.  Wavefront w then takes the step's 32-token block w from
// LDS (so over the chunk: blocks w, w + 4, w + 8, ...), processed as:
//  * scores S^T = K q^T on 16x16x32 MFMA, two 16-token tiles, the G query
//    heads of the group in column slots 0..G-1: lane l reads 16 bytes of one
//    key row per tile and ends holding head l % 16's scores of the eight
//    consecutive tokens 8 (l / 16) .. +7 (see attn_tok);
//  * online softmax per head: lane l keeps head l % 16's running maximum and
//    a partial sum over its own tokens;
//  * O += P V on 16x16x32 MFMA: the lane's eight weights (two tiles x four
//    tokens) are its A fragment as they stand -- split into two bf16 halves
//    hi + lo (two MFMAs) so P keeps about 16 significant bits -- and the
//    matching B fragment (those eight tokens of one dimension) comes from
//    the token-major value rows by two transposed LDS reads (lds_read_tr16);
//  * masked tokens (past the row's length) contribute exact zeros: their
//    value fragments are zero-filled, never multiplied; loads past the
//    length read clamped (real) positions.
// The four wavefront partials are combined in wavefront order.  Two blocks
// share a CU (64 KB of LDS each for d = 128): one computes while the
// other's step is in flight.
// LDS layouts, 16-byte units, XOR-swizzled so that a fragment read hits
// distinct bank groups: key unit (token t, chunk c) at t KCH + (c ^ ks(t))
// (16 lanes: 16 tokens of one chunk), value unit (token t, chunk c) at
// t KCH + (c ^ vtile_swz<KCH>(t)) (a transposed read: 4 tokens x 32 bytes
// per 16 lanes).
// ---------------------------------------------------------------------------

// Token order inside a 32-token block.  Score tile T's MFMA row m carries
// token 8 (m / 4) + 4 T + m % 4, so that lane group kg ends up holding the
// scores of tokens 8 kg .. 8 kg + 7 (tile 0 rows 4 kg + i, tile 1 rows
// 4 kg + i): its P fragment is eight consecutive tokens and its value
// fragment those eight tokens of one dimension.
__device__ __forceinline__ int attn_tok(int T, int m) { return 8 * (m >> 2) + 4 * T + (m & 3); }

// key-row swizzle: the 16 tokens a fragment read touches, {8 a + 4 T + b},
// map to 16 distinct (row parity, chunk) bank groups
template <int KCH>
__device__ __forceinline__ int attn_kswz(int t)
{
    if constexpr (KCH == 16) return (((t >> 3) & 3) << 2) | (t & 3);
    else return (((t >> 3) & 3) << 1) | ((t >> 1) & 1);
}

template <int D, int G>
__global__ __launch_bounds__(256) void k_attn_split(const uint16_t *__restrict__ q, const uint8_t *__restrict__ valid,
                                                    const int32_t *__restrict__ pos,
                                                    const int32_t *__restrict__ slot_of_row, int slot_const,
                                                    int nq, int nkv, uint16_t *__restrict__ kc,
                                                    uint16_t *__restrict__ vc, KvView kv, int chunk,
                                                    int max_splits, float *__restrict__ ws, QkvIn qi,
                                                    const int32_t *__restrict__ row_order)
{
    constexpr int ET = D / 16;
    constexpr int KCH = D / 8;                        // 16-byte chunks per key row
    constexpr int STEP = 128;                         // tokens per step, 32 per wavefront
    constexpr int KU = STEP * KCH, VU = STEP * KCH;    // 16-byte units of the step's keys, values
    constexpr int K_OPS = KU / 256, V_OPS = VU / 256;
    static_assert(K_OPS * 256 == KU && V_OPS * 256 == VU, "step loads cover the block");
    static_assert(4 * G * D * 4 <= (KU + VU) * 16, "wavefront partials fit the tile");
    __shared__ __attribute__((aligned(16))) uint4 tile[KU + VU];
    __shared__ float cm[4][16], cl[4][16];
    __shared__ int32_t pgs[2][64];                    // paged: the pages of a step, fetched one step ahead
    __shared__ __attribute__((aligned(16))) uint16_t qs[G * D];     // fused epilogue: the group's q
    __shared__ __attribute__((aligned(16))) uint16_t kvn[2 * D];    // fused epilogue: the new token's k, v
    typedef __attribute__((address_space(3))) void lds_void;

    // grid (kv head, split, row): the kv heads of a split run side by side,
    // so the concurrently streamed value rows (2 max_seq_len bytes apart
    // within a head) spread over the memory channels; with the splits of one
    // head side by side instead, a load-only replica streamed 11% slower.
    // Grid z takes the rows in row_order when given (the host puts live rows
    // longest first): any permutation of 0..rows-1 gives the same results.
    const int kvh = blockIdx.x, split = blockIdx.y, r = row_order != nullptr ? row_order[blockIdx.z] : blockIdx.z;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    if (valid != nullptr && !valid[r]) return;
    const int n = pos[r] + 1;
    const int t0 = split * chunk;
    if (t0 >= n) return;
    const int t1 = min(n, t0 + chunk);
    const int slot = row_slot(slot_of_row, slot_const, r);
    const int hl = lane & 15, kg = lane >> 4;
    const bool fused = qi.part != nullptr;
    const int pnew = n - 1;                           // the new token's position
    const bool owns_new = fused && t1 == n;           // the split that holds it appends and patches it

    // q^T fragments (B operand of the scores): lane l supplies head l % 16,
    // dims 32 kk + 8 (l / 16) .. +7; from q, or (fused) from qs below
    bf16x8 qf[D / 32];
    const uint4 zq = {0u, 0u, 0u, 0u};
    if (!fused) {
        const uint16_t *qr = q + (size_t)r * nq * D + ((size_t)kvh * G + hl) * D + kg * 8;
#pragma unroll
        for (int kk = 0; kk < D / 32; ++kk) {
            uint4 v = zq;
            if (hl < G) v = *(const uint4 *)(qr + 32 * kk);
            qf[kk] = __builtin_bit_cast(bf16x8, v);
        }
    }
    const float scale = 1.0f / sqrtf((float)D);
    f32x4 oacc[ET];
#pragma unroll
    for (int et = 0; et < ET; ++et) oacc[et] = (f32x4){0.f, 0.f, 0.f, 0.f};
    float mrun = -INFINITY, lrun = 0.f;

    // the step's loads: unit u = 256 j + tid of the key part (token u / KCH)
    // or of the value part (dimension u / 16); positions past the chunk read
    // the last real key, or the last real 8-token value chunk.  A paged
    // cache's page of position t is pgs[buf][t / ps - tb0 / ps] (a step spans
    // at most 128 / ps + 1 <= 9 pages), so no load waits on a page-table read.
    const int kmax = t1 - 1;
    const bool paged = kv.layout == 1;
    const int ps = paged ? kv.page_size : 1;
    const int last_page = kmax / ps;
    auto fetch_pages = [&](int tb0, int buf) {        // wavefront 0, lane l: page tb0 / ps + l (clamped)
        if (paged && wave == 0) {
            const int pi = min(tb0 / ps + lane, last_page);
            __builtin_amdgcn_global_load_lds((const void *)(kv.page_table + (size_t)slot * kv.max_pages_per_seq + pi),
                                             (lds_void *)&pgs[buf][0], 4, 0, 0);
        }
    };
    auto issue = [&](int tb0, int buf) {
        uint4 *base = tile + wave * 64;
        const int p0 = tb0 / ps;
#pragma unroll
        for (int j = 0; j < K_OPS; ++j) {
            const int u = j * 256 + tid, tk = u / KCH, c = (u % KCH) ^ attn_kswz<KCH>(tk);
            const int t = min(tb0 + tk, kmax);
            size_t off;
            if (paged) off = (((size_t)pgs[buf][t / ps - p0] * nkv + kvh) * ps + t % ps) * D;
            else off = (((size_t)slot * nkv + kvh) * kv.max_seq_len + t) * D;
            __builtin_amdgcn_global_load_lds((const void *)(kc + off + 8 * c), (lds_void *)(base + j * 256), 16, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < V_OPS; ++j) {
            const int u = j * 256 + tid, tv = u / KCH, c = (u % KCH) ^ vtile_swz<KCH>(tv);
            const int t = min(tb0 + tv, kmax);
            size_t off;
            if (paged) off = (((size_t)pgs[buf][t / ps - p0] * nkv + kvh) * ps + t % ps) * D;
            else off = (((size_t)slot * nkv + kvh) * kv.max_seq_len + t) * D;
            __builtin_amdgcn_global_load_lds((const void *)(vc + off + 8 * c), (lds_void *)(base + KU + j * 256), 16, 0,
                                             0);
        }
    };

    const int nsteps = (t1 - t0 + STEP - 1) / STEP;
    const uint4 z4 = {0u, 0u, 0u, 0u};
    fetch_pages(t0, 0);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    lds_barrier();
    // Step i's loads are issued as soon as every wavefront has taken step
    // i - 1's fragments out of the tile into registers, so they are in flight
    // while step i - 1 is computed; a paged cache's pages for step i + 1 are
    // fetched right behind them.
    issue(t0, 0);
    if (nsteps > 1) fetch_pages(t0 + STEP, 1);
    for (int st_i = 0; st_i < nsteps; ++st_i) {
        const int tb0 = t0 + STEP * st_i;
        if (fused && st_i == 0) {
            // The QKV epilogue while the first step's loads are in flight:
            // pair pi < G d/2 is q (head pi / (d/2)); the owner of the new
            // token also makes its k (rotated) and v pairs, appends them to
            // the cache and keeps them in kvn for the patch below.
            const int nqkv = (nq + 2 * nkv) * D, nqp = G * (D / 2);
            const float *pb = qi.part + (size_t)r * nqkv;
            const float2 *rt = qi.rope + (size_t)pnew * (D / 2);
            const int npairs = nqp + (owns_new ? D : 0);
            for (int pi = tid; pi < npairs; pi += 256) {
                int i, c0, which;                     // 0: q, 1: k, 2: v
                if (pi < nqp) {
                    i = pi % (D / 2);
                    c0 = (kvh * G + pi / (D / 2)) * D + i;
                    which = 0;
                } else if (pi < nqp + D / 2) {
                    i = pi - nqp;
                    c0 = (nq + kvh) * D + i;
                    which = 1;
                } else {
                    i = pi - nqp - D / 2;
                    c0 = (nq + nkv + kvh) * D + i;
                    which = 2;
                }
                float2 cs = {1.f, 0.f};
                if (which < 2) cs = rt[i];
                uint16_t b0, b1;
                qkv_pair(pb, qi.stride, qi.S, c0, D / 2, which < 2, cs, b0, b1);
                if (which == 0) {
                    const int hh = pi / (D / 2);
                    qs[hh * D + i] = b0;
                    qs[hh * D + i + D / 2] = b1;
                } else if (which == 1) {
                    kvn[i] = b0;
                    kvn[i + D / 2] = b1;
                    uint16_t *dst = kc + kv_offset(kv, nkv, D, slot, kvh, pnew);
                    dst[i] = b0;
                    dst[i + D / 2] = b1;
                } else {
                    kvn[D + i] = b0;
                    kvn[D + i + D / 2] = b1;
                    vc[v_offset(kv, nkv, D, slot, kvh, pnew, i)] = b0;
                    vc[v_offset(kv, nkv, D, slot, kvh, pnew, i + D / 2)] = b1;
                }
            }
        }
        if (fused && st_i == 0) __builtin_amdgcn_s_waitcnt(0);   // also the qs / kvn stores
        else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
        lds_barrier();                                // the step (and the next step's pages) are in LDS
        if (fused && st_i == 0) {
            const uint16_t *qr = qs + hl * D + kg * 8;
#pragma unroll
            for (int kk = 0; kk < D / 32; ++kk) {
                uint4 v = zq;
                if (hl < G) v = *(const uint4 *)(qr + 32 * kk);
                qf[kk] = __builtin_bit_cast(bf16x8, v);
            }
        }
        if (owns_new && pnew >= tb0 && pnew < tb0 + STEP) {
            // the step holds the new token: its cache entries may have
            // landed before the append, so its tile slots take kvn
            const int tl = pnew - tb0;
            if (tid < KCH) {
                tile[tl * KCH + (tid ^ attn_kswz<KCH>(tl))] = reinterpret_cast<const uint4 *>(kvn)[tid];
            } else if (tid >= 64 && tid < 64 + KCH) {
                const int c = tid - 64;
                tile[KU + tl * KCH + (c ^ vtile_swz<KCH>(tl))] = reinterpret_cast<const uint4 *>(kvn + D)[c];
            }
            __builtin_amdgcn_s_waitcnt(0);
            lds_barrier();
        }
        const int tb = tb0 + 32 * wave;
        const bool active = tb < t1;                  // wave-uniform: some token of this 32-token block is real
        const int wt1 = t1;
        // fragments from LDS
        bf16x8 kf[2][D / 32];
        uint4 vfr[ET];
        if (active) {
#pragma unroll
        for (int T = 0; T < 2; ++T) {
            const int tl = 32 * wave + attn_tok(T, hl);
#pragma unroll
            for (int kk = 0; kk < D / 32; ++kk)
                kf[T][kk] = __builtin_bit_cast(bf16x8, tile[tl * KCH + ((kg + 4 * kk) ^ attn_kswz<KCH>(tl))]);
        }
        {
            // value fragments: lane (hl, kg) takes dimension 16 et + hl of the
            // eight tokens 8 kg .. 8 kg + 7 of its 32-token block by two
            // transposed reads (tokens 4 r + 0..3); in its 16-lane group, lane
            // a + 4 q points at token 8 kg + 4 r + q, dimensions 16 et + 4 a ..
            const int nv = min(8, wt1 - (tb + 8 * kg));   // how many of the lane's eight tokens are real
            const int a = hl & 3, qq = hl >> 2;
#pragma unroll
            for (int et = 0; et < ET; ++et) {
                uint2 part[2];
#pragma unroll
                for (int r = 0; r < 2; ++r) {
                    const int tv = 32 * wave + 8 * kg + 4 * r + qq;
                    const int c = 2 * et + (a >> 1);
                    part[r] = lds_read_tr16(reinterpret_cast<const char *>(tile + KU + tv * KCH + (c ^ vtile_swz<KCH>(tv))) +
                                            8 * (a & 1));
                }
                uint4 v = {part[0].x, part[0].y, part[1].x, part[1].y};   // low half = earlier token
                if (nv < 8) {   // zero the tokens past the row's length
                    uint32_t *w = (uint32_t *)&v;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        if (2 * j >= nv) w[j] = 0u;
                        else if (2 * j + 1 >= nv) w[j] &= 0x0000ffffu;
                    }
                }
                vfr[et] = v;
            }
        }
        }
        // the tile is free once every wavefront holds its fragments: the next
        // step's loads (and the pages of the one after) go out now
        __builtin_amdgcn_s_waitcnt(0xC07F);           // lgkmcnt(0): this wavefront's LDS reads are done
        lds_barrier();
        if (st_i + 1 < nsteps) {
            issue(tb0 + STEP, (st_i + 1) & 1);
            if (st_i + 2 < nsteps) fetch_pages(tb0 + 2 * STEP, st_i & 1);
        }
        if (!active) continue;
        f32x4 st[2];
#pragma unroll
        for (int T = 0; T < 2; ++T) {
            st[T] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < D / 32; ++kk)
                st[T] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[T][kk], qf[kk], st[T], 0, 0, 0);
        }
        // lane (hl, kg) now holds head hl's scores of tokens tb + 8 kg + 4 T + i
        float mt = -INFINITY;
#pragma unroll
        for (int T = 0; T < 2; ++T)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float sv = (tb + 8 * kg + 4 * T + i < wt1) ? st[T][i] * scale : -INFINITY;
                st[T][i] = sv;
                mt = fmaxf(mt, sv);
            }
        mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
        mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
        const float mnew = fmaxf(mrun, mt);              // finite: every block has a real token
        const float alpha = __expf(mrun - mnew);         // 0 on the first block
        // each weight enters the matrix core as two bf16 halves, p = hi + lo,
        // which carry about 16 significant bits; the sum uses the fp32 weight
        uint16_t pw[8], pl[8];
        float ls = 0.f;
#pragma unroll
        for (int T = 0; T < 2; ++T)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float pe = __expf(st[T][i] - mnew);
                ls += pe;
                pw[4 * T + i] = f2bf(pe);
                pl[4 * T + i] = f2bf(pe - bf2f(pw[4 * T + i]));
            }
        lrun = lrun * alpha + ls;
        mrun = mnew;
        // rescale the accumulators: lane l holds heads 4 (l / 16) + i
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float ai = __shfl(alpha, 4 * kg + i, 64);
#pragma unroll
            for (int et = 0; et < ET; ++et) oacc[et][i] *= ai;
        }
        bf16x8 pf, pfl;
        {
            uint4 pv, pq;
            pv.x = (uint32_t)pw[0] | ((uint32_t)pw[1] << 16);
            pv.y = (uint32_t)pw[2] | ((uint32_t)pw[3] << 16);
            pv.z = (uint32_t)pw[4] | ((uint32_t)pw[5] << 16);
            pv.w = (uint32_t)pw[6] | ((uint32_t)pw[7] << 16);
            pq.x = (uint32_t)pl[0] | ((uint32_t)pl[1] << 16);
            pq.y = (uint32_t)pl[2] | ((uint32_t)pl[3] << 16);
            pq.z = (uint32_t)pl[4] | ((uint32_t)pl[5] << 16);
            pq.w = (uint32_t)pl[6] | ((uint32_t)pl[7] << 16);
            pf = __builtin_bit_cast(bf16x8, pv);
            pfl = __builtin_bit_cast(bf16x8, pq);
        }
#pragma unroll
        for (int et = 0; et < ET; ++et) {
            const bf16x8 vf = __builtin_bit_cast(bf16x8, vfr[et]);
            oacc[et] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pf, vf, oacc[et], 0, 0, 0);
            oacc[et] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pfl, vf, oacc[et], 0, 0, 0);
        }
    }
    // per-head sum over the four 16-lane groups (fixed order)
    lrun += __shfl_xor(lrun, 16, 64);
    lrun += __shfl_xor(lrun, 32, 64);

    // combine the four wavefronts in wavefront order (partials staged in the idle tile)
    lds_barrier();                                    // every wavefront is done with the last step
    float *ca = reinterpret_cast<float *>(tile);      // [4][G D]
    if (lane < 16) {
        cm[wave][lane] = mrun;
        cl[wave][lane] = lrun;
    }
#pragma unroll
    for (int et = 0; et < ET; ++et)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int g = 4 * kg + i;
            if (g < G) ca[wave * G * D + g * D + 16 * et + hl] = oacc[et][i];
        }
    __syncthreads();
    float *o = ws + (((size_t)r * nkv + kvh) * max_splits + split) * (G * (D + 2));
    for (int idx = threadIdx.x; idx < G * D; idx += 256) {
        const int g = idx / D;
        float M = cm[0][g];
#pragma unroll
        for (int w = 1; w < 4; ++w) M = fmaxf(M, cm[w][g]);
        float L = 0.f, A = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const float f = __expf(cm[w][g] - M);   // empty wavefronts: exp(-inf) = 0
            L += cl[w][g] * f;
            A += ca[w * G * D + idx] * f;
        }
        o[2 * G + idx] = A;
        if (idx % D == 0) {
            o[g] = M;
            o[G + g] = L;
        }
    }
}

// Merge of a row's splits in split order (any number of splits; the plans
// with more than 8).  Block (HB query heads of one kv head, row), one thread per (head, dimension).  Each head's (max, sum) pair
// of every split goes to LDS while each thread's values of the first 32
// splits load into registers (one round trip for up to 32 splits, the
// small-batch case); then, per head, the exact maximum M over the splits,
// the weights f_s = exp(m_s - M) and L = sum_s l_s f_s in split order by one
// thread; each thread folds its dimension over the splits in split order
// and writes A / L in bf16.
template <int D, int G>
constexpr int merge_heads() { return G < 512 / D ? G : 512 / D; }

template <int D, int G>
__global__ __launch_bounds__((D * merge_heads<D, G>())) void k_attn_merge(
    const float *__restrict__ ws, const uint8_t *__restrict__ valid, const int32_t *__restrict__ pos, int nq, int nkv,
    int chunk, int max_splits, uint16_t *__restrict__ o)
{
    constexpr int PF = 32;                            // splits whose values are in flight at once
    constexpr int HB = merge_heads<D, G>();           // divides G
    const int hl = threadIdx.x / D, dd = threadIdx.x % D;
    const int hq = blockIdx.x * HB + hl, r = blockIdx.y;
    const int kvh = hq / G, g = hq - kvh * G;
    uint16_t *orow = o + (size_t)r * nq * D + (size_t)hq * D;
    if (valid != nullptr && !valid[r]) {
        orow[dd] = 0;
        return;
    }
    extern __shared__ float fs[];                     // per head: [max_splits] maxima then weights, [max_splits] sums
    __shared__ float ML[HB][2];
    const int n = pos[r] + 1;
    const int ns = (n + chunk - 1) / chunk;
    float *fm = fs + (size_t)hl * 2 * max_splits, *fl = fm + max_splits;
    const int stride = G * (D + 2);
    const float *base = ws + ((size_t)r * nkv + kvh) * max_splits * stride;
    const float *a = base + 2 * G + g * D + dd;
    float v[PF];
#pragma unroll
    for (int u = 0; u < PF; ++u)
        if (u < ns) v[u] = a[(size_t)u * stride];
    for (int sp = dd; sp < ns; sp += D) {
        fm[sp] = base[(size_t)sp * stride + g];
        fl[sp] = base[(size_t)sp * stride + G + g];
    }
    __syncthreads();
    if (dd == 0) {
        float M = -INFINITY;
        for (int sp = 0; sp < ns; ++sp) M = fmaxf(M, fm[sp]);
        ML[hl][0] = M;
    }
    __syncthreads();
    for (int sp = dd; sp < ns; sp += D) fm[sp] = __expf(fm[sp] - ML[hl][0]);
    __syncthreads();
    if (dd == 0) {
        float L = 0.f;
        for (int sp = 0; sp < ns; ++sp) L += fl[sp] * fm[sp];
        ML[hl][1] = L;
    }
    __syncthreads();
    float acc = 0.f;
    for (int sp = 0; sp < ns; sp += PF) {
        if (sp > 0)
#pragma unroll
            for (int u = 0; u < PF; ++u)
                if (sp + u < ns) v[u] = a[(size_t)(sp + u) * stride];
#pragma unroll
        for (int u = 0; u < PF; ++u)
            if (sp + u < ns) acc += v[u] * fm[sp + u];
    }
    orow[dd] = f2bf(acc / ML[hl][1]);
}

// Merge of a row's splits in split order, for few splits (up to 8, the
// large-batch plans).  Block (kvh, row), 256 threads.  Every split's (max,
// sum) pair is loaded in one round into LDS; per head
// the exact maximum M over the splits, weights f_s = exp(m_s - M) and
// L = sum_s l_s f_s walked in split order by one thread; then each thread
// folds its E output elements over the splits in split order, eight splits'
// loads issued ahead of the adds, and writes A / L in bf16: the arithmetic
// of k_attn_merge, in the same order.  A plan uses one of the two for all
// its rows.
template <int D, int G>
__global__ __launch_bounds__(256) void k_attn_merge_kv(const float *__restrict__ ws, const uint8_t *__restrict__ valid,
                                                    const int32_t *__restrict__ pos, int nq, int nkv, int chunk,
                                                    int max_splits, uint16_t *__restrict__ o)
{
    constexpr int E = (G * D + 255) / 256;           // output elements per thread
    const int kvh = blockIdx.x, r = blockIdx.y, tid = threadIdx.x;
    uint16_t *orow = o + (size_t)r * nq * D + (size_t)kvh * G * D;
    if (valid != nullptr && !valid[r]) {
        for (int i = tid; i < G * D; i += 256) orow[i] = 0;
        return;
    }
    extern __shared__ float fs[];          // [G][ns] maxima then weights, [G][ns] sums, [G] M, [G] L
    const int n = pos[r] + 1;
    const int ns = (n + chunk - 1) / chunk;
    float *fm = fs, *fl = fs + G * max_splits, *Mg = fl + G * max_splits, *Lg = Mg + G;
    const int stride = G * (D + 2);
    const float *base = ws + ((size_t)r * nkv + kvh) * max_splits * stride;
    for (int idx = tid; idx < G * ns; idx += 256) {
        const int g = idx / ns, sp = idx - g * ns;
        fm[idx] = base[(size_t)sp * stride + g];
        fl[idx] = base[(size_t)sp * stride + G + g];
    }
    __syncthreads();
    if (tid < G) {
        float M = -INFINITY;
        for (int sp = 0; sp < ns; ++sp) M = fmaxf(M, fm[tid * ns + sp]);
        Mg[tid] = M;
    }
    __syncthreads();
    for (int idx = tid; idx < G * ns; idx += 256) fm[idx] = __expf(fm[idx] - Mg[idx / ns]);
    __syncthreads();
    if (tid < G) {
        float L = 0.f;
        for (int sp = 0; sp < ns; ++sp) L += fl[tid * ns + sp] * fm[tid * ns + sp];
        Lg[tid] = L;
    }
    __syncthreads();
    float acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.f;
    const float *a = base + 2 * G;
    int sp = 0;
    for (; sp + 8 <= ns; sp += 8) {
        float v[8][E];
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const int idx = tid + 256 * e;
                v[u][e] = idx < G * D ? a[(size_t)(sp + u) * stride + idx] : 0.f;
            }
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const int idx = tid + 256 * e;
                if (idx < G * D) acc[e] += v[u][e] * fm[(idx / D) * ns + sp + u];
            }
    }
    for (; sp < ns; ++sp)
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int idx = tid + 256 * e;
            if (idx < G * D) acc[e] += a[(size_t)sp * stride + idx] * fm[(idx / D) * ns + sp];
        }
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int idx = tid + 256 * e;
        if (idx < G * D) orow[idx] = f2bf(acc[e] / Lg[idx / D]);
    }
}

template <int D, int G>
static void launch_attn_dg(const uint16_t *q, int rows, const uint8_t *valid, const int32_t *pos,
                           const int32_t *slot_of_row, int slot_const, int nq, int nkv, uint16_t *kc,
                           uint16_t *vc, KvView kv, int chunk, int max_splits, float *ws, hipStream_t st, QkvIn qi,
                           const int32_t *row_order)
{
    KLAUNCH((k_attn_split<D, G>), dim3(nkv, max_splits, rows), dim3(256), 0, st, q, valid, pos,
                       slot_of_row, slot_const, nq, nkv, kc, vc, kv, chunk, max_splits, ws, qi, row_order);
}

template <int D, int G>
static void launch_merge_dg(const float *ws, int rows, const uint8_t *valid, const int32_t *pos, int nq,
                            int nkv, int chunk, int max_splits, uint16_t *o, hipStream_t st)
{
    if (max_splits <= 8) {   // one round trip either way: the per-kv-head layout launches fewer wavefronts
        const size_t shm = sizeof(float) * (2 * G * max_splits + 2 * G);
        KLAUNCH((k_attn_merge_kv<D, G>), dim3(nkv, rows), dim3(256), shm, st, ws, valid, pos, nq, nkv,
                           chunk, max_splits, o);
        return;
    }
    constexpr int HB = merge_heads<D, G>();
    const size_t shm = sizeof(float) * 2 * HB * max_splits;
    KLAUNCH((k_attn_merge<D, G>), dim3(nq / HB, rows), dim3(D * HB), shm, st, ws, valid, pos, nq, nkv,
                       chunk, max_splits, o);
}

#define CORUN_ATTN_DISPATCH(FN, ...)                                                \
    do {                                                                            \
        const int G_ = nq / nkv;                                                    \
        if (d == 64) {                                                              \
            switch (G_) {                                                           \
            case 1: FN<64, 1>(__VA_ARGS__); break;                                  \
            case 2: FN<64, 2>(__VA_ARGS__); break;                                  \
            case 4: FN<64, 4>(__VA_ARGS__); break;                                  \
            case 8: FN<64, 8>(__VA_ARGS__); break;                                  \
            default: return hipErrorInvalidValue;                                   \
            }                                                                       \
        } else if (d == 128) {                                                      \
            switch (G_) {                                                           \
            case 1: FN<128, 1>(__VA_ARGS__); break;                                 \
            case 2: FN<128, 2>(__VA_ARGS__); break;                                 \
            case 4: FN<128, 4>(__VA_ARGS__); break;                                 \
            case 8: FN<128, 8>(__VA_ARGS__); break;                                 \
            case 16: FN<128, 16>(__VA_ARGS__); break;                               \
            default: return hipErrorInvalidValue;                                   \
            }                                                                       \
        } else {                                                                    \
            return hipErrorInvalidValue;                                            \
        }                                                                           \
    } while (0)

hipError_t launch_attn_split(const uint16_t *q, int rows, const uint8_t *valid, const int32_t *pos,
                             const int32_t *slot_of_row, int slot_const, int nq, int nkv, int d,
                             uint16_t *kc, uint16_t *vc, KvView kv, int chunk, int max_splits,
                             float *ws, hipStream_t st, QkvIn qi, const int32_t *row_order)
{
    CORUN_ATTN_DISPATCH(launch_attn_dg, q, rows, valid, pos, slot_of_row, slot_const, nq, nkv, kc, vc, kv, chunk,
                        max_splits, ws, st, qi, row_order);
    return hipGetLastError();
}

hipError_t launch_attn_merge(const float *ws, int rows, const uint8_t *valid, const int32_t *pos, int nq, int nkv,
                             int d, int chunk, int max_splits, uint16_t *o, hipStream_t st)
{
    CORUN_ATTN_DISPATCH(launch_merge_dg, ws, rows, valid, pos, nq, nkv, chunk, max_splits, o, st);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// SwiGLU epilogue of the gate/up projection
// ---------------------------------------------------------------------------
__global__ void k_swiglu(const float *__restrict__ part, int S, long long part_stride, int F,
                         uint16_t *__restrict__ a, int lda)
{
    const int nb = (F + 255) / 256;
    const int r = blockIdx.x / nb;
    const int j = (blockIdx.x % nb) * 256 + threadIdx.x;
    if (j >= F) return;
    const float *p = part + (size_t)r * 2 * F;
    float gs = 0.f, us = 0.f;
    for (int s = 0; s < S; ++s) {
        gs += p[s * part_stride + j];
        us += p[s * part_stride + F + j];
    }
    a[(size_t)r * lda + j] = swiglu_bf16(gs, us);
}

hipError_t launch_swiglu(const float *part, int S, long long part_stride, int rows, int F, uint16_t *a, int lda,
                         hipStream_t st)
{
    const long long blocks = (long long)rows * ((F + 255) / 256);
    KLAUNCH(k_swiglu, dim3((unsigned)blocks), dim3(256), 0, st, part, S, part_stride, F, a, lda);
    return hipGetLastError();
}

__global__ void k_reduce_splits(const float *__restrict__ part, int S, long long stride, long long n,
                                float *__restrict__ out)
{
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x) {
        float v = 0.f;
        for (int s = 0; s < S; ++s) v += part[s * stride + i];
        out[i] = v;
    }
}

hipError_t launch_reduce_splits(const float *part, int S, long long stride, long long n, float *out, hipStream_t st)
{
    long long blocks = std::min<long long>((n + 255) / 256, 65536);
    KLAUNCH(k_reduce_splits, dim3((unsigned)blocks), dim3(256), 0, st, part, S, stride, n, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Greedy argmax: first index of the maximum.  (value, index) under
// "larger value, then smaller index" is a total order, so any combining tree
// gives the same, exact answer.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_argmax(const float *__restrict__ logits, int V,
                                                const uint8_t *__restrict__ valid, int32_t *__restrict__ next)
{
    const int r = blockIdx.x;
    if (valid != nullptr && !valid[r]) {
        if (threadIdx.x == 0) next[r] = -1;
        return;
    }
    const float *l = logits + (size_t)r * V;
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    for (int i = threadIdx.x; i < V; i += 256) better(bv, bi, l[i], i);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const float v2 = __shfl_xor(bv, off, 64);
        const int i2 = __shfl_xor(bi, off, 64);
        better(bv, bi, v2, i2);
    }
    __shared__ float sv[4];
    __shared__ int si[4];
    if ((threadIdx.x & 63) == 0) {
        sv[threadIdx.x >> 6] = bv;
        si[threadIdx.x >> 6] = bi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < 4; ++w) better(bv, bi, sv[w], si[w]);
        next[r] = (bi == 0x7fffffff) ? 0 : bi;
    }
}

__global__ __launch_bounds__(256) void k_argmax_partials(const ArgBest *__restrict__ part, int np,
                                                         const uint8_t *__restrict__ valid, int32_t *__restrict__ next)
{
    const int r = blockIdx.x;
    if (valid != nullptr && !valid[r]) {
        if (threadIdx.x == 0) next[r] = -1;
        return;
    }
    const ArgBest *p = part + (size_t)r * np;
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    for (int i = threadIdx.x; i < np; i += 256) better(bv, bi, p[i].v, p[i].i);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const float v2 = __shfl_xor(bv, off, 64);
        const int i2 = __shfl_xor(bi, off, 64);
        better(bv, bi, v2, i2);
    }
    __shared__ float sv[4];
    __shared__ int si[4];
    if ((threadIdx.x & 63) == 0) {
        sv[threadIdx.x >> 6] = bv;
        si[threadIdx.x >> 6] = bi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < 4; ++w) better(bv, bi, sv[w], si[w]);
        next[r] = (bi == 0x7fffffff) ? 0 : bi;
    }
}

hipError_t launch_argmax_partials(const ArgBest *part, int rows, int np, const uint8_t *valid, int32_t *next,
                                  hipStream_t st)
{
    KLAUNCH(k_argmax_partials, dim3(rows), dim3(256), 0, st, part, np, valid, next);
    return hipGetLastError();
}

hipError_t launch_argmax(const float *logits, int rows, int V, const uint8_t *valid, int32_t *next, hipStream_t st)
{
    KLAUNCH(k_argmax, dim3(rows), dim3(256), 0, st, logits, V, valid, next);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Device-side step feedback for multi-step runs.
// ---------------------------------------------------------------------------
__global__ void k_feedback(int32_t *tokens, int32_t *seq_lens, const uint8_t *valid, const int32_t *next, int B,
                           int32_t *history, int32_t *counter, int max_hist)
{
    const int c = *counter;
    for (int b = threadIdx.x; b < B; b += blockDim.x) {
        if (c < max_hist) history[(size_t)c * B + b] = next[b];
        if (valid[b]) {
            tokens[b] = next[b];
            seq_lens[b] += 1;
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) *counter = c + 1;
}

hipError_t launch_feedback(int32_t *tokens, int32_t *seq_lens, const uint8_t *valid, const int32_t *next, int B,
                           int32_t *history, int32_t *counter, int max_hist, hipStream_t st)
{
    KLAUNCH(k_feedback, dim3(1), dim3(256), 0, st, tokens, seq_lens, valid, next, B, history, counter,
                       max_hist);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Setup kernels
// ---------------------------------------------------------------------------
__global__ void k_rope_table(float2 *tab, int d, double theta)
{
    const int p = blockIdx.x, i = threadIdx.x;
    if (i >= d / 2) return;
    const double w = pow(theta, -2.0 * i / d);
    const double a = (double)p * w;
    tab[(size_t)p * (d / 2) + i] = make_float2((float)cos(a), (float)sin(a));
}

hipError_t launch_rope_table(float2 *tab, int max_pos, int d, double theta, hipStream_t st)
{
    KLAUNCH(k_rope_table, dim3(max_pos), dim3(64), 0, st, tab, d, theta);
    return hipGetLastError();
}

__global__ void k_fill_u32(uint32_t *p, long long n, uint32_t v)
{
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x)
        p[i] = v;
}

hipError_t launch_fill_u32(uint32_t *p, long long n_words, uint32_t v, hipStream_t st)
{
    if (n_words <= 0) return hipSuccess;
    long long blocks = (n_words + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    KLAUNCH(k_fill_u32, dim3((unsigned)blocks), dim3(256), 0, st, p, n_words, v);
    return hipGetLastError();
}

// Tile-packed copy of a row-major [N, K] weight: P[nt][kb][r][c] =
// W[nt * 128 + r][kb * 64 + c], zero for rows past N.  One thread per
// 16 bytes of P.
__global__ void k_pack_weights(const uint16_t *__restrict__ W, int N, int K, uint16_t *__restrict__ P,
                               long long units, int half)
{
    const int kt = K / 64;
    for (long long u = (long long)blockIdx.x * blockDim.x + threadIdx.x; u < units;
         u += (long long)gridDim.x * blockDim.x) {
        const int c8 = (int)(u & 7), r = (int)((u >> 3) & 127);
        const long long tile = u >> 10, nt = tile / kt;
        const int kb = (int)(tile % kt);
        // interleaved: rows 0..63 of tile nt are rows 64 nt.. of the first
        // half, rows 64..127 the same rows of the second half
        const long long row = half > 0 ? (r < 64 ? 0 : half) + nt * 64 + (r & 63) : nt * 128 + r;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (row < N) v = *reinterpret_cast<const uint4 *>(W + row * K + kb * 64 + 8 * c8);
        reinterpret_cast<uint4 *>(P)[u] = v;
    }
}

size_t packed_weight_elems(int N, int K) { return (size_t)(N + 127) / 128 * 128 * K; }

hipError_t launch_pack_weights(const uint16_t *W, int N, int K, uint16_t *P, hipStream_t st, bool interleave)
{
    if (N <= 0 || K <= 0 || K % 64 != 0 || (interleave && N % 128 != 0)) return hipErrorInvalidValue;
    const long long units = (long long)packed_weight_elems(N, K) / 8;
    long long blocks = (units + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    KLAUNCH(k_pack_weights, dim3((unsigned)blocks), dim3(256), 0, st, W, N, K, P, units,
                       interleave ? N / 2 : 0);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Small-batch projections (M <= 16 rows) from a fragment-packed weight copy.
//
// Fragment-packed layout (launch_pack_frag): [N / 16][ceil(K / 32)][64][8]
// bf16, where lane l of (column tile t, K block b) holds the eight weights
// W[row(t, l % 16)][32 b + 8 (l / 16) .. +7] -- exactly the B operand of
// v_mfma_f32_16x16x32_bf16 for 16 output columns and 32 K elements, K past
// the weight's width zero.  One wavefront load then reads 1 KB of contiguous
// memory (eight whole 128-byte lines) straight into the fragment registers:
// no LDS staging and no 16-rows-of-64-bytes access, which caps a stream
// near 4.7 TB/s.  row(t, r) is the identity (16 t + r), or pairs columns so
// that an epilogue finds both halves of an operation in lanes r and r ^ 8:
//  * rotation pairs (qkv): tile t = (head t / (d / 16), a = t % (d / 16))
//    holds head elements 8 a .. 8 a + 7 in rows 0..7 and d / 2 + 8 a .. +7
//    in rows 8..15;
//  * gate/up ([2F, K], gate rows first): rows 0..7 of tile t are gate
//    features 8 t .. 8 t + 7, rows 8..15 the up rows of the same features.
// ---------------------------------------------------------------------------
__global__ void k_pack_frag(const uint16_t *__restrict__ W, int N, int K, int mode, int d,
                            uint4 *__restrict__ P, long long units)
{
    const int nkb = (K + 31) / 32;
    for (long long u = (long long)blockIdx.x * blockDim.x + threadIdx.x; u < units;
         u += (long long)gridDim.x * blockDim.x) {
        const int l = (int)(u & 63), r = l & 15, c = l >> 4;
        const long long tb = u >> 6, t = tb / nkb;
        const int kb = (int)(tb % nkb);
        long long row;
        if (mode == 1) {
            const int per = d / 16;
            const long long hd = t / per;
            const int a = (int)(t % per);
            row = hd * d + (r < 8 ? 8 * a + r : d / 2 + 8 * a + (r - 8));
        } else if (mode == 2) {
            row = r < 8 ? 8 * t + r : N / 2 + 8 * t + (r - 8);
        } else {
            row = 16 * t + r;
        }
        const int k0 = 32 * kb + 8 * c;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (k0 < K) v = *reinterpret_cast<const uint4 *>(W + row * K + k0);
        P[u] = v;
    }
}

size_t frag_packed_elems(int N, int K) { return (size_t)N * ((K + 31) / 32 * 32); }

hipError_t launch_pack_frag(const uint16_t *W, int N, int K, int mode, int d, uint16_t *P, hipStream_t st)
{
    if (N <= 0 || K <= 0 || N % 16 != 0 || K % 8 != 0) return hipErrorInvalidValue;
    if (mode == 1 && (d % 16 != 0 || N % d != 0)) return hipErrorInvalidValue;
    const long long units = (long long)frag_packed_elems(N, K) / 8;
    long long blocks = (units + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    KLAUNCH(k_pack_frag, dim3((unsigned)blocks), dim3(256), 0, st, W, N, K, mode, d,
            reinterpret_cast<uint4 *>(P), units);
    return hipGetLastError();
}

// The projection.  Workgroup = one 16-column tile over the whole of K: four
// wavefronts take four contiguous quarters of the K blocks and their 16 x 16
// fp32 tiles are added in wavefront order (0 + 1 + 2 + 3); every output
// element is that one fixed chain whatever its row.  Each wavefront streams
// its weights U blocks at a time, double-buffered: batch i + 1's loads are
// issued before batch i's products (and after batch i's activation loads,
// so that waiting on those never drains the weight stream).  A rows >= M
// are zero fragments and are never stored.
//
// The A operand is bf16 activations from memory, or (NORM) the RMSNorm of
// the fp32 residual: the rows' 1 / rms from the per-16-column sums of
// squares their producer wrote (each wavefront adds a row's sums lane by
// lane, then the DPP tree), then bf16(x * rstd * g) per element, the norm
// kernel's rounding, written once into LDS in fragment order while the first
// weights are in flight (2 K M bytes: unit (4 kb + c) M + m holds row m's
// elements 32 kb + 8 c .. +7).
// Epilogues (wavefront 0; lane l holds column l % 16, rows 4 (l / 16) + i):
//  GV_RESID:  x[row][col] += y (each element owned by one thread, no
//             partials), and the sum of squares of the tile's 16 new
//             values of each row (row16_sum) to ss[row][tile] for the next
//             norm;
//  GV_QKV:    bf16 rounding, rotation at the row's position, bf16 rounding
//             (the split-partials epilogue's arithmetic on one sum), q to
//             the q buffer, k and v appended to the row's cache slot;
//             padding rows write nothing;
//  GV_SWIGLU: act[row][feature] = SwiGLU of the gate and up sums.
// ---------------------------------------------------------------------------
template <int U, int EPI, bool NORM>
__global__ __launch_bounds__(256) void k_gemv(const uint4 *__restrict__ Wp, int M, int N, int K, GemvIn in,
                                              GemvOut out)
{
    extern __shared__ __attribute__((aligned(16))) uint4 hs[];
    __shared__ f32x4 red[3][64];
    __shared__ float rs[16];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int t = blockIdx.x;
    const int nkb = (K + 31) / 32;
    const int kb0 = wave * nkb / 4, kb1 = (wave + 1) * nkb / 4;
    const int r = lane & 15, c = lane >> 4;
    const bool arow = r < M;
    const uint4 *wp = Wp + (size_t)t * nkb * 64 + lane;
    const uint4 z = {0u, 0u, 0u, 0u};
    // Every load of the main loop is unconditional (clamped addresses,
    // selects instead of branches), so the wait before a batch's products
    // counts exactly the loads issued after it and leaves them in flight.
    // Blocks past the wavefront's last are clamped re-reads of it, never
    // multiplied.
    auto wload = [&](uint4 (&w)[U], int kb) {
#pragma unroll
        for (int u = 0; u < U; ++u) w[u] = wp[(size_t)min(kb + u, kb1 - 1) * 64];
    };
    const int rr = min(r, M - 1);
    auto aload = [&](uint4 (&a)[U], int kb) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = min(kb + u, kb1 - 1);
            uint4 v;
            if constexpr (NORM) {
                v = hs[(4 * k + c) * M + rr];
                a[u] = arow ? v : z;
            } else {
                const int k0 = 32 * k + 8 * c;
                v = *reinterpret_cast<const uint4 *>(in.a + (size_t)rr * in.lda + min(k0, K - 8));
                a[u] = (arow && k0 < K) ? v : z;
            }
        }
    };
    uint4 wa[U], wb[U], aa[U], ab[U];
    wload(wa, kb0);                                  // two batches of weights go out before anything else
    if constexpr (!NORM) aload(aa, kb0);
    wload(wb, kb0 + U);
    if constexpr (!NORM) aload(ab, kb0 + U);
    if constexpr (NORM) {
        for (int m = wave; m < M; m += 4) {
            const float *sr = in.ss + (size_t)m * (K / 16);
            float a = 0.f;
            for (int j = lane; 4 * j < K / 16; j += 64) {
                const float4 v = *reinterpret_cast<const float4 *>(sr + 4 * j);
                a += v.x;
                a += v.y;
                a += v.z;
                a += v.w;
            }
            a = wave_sum_dpp(a);
            if (lane == 0) rs[m] = 1.0f / sqrtf(a / (float)K + in.eps);
        }
        __syncthreads();
        const int units = (K / 8) * M;
        for (int u = threadIdx.x; u < units; u += 256) {
            const int m = u % M, k0 = 8 * (u / M);
            const float rstd = rs[m];
            const float *xr = in.x + (size_t)m * K + k0;
            const float4 x0 = *reinterpret_cast<const float4 *>(xr);
            const float4 x1 = *reinterpret_cast<const float4 *>(xr + 4);
            const uint4 gg = *reinterpret_cast<const uint4 *>(in.g + k0);
            uint4 h;
            h.x = (uint32_t)f2bf(x0.x * rstd * bf2f((uint16_t)gg.x)) |
                  ((uint32_t)f2bf(x0.y * rstd * bf2f((uint16_t)(gg.x >> 16))) << 16);
            h.y = (uint32_t)f2bf(x0.z * rstd * bf2f((uint16_t)gg.y)) |
                  ((uint32_t)f2bf(x0.w * rstd * bf2f((uint16_t)(gg.y >> 16))) << 16);
            h.z = (uint32_t)f2bf(x1.x * rstd * bf2f((uint16_t)gg.z)) |
                  ((uint32_t)f2bf(x1.y * rstd * bf2f((uint16_t)(gg.z >> 16))) << 16);
            h.w = (uint32_t)f2bf(x1.z * rstd * bf2f((uint16_t)gg.w)) |
                  ((uint32_t)f2bf(x1.w * rstd * bf2f((uint16_t)(gg.w >> 16))) << 16);
            hs[u] = h;
        }
        __syncthreads();
        aload(aa, kb0);
        aload(ab, kb0 + U);
    }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    auto mma = [&](const uint4 (&a)[U], const uint4 (&w)[U], int kb) {
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (kb + u < kb1)
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[u]),
                                                              __builtin_bit_cast(bf16x8, w[u]), acc, 0, 0, 0);
    };
    for (int kb = kb0; kb < kb1; kb += 2 * U) {
        mma(aa, wa, kb);
        wload(wa, kb + 2 * U);
        aload(aa, kb + 2 * U);
        mma(ab, wb, kb + U);
        wload(wb, kb + 3 * U);
        aload(ab, kb + 3 * U);
    }
    if (wave > 0) red[wave - 1][lane] = acc;
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int w2 = 0; w2 < 3; ++w2) {
        const f32x4 o = red[w2][lane];
        acc[0] += o[0];
        acc[1] += o[1];
        acc[2] += o[2];
        acc[3] += o[3];
    }
    if constexpr (EPI == GV_RESID) {
        const int col = 16 * t + r;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = 4 * c + i;
            float xn = 0.f;
            if (row < M) {
                float *xp = out.x + (size_t)row * N + col;
                xn = *xp + acc[i];
                *xp = xn;
            }
            const float sq = row16_sum(xn * xn);      // the tile's 16 columns of this row
            if (row < M && r == 0) out.ss[(size_t)row * (N / 16) + t] = sq;
        }
    } else if constexpr (EPI == GV_SWIGLU) {
        const int F = N / 2;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float up = __shfl_xor(acc[i], 8, 64);
            const int row = 4 * c + i;
            if (r < 8 && row < M) out.act[(size_t)row * F + 8 * t + r] = swiglu_bf16(acc[i], up);
        }
    } else {   // GV_QKV
        const int d = out.d, half = d / 2, per = d / 16;
        const int hd = t / per, e0 = 8 * (t % per) + r;
        const int nq = out.nq, nkv = out.nkv;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float other = __shfl_xor(acc[i], 8, 64);
            const int row = 4 * c + i;
            if (r >= 8 || row >= M || (out.valid != nullptr && !out.valid[row])) continue;
            const int p = out.pos[row];
            float x0 = bf2f(f2bf(acc[i]));
            float x1 = bf2f(f2bf(other));
            if (hd < nq + nkv) {
                const float2 cs = out.rope[(size_t)p * half + e0];
                const float y0 = __builtin_fmaf(x0, cs.x, -(x1 * cs.y));
                const float y1 = __builtin_fmaf(x1, cs.x, x0 * cs.y);
                x0 = y0;
                x1 = y1;
            }
            const uint16_t b0 = f2bf(x0), b1 = f2bf(x1);
            if (hd < nq) {
                uint16_t *qr = out.q + (size_t)row * nq * d + (size_t)hd * d;
                qr[e0] = b0;
                qr[e0 + half] = b1;
            } else if (hd < nq + nkv) {
                uint16_t *dst = out.kc + kv_offset(out.kv, nkv, d, row, hd - nq, p);
                dst[e0] = b0;
                dst[e0 + half] = b1;
            } else {
                const int kvh = hd - nq - nkv;
                out.vc[v_offset(out.kv, nkv, d, row, kvh, p, e0)] = b0;
                out.vc[v_offset(out.kv, nkv, d, row, kvh, p, e0 + half)] = b1;
            }
        }
    }
}

hipError_t launch_gemv(const uint16_t *Wp, int M, int N, int K, int epi, const GemvIn &in, const GemvOut &out,
                       hipStream_t st)
{
    // every wavefront gets at least one of the ceil(K / 32) K blocks
    if (M <= 0 || M > 16 || N % 16 != 0 || K % 16 != 0 || K < 128) return hipErrorInvalidValue;
    const bool norm = in.a == nullptr;
    // the normed rows live in LDS (2 K M bytes); the sums of squares come in groups of 16 x 4
    if (norm && (K % 64 != 0 || (size_t)2 * K * M > 128 * 1024)) return hipErrorInvalidValue;
    if (epi == GV_QKV && (out.d % 16 != 0 || N % out.d != 0)) return hipErrorInvalidValue;
    const dim3 grid(N / 16), block(256);
    const uint4 *W = reinterpret_cast<const uint4 *>(Wp);
    const unsigned lds = norm ? (unsigned)(2 * K * M) : 0u;
    if (norm) {   // the normed rows may exceed the default 64 KB of dynamic LDS (a host-side attribute, per device)
        hipError_t e = hipFuncSetAttribute((const void *)k_gemv<8, GV_QKV, true>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 128 * 1024);
        if (e == hipSuccess)
            e = hipFuncSetAttribute((const void *)k_gemv<8, GV_SWIGLU, true>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, 128 * 1024);
        if (e != hipSuccess) return e;
    }
    if (epi == GV_RESID && !norm)
        KLAUNCH((k_gemv<8, GV_RESID, false>), grid, block, 0, st, W, M, N, K, in, out);
    else if (epi == GV_QKV && norm)
        KLAUNCH((k_gemv<8, GV_QKV, true>), grid, block, lds, st, W, M, N, K, in, out);
    else if (epi == GV_SWIGLU && norm)
        KLAUNCH((k_gemv<8, GV_SWIGLU, true>), grid, block, lds, st, W, M, N, K, in, out);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

__global__ void k_iota(int32_t *p, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = i;
}

hipError_t launch_iota(int32_t *p, int n, hipStream_t st)
{
    KLAUNCH(k_iota, dim3((n + 255) / 256), dim3(256), 0, st, p, n);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Mixture-of-experts layer.
//
// Routing (one wavefront per row): the router logits (split partials added in
// split order), the top_k largest with ties to the lower expert id (exact
// selections), and weights exp(l_r - l_0) / sum_r' exp(l_r' - l_0) summed in
// rank order -- the renormalised top_k of a softmax over all experts.
//
// Dispatch (one workgroup): assignment a = b top_k + r goes to expert
// sel[a]; each expert's assignments are listed in increasing a, and the
// lists are cut into 16-row tiles placed, expert by expert, into a fixed
// pool of E + ceil(rows top_k / 16) tile slots -- enough for any routing, so
// no assignment is ever dropped and the launch never depends on the routing.
// A row's expert result does not depend on the tile or the tile row it lands
// in: each output element's K reduction runs in one fixed order.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_moe_route(const float *__restrict__ part, int S, long long part_stride,
                                                  int E, int top_k, const uint8_t *__restrict__ valid,
                                                  int32_t *__restrict__ sel, float *__restrict__ wsel,
                                                  int32_t *__restrict__ sel_trace, float *__restrict__ logit_trace)
{
    const int b = blockIdx.x, lane = threadIdx.x;
    if (valid != nullptr && !valid[b]) {
        if (lane < top_k) {
            sel[(size_t)b * top_k + lane] = -1;
            wsel[(size_t)b * top_k + lane] = 0.f;
            if (sel_trace != nullptr) sel_trace[(size_t)b * top_k + lane] = -1;
        }
        return;
    }
    constexpr int EPL = 4;   // E <= 256
    float l[EPL];
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
        const int e = lane + 64 * j;
        float v = -INFINITY;
        if (e < E) {   // partials in split order, loads issued in batches of up to 8
            v = 0.f;
            for (int s = 0; s < S; s += 8) {
                float p8[8];
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (s + u < S) p8[u] = part[(s + u) * part_stride + (size_t)b * E + e];
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (s + u < S) v += p8[u];
            }
        }
        l[j] = v;
        if (logit_trace != nullptr && e < E) logit_trace[(size_t)b * E + e] = v;
    }
    float top_l[16];
    int top_e[16];
    for (int r = 0; r < top_k; ++r) {
        float bv = -INFINITY;
        int bi = 0x7fffffff;
#pragma unroll
        for (int j = 0; j < EPL; ++j)
            if (lane + 64 * j < E) better(bv, bi, l[j], lane + 64 * j);
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            const float v2 = __shfl_xor(bv, off, 64);
            const int i2 = __shfl_xor(bi, off, 64);
            better(bv, bi, v2, i2);
        }
        top_l[r] = bv;
        top_e[r] = bi;
#pragma unroll
        for (int j = 0; j < EPL; ++j)
            if (lane + 64 * j == bi) l[j] = -INFINITY;    // never chosen again (NaN-free logits assumed)
    }
    if (lane == 0) {
        float z = 0.f;
        float ev[16];
        for (int r = 0; r < top_k; ++r) {
            ev[r] = __expf(top_l[r] - top_l[0]);
            z += ev[r];
        }
        for (int r = 0; r < top_k; ++r) {
            sel[(size_t)b * top_k + r] = top_e[r];
            wsel[(size_t)b * top_k + r] = ev[r] / z;
            if (sel_trace != nullptr) sel_trace[(size_t)b * top_k + r] = top_e[r];
        }
    }
}

hipError_t launch_moe_route(const float *part, int S, long long part_stride, int rows, int E, int top_k,
                            const uint8_t *valid, int32_t *sel, float *wsel, hipStream_t st, int32_t *sel_trace,
                            float *logit_trace)
{
    if (E > 256 || top_k > 16 || top_k > E) return hipErrorInvalidValue;
    KLAUNCH(k_moe_route, dim3(rows), dim3(64), 0, st, part, S, part_stride, E, top_k, valid, sel, wsel,
                       sel_trace, logit_trace);
    return hipGetLastError();
}

// tiles[slot] = {expert, first list index, count}; count 0 = unused slot.
// Dispatch: counts per expert (integer LDS atomics: order-independent), an
// exclusive scan over experts for list and tile offsets, tiles written by
// their expert's thread, then assignments ranked 1024 at a time: each
// expert's assignments of the chunk set their bit in the expert's 1024-bit
// mask, and an assignment's rank among its expert's is the popcount below
// its bit plus what earlier chunks placed.  Every output is a function of
// sel alone.
__global__ __launch_bounds__(1024) void k_moe_dispatch(const int32_t *__restrict__ sel, int n_assign, int E,
                                                       int n_slots, int32_t *__restrict__ list,
                                                       int32_t *__restrict__ tiles)
{
    __shared__ int cnt[256], base[256], toff[257], scan_v[256], scan_w[256];
    __shared__ uint32_t mask[256 * 32];
    const int tid = threadIdx.x;
    if (tid < 256) cnt[tid] = 0;
    __syncthreads();
    for (int a = tid; a < n_assign; a += 1024) {
        const int e = sel[a];
        if (e >= 0) atomicAdd(&cnt[e], 1);
    }
    __syncthreads();
    // exclusive scans of counts and tile counts over the experts (Hillis-Steele)
    const int c = tid < E ? cnt[tid] : 0, nt = (c + 15) / 16;
    int v = c, w = nt;
    for (int off = 1; off < 256; off <<= 1) {
        if (tid < 256) {
            scan_v[tid] = v;
            scan_w[tid] = w;
        }
        __syncthreads();
        if (tid < 256 && tid >= off) {
            v += scan_v[tid - off];
            w += scan_w[tid - off];
        }
        __syncthreads();
    }
    if (tid < 256) {
        base[tid] = v - c;
        toff[tid] = w - nt;
        if (tid == 255) toff[256] = w;
    }
    __syncthreads();
    if (tid < E)
        for (int j = 0; j < nt; ++j) {
            const int slot = toff[tid] + j;
            tiles[3 * slot + 0] = tid;
            tiles[3 * slot + 1] = base[tid] + 16 * j;
            tiles[3 * slot + 2] = min(16, c - 16 * j);
        }
    for (int slot = toff[256] + tid; slot < n_slots; slot += 1024) {
        tiles[3 * slot + 0] = 0;
        tiles[3 * slot + 1] = 0;
        tiles[3 * slot + 2] = 0;
    }
    for (int c0 = 0; c0 < n_assign; c0 += 1024) {
        for (int i = tid; i < 256 * 32; i += 1024) mask[i] = 0u;
        __syncthreads();
        const int a = c0 + tid;
        const int e = a < n_assign ? sel[a] : -1;
        if (e >= 0) atomicOr(&mask[e * 32 + (tid >> 5)], 1u << (tid & 31));
        __syncthreads();
        if (e >= 0) {
            int rank = __popc(mask[e * 32 + (tid >> 5)] & ((1u << (tid & 31)) - 1u));
            for (int j = 0; j < (tid >> 5); ++j) rank += __popc(mask[e * 32 + j]);
            list[base[e] + rank] = a;
        }
        __syncthreads();
        if (tid < E) {   // advance each expert's base past this chunk's assignments
            int n = 0;
            for (int j = 0; j < 32; ++j) n += __popc(mask[tid * 32 + j]);
            base[tid] += n;
        }
        __syncthreads();
    }
}

hipError_t launch_moe_dispatch(const int32_t *sel, int n_assign, int E, int n_slots, int32_t *list, int32_t *tiles,
                               hipStream_t st)
{
    if (E > 256) return hipErrorInvalidValue;
    KLAUNCH(k_moe_dispatch, dim3(1), dim3(1024), 0, st, sel, n_assign, E, n_slots, list, tiles);
    return hipGetLastError();
}

// Expert projection on one 16-row tile of assignments: row r of the tile is
// assignment list[start + r]; its A row is A[assignment / row_div]; the
// output row is the assignment.  Same MFMA lane layout and pipelining as
// k_gemm with one 16-row M tile; no split-K.
template <int NT, int KU>
__global__ __launch_bounds__(256) void k_moe_gemm(const uint16_t *__restrict__ A, int lda, int row_div,
                                                  const uint16_t *__restrict__ Wbase, long long w_expert_stride,
                                                  int N, int K, const int32_t *__restrict__ list,
                                                  const int32_t *__restrict__ tiles, float *__restrict__ out, int ldo)
{
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int r = lane & 15, kg = lane >> 4;
    const int slot = blockIdx.y;
    const int cnt = tiles[3 * slot + 2];
    if (cnt == 0) return;
    const int expert = tiles[3 * slot + 0], start = tiles[3 * slot + 1];
    const int ncb = (N + 16 * NT - 1) / (16 * NT);
    const int cb = blockIdx.x * 4 + wave;
    if (cb >= ncb) return;
    const int n0 = cb * 16 * NT;
    const int nvalid = min(NT, (N - n0) / 16);
    const uint16_t *W = Wbase + (size_t)expert * w_expert_stride;
    const bool arow = r < cnt;
    const int my_a = arow ? list[start + r] : 0;
    const uint16_t *ap = A + (size_t)(my_a / row_div) * lda + kg * 8;
    const uint16_t *wp[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) wp[nt] = W + (size_t)(n0 + 16 * min(nt, nvalid - 1) + r) * K + kg * 8;
    f32x4 acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] = (f32x4){0.f, 0.f, 0.f, 0.f};
    const uint4 z = {0u, 0u, 0u, 0u};
    int k = 0;
    for (; k + 32 * KU <= K; k += 32 * KU) {
        bf16x8 wf[NT][KU], af[KU];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int u = 0; u < KU; ++u) wf[nt][u] = __builtin_bit_cast(bf16x8, *(const uint4 *)(wp[nt] + k + 32 * u));
#pragma unroll
        for (int u = 0; u < KU; ++u) {
            uint4 v = z;
            if (arow) v = *(const uint4 *)(ap + k + 32 * u);
            af[u] = __builtin_bit_cast(bf16x8, v);
        }
#pragma unroll
        for (int u = 0; u < KU; ++u)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[u], wf[nt][u], acc[nt], 0, 0, 0);
    }
    for (; k < K; k += 32) {
        const bool in = (k + kg * 8) < K;
        bf16x8 wf[NT], af;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            uint4 v = z;
            if (in) v = *(const uint4 *)(wp[nt] + k);
            wf[nt] = __builtin_bit_cast(bf16x8, v);
        }
        {
            uint4 v = z;
            if (in && arow) v = *(const uint4 *)(ap + k);
            af = __builtin_bit_cast(bf16x8, v);
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, wf[nt], acc[nt], 0, 0, 0);
    }
    // output rows: tile row 4 kg + i holds assignment list[start + 4 kg + i]
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int tr = kg * 4 + i;
        if (tr < cnt) {
            const int a = list[start + tr];
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                if (nt < nvalid) out[(size_t)a * ldo + n0 + 16 * nt + r] = acc[nt][i];
        }
    }
}

hipError_t launch_moe_gemm(const uint16_t *A, int lda, int row_div, const uint16_t *W, long long w_expert_stride, int N,
                           int K, const int32_t *list, const int32_t *tiles, int n_slots, float *out, int ldo,
                           hipStream_t st)
{
    constexpr int NT = 4;
    const int ncb = (N + 16 * NT - 1) / (16 * NT);
    KLAUNCH((k_moe_gemm<NT, 4>), dim3((ncb + 3) / 4, n_slots), dim3(256), 0, st, A, lda, row_div, W,
                       w_expert_stride, N, K, list, tiles, out, ldo);
    return hipGetLastError();
}

hipError_t launch_moe_gemm_dma(const uint16_t *A, int lda, int row_div, const uint16_t *W, long long w_expert_stride,
                               bool packed, int N, int K, const int32_t *list, const int32_t *tiles, int n_slots,
                               float *out, uint16_t *act, int ldo, hipStream_t st)
{
    if (K % 64 != 0 || N <= 0 || (act != nullptr && (!packed || N % 128 != 0))) return hipErrorInvalidValue;
    const ExpertTiles et{list, tiles, row_div, w_expert_stride};
    const dim3 grid((N + 127) / 128, n_slots);
    if (act != nullptr)
        KLAUNCH((k_gemm_dma<32, 128, 64, 4, 1, 2, true, true, true>), grid, dim3(128), 0, st, A, lda, W, 16,
                           N, K, K, nullptr, 0, ldo, nullptr, act, et);
    else if (packed)
        KLAUNCH((k_gemm_dma<32, 128, 64, 4, 1, 2, true, false, true>), grid, dim3(128), 0, st, A, lda, W,
                           16, N, K, K, out, 0, ldo, nullptr, nullptr, et);
    else
        KLAUNCH((k_gemm_dma<32, 128, 64, 4, 1, 2, false, false, true>), grid, dim3(128), 0, st, A, lda, W,
                           16, N, K, K, out, 0, ldo, nullptr, nullptr, et);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Causal attention of the isolated prefill (flash-style, no split): the
// prompt runs alone, so any fixed order is allowed; this one takes, for every
// query, the keys in tiles of 64 in increasing order with the online softmax.
// A chunk of a longer prompt (chunked prefill) has its queries at positions
// p0 .. p0 + n - 1 and reads the keys of positions before p0 from the cache,
// where the prompt's earlier chunks wrote them; p0 = 0 is the whole prompt.
//
// Work units of one KV head: (block of 32 queries, one query head of the
// group).  A workgroup of eight wavefronts (two per SIMD, so one wavefront's
// softmax runs while the other's matrix products do) takes eight consecutive
// units in [block][head] order, latest blocks first, one per wavefront; the
// eight share key and value tiles ([key][d] rows, as the cache stores them),
// streamed global -> LDS by direct 16-byte
// loads through a ring of three stages (one tile in use, two in flight),
// waited on with a fixed vmcnt.
//  * S^T = K Q^T on v_mfma_f32_32x32x16_bf16, two 32-key x 32-query tiles;
//    MFMA row m carries key pk(m) (bits 2 and 3 of m swapped), so lane l
//    ends holding, for query l % 32, the eight consecutive keys
//    16 s + 8 (l / 32) .. +7 of each 16-key step s -- exactly the P^T
//    operand of
//  * O^T += V^T P^T on the same instruction: its V^T operand (eight keys of
//    one dimension) comes from the value rows by two transposed LDS reads.
// Each lane's O^T values belong to one query, so the softmax max and sum
// need one exchange between the two lane halves and the rescale is a
// per-lane scalar, skipped when no lane's maximum moved.  P enters the matrix
// core rounded to bf16; the row sum adds the rounded values (bf16 dot).  Keys
// past the prompt load clamped (real) rows: their scores are masked to -inf
// by selection, and their values are zeroed in LDS in the last, partial
// tile, so nothing stale in the cache reaches the sums.  The output goes
// back through LDS for row-contiguous stores.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int pf_key_of_row(int m) { return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1); }

template <int KC>
__device__ __forceinline__ int pf_swz(int r, int c)
{
    // KC 16-byte chunks per row: 16 (256-byte rows) or 8 (128-byte rows)
    if constexpr (KC == 16) return r * 16 + (c ^ (r & 15));
    else return r * 8 + (c ^ ((r >> 1) & 7));
}

// One workgroup of the kernel: kv head kvh, unit group grp of one prompt.
template <int D>
__device__ __forceinline__ void prefill_attn_block(const uint16_t *__restrict__ q, int n, int p0, int nq, int nkv,
                                                   int slot, const uint16_t *__restrict__ kc,
                                                   const uint16_t *__restrict__ vc, const KvView &kv,
                                                   uint16_t *__restrict__ o, int kvh, int grp)
{
    constexpr int NW = 8, NT = 64 * NW;              // wavefronts, threads
    constexpr int QB = 32, BKT = 64;                  // queries per wavefront, keys per tile
    constexpr int DT = D / 32, KS = D / 16;           // 32-dim output tiles, 16-dim score steps
    constexpr int KCH = D / 8;                        // 16-byte chunks per key row
    constexpr int K_OPS = BKT * KCH / NT, V_OPS = BKT * KCH / NT, OPS = K_OPS + V_OPS;
    constexpr int NST = 3, P = NST - 1;
    constexpr int KSTAGE = BKT * KCH, STAGE = 2 * KSTAGE;     // 16-byte units: key rows, then value rows
    constexpr int OPITCH = D + 8;                     // output staging row (elements)
    static_assert(K_OPS >= 1 && V_OPS >= 1, "tile loads cover the workgroup");
    static_assert(NW * QB * OPITCH * 2 <= NST * STAGE * 16, "output staging fits the ring");
    __shared__ __attribute__((aligned(16))) uint4 ring[NST * STAGE];
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

    const int G = nq / nkv;
    // queries are the n positions p0 .. p0 + n - 1 (q and o rows 0 .. n - 1);
    // keys are positions 0 .. Lk - 1 of the slot's cache, the first p0 of
    // them written by earlier chunks of the same prompt
    const int Lk = p0 + n;
    // grid (kv head, unit group): workgroups are dispatched x fastest, so the
    // groups with the latest (longest) query blocks of every kv head go first
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int r32 = lane & 31, h = lane >> 5;
    const int nqb = (n + QB - 1) / QB;
    const int units = nqb * G;
    const int u = units - 1 - (grp * NW + wave);                // latest blocks first
    const bool active = u >= 0;
    const int qb = active ? u / G : 0, g = active ? u % G : 0;
    const int hq = kvh * G + g;
    const int q0 = qb * QB;                                     // chunk row of the block's first query
    const int u_first = units - 1 - grp * NW;
    const int wg_last_q = p0 + min(n, (u_first / G + 1) * QB) - 1;
    const int my_last_q = active ? p0 + min(n, q0 + QB) - 1 : -1;
    const int ntiles = __builtin_amdgcn_readfirstlane(wg_last_q / BKT + 1);   // uniform: scalar branches

    // tile loads: op j of thread t is 16-byte unit 512 j + t of the K part
    // or of the V part (token-major both, row = unit / KCH)
    typedef __attribute__((address_space(3))) void lds_void;
    auto issue = [&](int slot_, int k0) {
        uint4 *base = ring + slot_ * STAGE + wave * 64;
#pragma unroll
        for (int j = 0; j < K_OPS; ++j) {
            const int gi = j * NT + tid, r = gi / KCH, c = pf_swz<KCH>(r, gi % KCH) - r * KCH;
            const int key = min(k0 + r, Lk - 1);
            __builtin_amdgcn_global_load_lds((const void *)(kc + kv_offset(kv, nkv, D, slot, kvh, key) + 8 * c),
                                             (lds_void *)(base + j * NT), 16, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < V_OPS; ++j) {
            const int gi = j * NT + tid, r = gi / KCH, c = (gi % KCH) ^ vtile_swz<KCH>(r);
            const int key = min(k0 + r, Lk - 1);
            __builtin_amdgcn_global_load_lds((const void *)(vc + kv_offset(kv, nkv, D, slot, kvh, key) + 8 * c),
                                             (lds_void *)(base + KSTAGE + j * NT), 16, 0, 0);
        }
    };

    // Q^T operand: lane l supplies query q0 + l % 32, dims 16 s + 8 (l / 32) .. +7
    bf16x8 qf[KS];
    {
        const int qq = q0 + r32;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            uint4 v = {0u, 0u, 0u, 0u};
            if (active && qq < n) v = *(const uint4 *)(q + (size_t)qq * nq * D + (size_t)hq * D + 16 * ks + 8 * h);
            qf[ks] = __builtin_bit_cast(bf16x8, v);
        }
    }
    f32x16 acc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int j = 0; j < 16; ++j) acc[dt][j] = 0.f;
    float mrow = -INFINITY, lpart = 0.f;
    const float scale2 = 1.4426950408889634f / sqrtf((float)D);   // log2(e) / sqrt(d)
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
    const int qq = p0 + q0 + r32;                     // this lane's query position

    // P stages go out whatever the tile count: a stage past the last tile
    // loads clamped (real) rows into a slot that no tile reads, and the wait
    // after the loop drains it.  So one constant wait here completes the q
    // fragments (loaded before the stages; vmcnt retires in order).  Without
    // it the compiler, unable to tell on entry to the loop whether they had
    // landed, waited for every load in flight (the whole ring) before each
    // tile's score products.
#pragma unroll
    for (int i = 0; i < P; ++i) issue(i, i * BKT);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(P * OPS));
    for (int i = 0; i < ntiles; ++i) {
        wait_stages<OPS, P - 1>(min(P - 1, ntiles - 1 - i));
        lds_barrier();
        const int k0 = i * BKT;
        uint4 *Kt = ring + (i % NST) * STAGE;
        uint4 *Vt = Kt + KSTAGE;
        if (k0 + BKT > Lk) {
            // last tile: zero the value rows of keys past the prompt
            const uint4 z = {0u, 0u, 0u, 0u};
            for (int it = tid; it < BKT * KCH; it += NT)
                if (k0 + it / KCH >= Lk) Vt[it] = z;
            lds_barrier();
        }
        if (i + P < ntiles) issue((i + P) % NST, (i + P) * BKT);
        if (k0 > my_last_q) continue;                 // wave-uniform: the whole tile is in this unit's future

        f32x16 st[2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int j = 0; j < 16; ++j) st[kt][j] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int kt = 0; kt < 2; ++kt) {
                const bf16x8 kf = __builtin_bit_cast(bf16x8, Kt[pf_swz<KCH>(32 * kt + pf_key_of_row(r32), 2 * ks + h)]);
                st[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], st[kt], 0, 0, 0);
            }
        // online softmax in base 2; lane holds keys k0 + 32 kt + 16 (j / 8) + 8 h + j % 8
        // of query qq; only tiles reaching past the wavefront's first query or
        // past the prompt need the mask
        float mt = -INFINITY;
        if (k0 + BKT - 1 > p0 + q0 || k0 + BKT > Lk) {
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const int key = k0 + 32 * kt + 16 * (j >> 3) + 8 * h + (j & 7);
                    const float sv = (key <= qq && key < Lk) ? st[kt][j] : -INFINITY;
                    st[kt][j] = sv;
                    mt = fmaxf(mt, sv);
                }
        } else {
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int j = 0; j < 16; ++j) mt = fmaxf(mt, st[kt][j]);
        }
        mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
        // running maximum in scaled units (scale2 > 0 keeps the order)
        const float mnew = fmaxf(mrow, mt * scale2);
        // a query with no visible key yet keeps mnew = -inf: its weights are 0
        const float moff = mnew == -INFINITY ? 0.f : mnew;
        float ls = 0.f;
        bf16x8 pf[4];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                uint32_t w[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    w[e] = f2bf2(__builtin_amdgcn_exp2f(__builtin_fmaf(st[kt][8 * half + 2 * e], scale2, -moff)),
                                 __builtin_amdgcn_exp2f(__builtin_fmaf(st[kt][8 * half + 2 * e + 1], scale2, -moff)));
                    ls = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), ones, ls, false);   // the rounded weights
                }
                pf[2 * kt + half] = __builtin_bit_cast(bf16x8, (uint4){w[0], w[1], w[2], w[3]});
            }
        // rescale only when some lane's maximum moved (alpha == 1 exactly otherwise)
        if (__ballot(mnew != mrow)) {
            const float alpha = mnew == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(mrow - mnew);
            lpart *= alpha;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int j = 0; j < 16; ++j) acc[dt][j] *= alpha;
        }
        lpart += ls;
        mrow = mnew;
        // O^T += V^T P^T over the tile's four 16-key steps.  The V^T operand
        // (lane l: dimension 32 dt + l % 32, keys 16 s16 + 8 h .. +7) comes
        // from the token-major value rows by two transposed reads per
        // 16-lane group (keys 4 r + 0..3): lane a + 4 q of the group points
        // at key 16 s16 + 8 h + 4 r + q, dimensions 32 dt + 16 (l / 16 % 2)
        // + 4 a ..
#pragma unroll
        for (int s16 = 0; s16 < 4; ++s16)
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const int a = lane & 3, qv = (lane >> 2) & 3, half16 = (lane >> 4) & 1;
                uint2 part[2];
#pragma unroll
                for (int r = 0; r < 2; ++r) {
                    const int key = 16 * s16 + 8 * h + 4 * r + qv;
                    const int c = 4 * dt + 2 * half16 + (a >> 1);
                    part[r] = lds_read_tr16(reinterpret_cast<const char *>(Vt + key * KCH + (c ^ vtile_swz<KCH>(key))) +
                                            8 * (a & 1));
                }
                const bf16x8 vf = __builtin_bit_cast(bf16x8, (uint4){part[0].x, part[0].y, part[1].x, part[1].y});
                acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[s16], acc[dt], 0, 0, 0);
            }
    }
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    lds_barrier();                                    // every wavefront is done with the ring

    // lane holds O^T[d = 32 dt + 8 (j / 4) + 4 h + j % 4][query l % 32]:
    // normalise, round, stage as [query][d] rows, store rows contiguously
    uint16_t *ost = (uint16_t *)ring + (size_t)wave * QB * OPITCH;
    {
        float L = lpart;
        L += __shfl_xor(L, 32, 64);
        const float inv = 1.0f / L;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int j = 0; j < 16; ++j)
                ost[r32 * OPITCH + 32 * dt + 8 * (j >> 2) + 4 * h + (j & 3)] = f2bf(acc[dt][j] * inv);
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);               // lgkmcnt(0): this wavefront's staging writes are done
    if (!active) return;
#pragma unroll 4
    for (int it = lane; it < QB * (D / 8); it += 64) {
        const int qr = it / (D / 8), c8 = it % (D / 8);
        const int qo = q0 + qr;
        if (qo < n)
            *(uint4 *)(o + (size_t)qo * nq * D + (size_t)hq * D + 8 * c8) = *(const uint4 *)(ost + qr * OPITCH + 8 * c8);
    }
}

template <int D>
__global__ __launch_bounds__(512) void k_prefill_attn(const uint16_t *__restrict__ q, int n, int p0, int nq, int nkv,
                                                      int slot, const uint16_t *__restrict__ kc,
                                                      const uint16_t *__restrict__ vc, KvView kv,
                                                      uint16_t *__restrict__ o)
{
    prefill_attn_block<D>(q, n, p0, nq, nkv, slot, kc, vc, kv, o, blockIdx.x, blockIdx.y);
}

// Several prompts in one launch (batched prefill): prompt i owns rows
// seq[i].row0 .. + len of q and o and the cache of seq[i].slot; the unit
// groups of all prompts follow one another along the grid's y, prompt i's
// starting at seq[i].grp0.  Each workgroup runs exactly the arithmetic of the
// same unit in the prompt's own launch.
template <int D>
__global__ __launch_bounds__(512) void k_prefill_attn_multi(const uint16_t *__restrict__ q,
                                                            const int32_t *__restrict__ seq, int nseq, int nq,
                                                            int nkv, const uint16_t *__restrict__ kc,
                                                            const uint16_t *__restrict__ vc, KvView kv,
                                                            uint16_t *__restrict__ o)
{
    const int g = blockIdx.y;
    int i = 0;
    while (i + 1 < nseq && seq[4 * (i + 1) + 3] <= g) ++i;
    const int row0 = seq[4 * i], len = seq[4 * i + 1], slot = seq[4 * i + 2], grp = g - seq[4 * i + 3];
    const size_t ofs = (size_t)row0 * nq * D;
    prefill_attn_block<D>(q + ofs, len, 0, nq, nkv, slot, kc, vc, kv, o + ofs, blockIdx.x, grp);
}

hipError_t launch_prefill_attn_multi(const uint16_t *q, const int32_t *seq, int nseq, int total_groups, int nq,
                                     int nkv, int d, const uint16_t *kc, const uint16_t *vc, KvView kv, uint16_t *o,
                                     hipStream_t st)
{
    if (nseq <= 0 || total_groups <= 0) return hipErrorInvalidValue;
    dim3 grid(nkv, total_groups);
    if (d == 128)
        KLAUNCH((k_prefill_attn_multi<128>), grid, dim3(512), 0, st, q, seq, nseq, nq, nkv, kc, vc, kv, o);
    else if (d == 64)
        KLAUNCH((k_prefill_attn_multi<64>), grid, dim3(512), 0, st, q, seq, nseq, nq, nkv, kc, vc, kv, o);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

// Row seq[i].row0 + seq[i].len - 1 of src (bf16 [.][H]) to row i of dst: the
// last position of every prompt of a batched prefill.
__global__ __launch_bounds__(256) void k_gather_last_rows(const uint16_t *__restrict__ src, const int32_t *__restrict__ seq,
                                                          int H, uint16_t *__restrict__ dst)
{
    const int i = blockIdx.x;
    const size_t row = (size_t)seq[4 * i] + seq[4 * i + 1] - 1;
    for (int c = threadIdx.x; c < H / 8; c += 256)
        *(uint4 *)(dst + (size_t)i * H + 8 * c) = *(const uint4 *)(src + row * H + 8 * c);
}

hipError_t launch_gather_last_rows(const uint16_t *src, const int32_t *seq, int n, int H, uint16_t *dst, hipStream_t st)
{
    if (n <= 0 || H % 8) return hipErrorInvalidValue;
    KLAUNCH(k_gather_last_rows, dim3(n), dim3(256), 0, st, src, seq, H, dst);
    return hipGetLastError();
}

hipError_t launch_prefill_attn(const uint16_t *q, int n, int p0, int nq, int nkv, int d, int slot, const uint16_t *kc,
                               const uint16_t *vc, KvView kv, uint16_t *o, hipStream_t st)
{
    if (n <= 0 || p0 < 0) return hipErrorInvalidValue;
    const int G = nq / nkv;
    const int units = ((n + 31) / 32) * G;
    dim3 grid(nkv, (units + 7) / 8);
    if (d == 128)
        KLAUNCH((k_prefill_attn<128>), grid, dim3(512), 0, st, q, n, p0, nq, nkv, slot, kc, vc, kv, o);
    else if (d == 64)
        KLAUNCH((k_prefill_attn<64>), grid, dim3(512), 0, st, q, n, p0, nq, nkv, slot, kc, vc, kv, o);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Request-bound seeded sampling: token = argmax_v (l_v / T + g_v) (the
// Gumbel-max rule, an exact draw from softmax(l / T)), g_v = -ln(-ln u_v),
// u_v from Philox4x32-10 keyed by the request's 64-bit seed with counter
// (t, v, 0, 0), t = the position of the token being sampled.  The variate is
// a function of (seed, t, v) only: no state is consumed, so padding rows and
// co-runners cannot shift a request's stream.  T <= 0 is greedy.  Decision
// and log-probability (of the chosen token under softmax(l / T), softmax(l)
// when greedy) in fp64; reductions in a fixed tree over 1024 threads:
// sequential per thread over its columns, then the 64-lane butterfly, then
// the 16 wavefronts in order.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1)
{
    // Salmon et al., SC 2011: per round (c0, c1, c2, c3) <- (hi(M1 c2) ^ c1 ^ k0,
    // lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0)); key += (W0, W1) between rounds
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint32_t lo0 = 0xD2511F53u * c[0], hi0 = __umulhi(0xD2511F53u, c[0]);
        const uint32_t lo1 = 0xCD9E8D57u * c[2], hi1 = __umulhi(0xCD9E8D57u, c[2]);
        const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
        c[0] = n0;
        c[1] = lo1;
        c[2] = n2;
        c[3] = lo0;
    }
}

__device__ __forceinline__ double gumbel_noise(uint32_t k0, uint32_t k1, int t, int v)
{
    uint32_t c[4] = {(uint32_t)t, (uint32_t)v, 0u, 0u};
    philox4x32_10(c, k0, k1);
    // u strictly inside (0, 1): ((c0 >> 6) 2^26 + (c1 >> 6) + 1/2) 2^-52, in
    // [2^-53, 1 - 2^-53], every value exact (53-bit integer part)
    const double u = ((double)(c[0] >> 6) * 67108864.0 + (double)(c[1] >> 6) + 0.5) * (1.0 / 4503599627370496.0);
    return -log(-log(u));
}

__device__ __forceinline__ void better_d(double &v, int &i, double v2, int i2)
{
    if (v2 > v || (v2 == v && i2 < i)) {
        v = v2;
        i = i2;
    }
}

__global__ __launch_bounds__(1024) void k_sample(const float *__restrict__ logits, long long ld, int V,
                                                 const uint8_t *__restrict__ valid, const int32_t *__restrict__ pos,
                                                 const uint64_t *__restrict__ seed, const float *__restrict__ temp,
                                                 int32_t *__restrict__ token, float *__restrict__ logprob)
{
    const int r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (!valid[r]) {
        if (tid == 0) {
            token[r] = -1;
            logprob[r] = 0.f;
        }
        return;
    }
    __shared__ double sz[16], sm[16];
    __shared__ int si[16];
    const float *l = logits + (size_t)r * ld;
    const float tf = temp[r];
    const bool greedy = !(tf > 0.0f);
    const double T = greedy ? 1.0 : (double)tf;
    const uint32_t k0 = (uint32_t)seed[r], k1 = (uint32_t)(seed[r] >> 32);
    const int t = pos[r];
    double bz = -INFINITY, M = -INFINITY;
    int bi = 0x7fffffff;
    for (int v = tid; v < V; v += 1024) {
        const double x = (double)l[v] / T;
        const double z = greedy ? x : x + gumbel_noise(k0, k1, t, v);
        better_d(bz, bi, z, v);
        M = fmax(M, x);
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        better_d(bz, bi, __shfl_xor(bz, off, 64), __shfl_xor(bi, off, 64));
        M = fmax(M, __shfl_xor(M, off, 64));
    }
    if (lane == 0) {
        sz[wave] = bz;
        si[wave] = bi;
        sm[wave] = M;
    }
    __syncthreads();
    bz = sz[0];
    bi = si[0];
    M = sm[0];
    for (int w = 1; w < 16; ++w) {
        better_d(bz, bi, sz[w], si[w]);
        M = fmax(M, sm[w]);
    }
    double S = 0.0;
    for (int v = tid; v < V; v += 1024) S += exp((double)l[v] / T - M);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) S += __shfl_xor(S, off, 64);
    __syncthreads();                                  // every thread has read sz/si/sm
    if (lane == 0) sm[wave] = S;
    __syncthreads();
    if (tid == 0) {
        double Ssum = 0.0;
        for (int w = 0; w < 16; ++w) Ssum += sm[w];
        token[r] = bi;
        logprob[r] = (float)((double)l[bi] / T - M - log(Ssum));
    }
}

hipError_t launch_sample(const float *logits, long long ld, int rows, int V, const uint8_t *valid, const int32_t *pos,
                         const uint64_t *seed, const float *temp, int32_t *token, float *logprob, hipStream_t st)
{
    if (rows <= 0 || V <= 0) return hipErrorInvalidValue;
    KLAUNCH(k_sample, dim3(rows), dim3(1024), 0, st, logits, ld, V, valid, pos, seed, temp, token,
                       logprob);
    return hipGetLastError();
}

hipError_t launch_proj(const uint16_t *A, int lda, const uint16_t *W, const GemmShape &g, float *out,
                       long long split_stride, int ldo, hipStream_t st, ArgBest *amax)
{
    if (g.bn > 0) return launch_gemm_dma(A, lda, W, g, out, split_stride, ldo, st, amax);
    if (g.bm > 0) return launch_gemm_tiled(A, lda, W, g, g.bm, out, split_stride, ldo, st, amax);
    return launch_gemm(A, lda, W, g, out, split_stride, ldo, st, amax);
}

}  // namespace corun
