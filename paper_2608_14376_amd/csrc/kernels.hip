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

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 -> bf16, round to nearest even; NaN stays NaN (quieted).
__device__ __forceinline__ uint16_t f2bf(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Fixed butterfly over the 64 lanes, then lane 0's value to every lane.
__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return __shfl(v, 0, 64);
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

__device__ __forceinline__ int row_slot(const int32_t *slot_of_row, int slot_const, int r)
{
    return slot_of_row ? slot_of_row[r] : (slot_const >= 0 ? slot_const : r);
}

// ---------------------------------------------------------------------------
// Embedding gather
// ---------------------------------------------------------------------------
__global__ void k_embed(const uint16_t *__restrict__ E, const int32_t *__restrict__ tokens,
                        const uint8_t *__restrict__ valid, int H, float *__restrict__ x)
{
    const int b = blockIdx.y;
    const int tok = (valid == nullptr || valid[b]) ? tokens[b] : 0;
    const uint16_t *src = E + (size_t)tok * H;
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < H; i += gridDim.x * blockDim.x)
        x[(size_t)b * H + i] = bf2f(src[i]);
}

hipError_t launch_embed(const uint16_t *E, const int32_t *tokens, const uint8_t *valid, int rows, int H,
                        float *x, hipStream_t st)
{
    dim3 grid((H + 255) / 256, rows);
    hipLaunchKernelGGL(k_embed, grid, dim3(256), 0, st, E, tokens, valid, H, x);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// RMSNorm with the residual add of the previous projection's split partials
// folded in.  One wavefront per row; lane l owns the float4 groups
// 4l + 256j.  The sum of squares runs sequentially per lane, then through the
// fixed butterfly.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_rmsnorm(float *__restrict__ x, const float *__restrict__ part,
                                                 int S, long long part_stride, int rows, int H,
                                                 const uint16_t *__restrict__ g, float eps,
                                                 uint16_t *__restrict__ h)
{
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    float *xr = x + (size_t)row * H;
    float ss = 0.f;
    for (int i = 4 * lane; i < H; i += 256) {
        float4 v = *(const float4 *)(xr + i);
        for (int s = 0; s < S; ++s) {
            float4 p = *(const float4 *)(part + s * part_stride + (size_t)row * H + i);
            v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
        }
        if (S > 0) *(float4 *)(xr + i) = v;
        ss += v.x * v.x;
        ss += v.y * v.y;
        ss += v.z * v.z;
        ss += v.w * v.w;
    }
    ss = wave_sum(ss);
    const float rstd = 1.0f / sqrtf(ss / (float)H + eps);
    uint16_t *hr = h + (size_t)row * H;
    for (int i = 4 * lane; i < H; i += 256) {
        float4 v = *(const float4 *)(xr + i);
        ushort4 o;
        o.x = f2bf(v.x * rstd * bf2f(g[i + 0]));
        o.y = f2bf(v.y * rstd * bf2f(g[i + 1]));
        o.z = f2bf(v.z * rstd * bf2f(g[i + 2]));
        o.w = f2bf(v.w * rstd * bf2f(g[i + 3]));
        *(ushort4 *)(hr + i) = o;
    }
}

hipError_t launch_rmsnorm(float *x, const float *part, int S, long long part_stride, int rows, int H,
                          const uint16_t *g, float eps, uint16_t *h, hipStream_t st)
{
    hipLaunchKernelGGL(k_rmsnorm, dim3((rows + 3) / 4), dim3(256), 0, st, x, part, S, part_stride, rows, H,
                       g, eps, h);
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
__global__ __launch_bounds__(256) void k_gemm(const uint16_t *__restrict__ A, int lda,
                                              const uint16_t *__restrict__ W, int M, int N, int K, int Kc,
                                              float *__restrict__ out, long long split_stride, int ldo)
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
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) ap[mt] = A + (size_t)(m0 + 16 * mt + r) * lda + kg * 8;

    f32x4 acc[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = (f32x4){0.f, 0.f, 0.f, 0.f};

    int k = kbeg;
    for (; k + 32 * KU <= kend; k += 32 * KU) {
        bf16x8 wf[NT][KU], af[MT][KU];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int u = 0; u < KU; ++u)
                wf[nt][u] = __builtin_bit_cast(bf16x8, *(const uint4 *)(wp[nt] + k + 32 * u));
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int u = 0; u < KU; ++u)
                af[mt][u] = __builtin_bit_cast(bf16x8, *(const uint4 *)(ap[mt] + k + 32 * u));
#pragma unroll
        for (int u = 0; u < KU; ++u)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
                    acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[mt][u], wf[nt][u], acc[mt][nt],
                                                                          0, 0, 0);
    }
    for (; k < kend; k += 32) {   // K tail, one 32-step at a time; K % 8 == 0
        const bool in = (k + kg * 8) < kend;
        const uint4 z = {0u, 0u, 0u, 0u};
        bf16x8 wf[NT], af[MT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
            wf[nt] = __builtin_bit_cast(bf16x8, in ? *(const uint4 *)(wp[nt] + k) : z);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            af[mt] = __builtin_bit_cast(bf16x8, in ? *(const uint4 *)(ap[mt] + k) : z);
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
}

hipError_t launch_gemm(const uint16_t *A, int lda, const uint16_t *W, const GemmShape &g, float *out,
                       long long split_stride, int ldo, hipStream_t st)
{
    constexpr int NT = 4;
    const int ncb = (g.N + 16 * NT - 1) / (16 * NT);
    const int rows_per_tile = 16 * g.mt;
    dim3 grid((ncb + 3) / 4, g.S, (g.M + rows_per_tile - 1) / rows_per_tile);
    switch (g.mt) {
    case 1:
        hipLaunchKernelGGL((k_gemm<1, NT, 4>), grid, dim3(256), 0, st, A, lda, W, g.M, g.N, g.K, g.Kc, out,
                           split_stride, ldo);
        break;
    case 2:
        hipLaunchKernelGGL((k_gemm<2, NT, 4>), grid, dim3(256), 0, st, A, lda, W, g.M, g.N, g.K, g.Kc, out,
                           split_stride, ldo);
        break;
    case 4:
        hipLaunchKernelGGL((k_gemm<4, NT, 2>), grid, dim3(256), 0, st, A, lda, W, g.M, g.N, g.K, g.Kc, out,
                           split_stride, ldo);
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
__global__ void k_qkv_post(const float *__restrict__ part, int S, long long part_stride,
                           const uint8_t *__restrict__ valid, const int32_t *__restrict__ pos,
                           const int32_t *__restrict__ slot_of_row, int slot_const, int nq, int nkv, int d,
                           const float2 *__restrict__ rope_tab, uint16_t *__restrict__ q,
                           uint16_t *__restrict__ kc, uint16_t *__restrict__ vc, KvView kv)
{
    const int hd = blockIdx.x, r = blockIdx.y, i = threadIdx.x;
    const int half = d >> 1;
    if (i >= half) return;
    if (valid != nullptr && !valid[r]) return;
    const int p = pos[r];
    const int ncols = (nq + 2 * nkv) * d;
    const int c0 = hd * d + i, c1 = c0 + half;
    float x0 = 0.f, x1 = 0.f;
    for (int s = 0; s < S; ++s) {
        const float *ps = part + s * part_stride + (size_t)r * ncols;
        x0 += ps[c0];
        x1 += ps[c1];
    }
    x0 = bf2f(f2bf(x0));
    x1 = bf2f(f2bf(x1));
    if (hd < nq + nkv) {
        const float2 cs = rope_tab[(size_t)p * half + i];
        const float y0 = x0 * cs.x - x1 * cs.y;
        const float y1 = x1 * cs.x + x0 * cs.y;
        x0 = y0;
        x1 = y1;
    }
    const uint16_t b0 = f2bf(x0), b1 = f2bf(x1);
    if (hd < nq) {
        q[(size_t)r * nq * d + c0] = b0;
        q[(size_t)r * nq * d + c1] = b1;
    } else {
        const int slot = row_slot(slot_of_row, slot_const, r);
        const bool is_k = hd < nq + nkv;
        const int kvh = is_k ? hd - nq : hd - nq - nkv;
        uint16_t *dst = (is_k ? kc : vc) + kv_offset(kv, nkv, d, slot, kvh, p);
        dst[i] = b0;
        dst[i + half] = b1;
    }
}

hipError_t launch_qkv_post(const float *part, int S, long long part_stride, int rows, const uint8_t *valid,
                           const int32_t *pos, const int32_t *slot_of_row, int slot_const, int nq, int nkv,
                           int d, const float2 *rope_tab, uint16_t *q, uint16_t *kc, uint16_t *vc, KvView kv,
                           hipStream_t st)
{
    hipLaunchKernelGGL(k_qkv_post, dim3(nq + 2 * nkv, rows), dim3(64), 0, st, part, S, part_stride, valid, pos,
                       slot_of_row, slot_const, nq, nkv, d, rope_tab, q, kc, vc, kv);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Split-KV decode attention.  The split count of a row is
// ceil((pos + 1) / chunk): a function of the row's own length only, so the
// split is request-local and the merge order (split index) is fixed.
// Block (split, kvh, row), one wavefront.  Scores: lane j takes tokens
// t0 + j + 64 i, each a sequential dot over d.  Softmax statistics: exact
// max, then a per-lane sequential sum and the fixed butterfly.  P V: lane j
// owns d/64 output columns and walks the chunk's tokens in order.
// ---------------------------------------------------------------------------
template <int D, int G>
__global__ __launch_bounds__(64) void k_attn_split(const uint16_t *__restrict__ q, const uint8_t *__restrict__ valid,
                                                   const int32_t *__restrict__ pos,
                                                   const int32_t *__restrict__ slot_of_row, int slot_const,
                                                   int nq, int nkv, const uint16_t *__restrict__ kc,
                                                   const uint16_t *__restrict__ vc, KvView kv, int chunk,
                                                   int max_splits, float *__restrict__ ws)
{
    constexpr int EPL = D / 64;
    const int split = blockIdx.x, kvh = blockIdx.y, r = blockIdx.z;
    const int lane = threadIdx.x;
    if (valid != nullptr && !valid[r]) return;
    const int n = pos[r] + 1;
    const int t0 = split * chunk;
    if (t0 >= n) return;
    const int t1 = min(n, t0 + chunk);
    const int slot = row_slot(slot_of_row, slot_const, r);

    extern __shared__ float smem[];
    float *qs = smem;            // [G][D]
    float *sc = smem + G * D;    // [G][chunk]
    const uint16_t *qr = q + (size_t)r * nq * D + (size_t)kvh * G * D;
    for (int i = lane; i < G * D; i += 64) qs[i] = bf2f(qr[i]);
    __syncthreads();

    const float scale = 1.0f / sqrtf((float)D);
    for (int t = t0 + lane; t < t1; t += 64) {
        const uint16_t *kr = kc + kv_offset(kv, nkv, D, slot, kvh, t);
        float a[G];
#pragma unroll
        for (int g = 0; g < G; ++g) a[g] = 0.f;
#pragma unroll
        for (int e = 0; e < D; e += 8) {
            uint4 raw = *(const uint4 *)(kr + e);
            const uint16_t *kv8 = (const uint16_t *)&raw;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float kf = bf2f(kv8[j]);
#pragma unroll
                for (int g = 0; g < G; ++g) a[g] += qs[g * D + e + j] * kf;
            }
        }
#pragma unroll
        for (int g = 0; g < G; ++g) sc[g * chunk + (t - t0)] = a[g] * scale;
    }
    __syncthreads();

    float mg[G], lg[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        float m = -INFINITY;
        for (int t = t0 + lane; t < t1; t += 64) m = fmaxf(m, sc[g * chunk + (t - t0)]);
        m = wave_max(m);
        float l = 0.f;
        for (int t = t0 + lane; t < t1; t += 64) {
            const float w = __expf(sc[g * chunk + (t - t0)] - m);
            sc[g * chunk + (t - t0)] = w;
            l += w;
        }
        mg[g] = m;
        lg[g] = wave_sum(l);
    }
    __syncthreads();

    float acc[G][EPL];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int j = 0; j < EPL; ++j) acc[g][j] = 0.f;
    for (int t = t0; t < t1; ++t) {
        const uint16_t *vr = vc + kv_offset(kv, nkv, D, slot, kvh, t) + lane * EPL;
        float vf[EPL];
        if constexpr (EPL == 2) {
            const uint32_t w2 = *(const uint32_t *)vr;
            vf[0] = __uint_as_float(w2 << 16);
            vf[1] = __uint_as_float(w2 & 0xffff0000u);
        } else {
            vf[0] = bf2f(vr[0]);
        }
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const float w = sc[g * chunk + (t - t0)];
#pragma unroll
            for (int j = 0; j < EPL; ++j) acc[g][j] += w * vf[j];
        }
    }
    float *o = ws + (((size_t)r * nkv + kvh) * max_splits + split) * (G * (D + 2));
    if (lane == 0) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
            o[g] = mg[g];
            o[G + g] = lg[g];
        }
    }
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int j = 0; j < EPL; ++j) o[2 * G + g * D + lane * EPL + j] = acc[g][j];
}

template <int D, int G>
__global__ __launch_bounds__(64) void k_attn_merge(const float *__restrict__ ws, const uint8_t *__restrict__ valid,
                                                   const int32_t *__restrict__ pos, int nq, int nkv, int chunk,
                                                   int max_splits, uint16_t *__restrict__ o)
{
    constexpr int EPL = D / 64;
    const int kvh = blockIdx.x, r = blockIdx.y, lane = threadIdx.x;
    uint16_t *orow = o + (size_t)r * nq * D + (size_t)kvh * G * D;
    if (valid != nullptr && !valid[r]) {
        for (int i = lane; i < G * D; i += 64) orow[i] = 0;
        return;
    }
    const int n = pos[r] + 1;
    const int ns = (n + chunk - 1) / chunk;
    const float *base = ws + ((size_t)r * nkv + kvh) * max_splits * (G * (D + 2));
    const int stride = G * (D + 2);
#pragma unroll
    for (int g = 0; g < G; ++g) {
        float M = -INFINITY;
        for (int s = 0; s < ns; ++s) M = fmaxf(M, base[s * stride + g]);
        float L = 0.f;
        float acc[EPL];
#pragma unroll
        for (int j = 0; j < EPL; ++j) acc[j] = 0.f;
        for (int s = 0; s < ns; ++s) {
            const float f = __expf(base[s * stride + g] - M);
            L += base[s * stride + G + g] * f;
#pragma unroll
            for (int j = 0; j < EPL; ++j) acc[j] += base[s * stride + 2 * G + g * D + lane * EPL + j] * f;
        }
#pragma unroll
        for (int j = 0; j < EPL; ++j) orow[g * D + lane * EPL + j] = f2bf(acc[j] / L);
    }
}

template <int D, int G>
static void launch_attn_dg(const uint16_t *q, int rows, const uint8_t *valid, const int32_t *pos,
                           const int32_t *slot_of_row, int slot_const, int nq, int nkv, const uint16_t *kc,
                           const uint16_t *vc, KvView kv, int chunk, int max_splits, float *ws, hipStream_t st)
{
    const size_t shm = sizeof(float) * (G * D + G * chunk);
    hipLaunchKernelGGL((k_attn_split<D, G>), dim3(max_splits, nkv, rows), dim3(64), shm, st, q, valid, pos,
                       slot_of_row, slot_const, nq, nkv, kc, vc, kv, chunk, max_splits, ws);
}

template <int D, int G>
static void launch_merge_dg(const float *ws, int rows, const uint8_t *valid, const int32_t *pos, int nq,
                            int nkv, int chunk, int max_splits, uint16_t *o, hipStream_t st)
{
    hipLaunchKernelGGL((k_attn_merge<D, G>), dim3(nkv, rows), dim3(64), 0, st, ws, valid, pos, nq, nkv, chunk,
                       max_splits, o);
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
                             const uint16_t *kc, const uint16_t *vc, KvView kv, int chunk, int max_splits,
                             float *ws, hipStream_t st)
{
    CORUN_ATTN_DISPATCH(launch_attn_dg, q, rows, valid, pos, slot_of_row, slot_const, nq, nkv, kc, vc, kv, chunk,
                        max_splits, ws, st);
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
    const int r = blockIdx.y;
    const int j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= F) return;
    const float *p = part + (size_t)r * 2 * F;
    float gs = 0.f, us = 0.f;
    for (int s = 0; s < S; ++s) {
        gs += p[s * part_stride + j];
        us += p[s * part_stride + F + j];
    }
    const float g = bf2f(f2bf(gs));
    const float u = bf2f(f2bf(us));
    const float silu = g / (1.0f + __expf(-g));
    a[(size_t)r * lda + j] = f2bf(silu * u);
}

hipError_t launch_swiglu(const float *part, int S, long long part_stride, int rows, int F, uint16_t *a, int lda,
                         hipStream_t st)
{
    hipLaunchKernelGGL(k_swiglu, dim3((F + 255) / 256, rows), dim3(256), 0, st, part, S, part_stride, F, a, lda);
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
    hipLaunchKernelGGL(k_reduce_splits, dim3((unsigned)blocks), dim3(256), 0, st, part, S, stride, n, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Greedy argmax: first index of the maximum.  (value, index) under
// "larger value, then smaller index" is a total order, so any combining tree
// gives the same, exact answer.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void better(float &v, int &i, float v2, int i2)
{
    if (v2 > v || (v2 == v && i2 < i)) {
        v = v2;
        i = i2;
    }
}

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

hipError_t launch_argmax(const float *logits, int rows, int V, const uint8_t *valid, int32_t *next, hipStream_t st)
{
    hipLaunchKernelGGL(k_argmax, dim3(rows), dim3(256), 0, st, logits, V, valid, next);
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
    hipLaunchKernelGGL(k_feedback, dim3(1), dim3(256), 0, st, tokens, seq_lens, valid, next, B, history, counter,
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
    hipLaunchKernelGGL(k_rope_table, dim3(max_pos), dim3(64), 0, st, tab, d, theta);
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
    hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)blocks), dim3(256), 0, st, p, n_words, v);
    return hipGetLastError();
}

__global__ void k_iota(int32_t *p, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = i;
}

hipError_t launch_iota(int32_t *p, int n, hipStream_t st)
{
    hipLaunchKernelGGL(k_iota, dim3((n + 255) / 256), dim3(256), 0, st, p, n);
    return hipGetLastError();
}

}  // namespace corun
