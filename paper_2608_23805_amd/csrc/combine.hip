// combine.hip -- publication of the layer output and slot generation words.
//
// The combine is the only kernel that writes the caller's output, and it does
// so only when the status word is clean: an invalid completion never makes
// data visible (the lifetime row of the paper's table of certificate
// obligations; its fatal fault cells publish nothing, "Integrated
// Deterministic Faults").  out[t] = shared(x_t) + sum over the token's
// experts in ascending id of the weighted contributions, summed in fp32 in
// that fixed order so the result does not depend on slot capacity.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace msi {

// Status handling shared by both combines.  With an arrival counter (small
// grids: one counter update per workgroup), thread 0 of each workgroup alone
// reads the status word and shares it through LDS, then counts the workgroup
// in; the ticket is checked at the end of the kernel, and the last workgroup
// to arrive (the counter wraps back to zero) clears the word, after every
// workgroup has read it, so the next forward starts from a clean word without
// a launch of its own.  Without a counter every thread reads the word.
// The launch's first workgroup, which has no rows of its own (one more than
// the rows need), publishes to pinned host words: the demanded experts
// (count, then ids) when `demand` is given, then status | STATUS_DONE with a
// system-scope release, so a host that sees the done bit also sees the list.
// The release waits for the host stores; in a workgroup of its own that wait
// runs beside the row work instead of before it.  Being dispatched first, it
// publishes when the combine starts (the status is final then: the expert
// kernels have completed), so the host returns and queues its next work
// while the row workgroups still write `out`.
__device__ __forceinline__ uint32_t combine_status(const CombinePublish &P, uint32_t &ticket)
{
    uint32_t st;
    ticket = 0u;
    if (P.arrive) {
        __shared__ uint32_t st_s;
        if (threadIdx.x == 0)
            st_s = __hip_atomic_load(P.status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __syncthreads();
        st = st_s;
        if (threadIdx.x == 0)
            ticket = atomicInc(P.arrive, gridDim.x - 1u);   // issued after this workgroup's read
    } else {
        st = __hip_atomic_load(P.status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (blockIdx.x == 0 && P.host) {
        if (P.demand) {
            const int n = P.demand[0];
            for (int i = threadIdx.x; i <= n; i += blockDim.x)
                __hip_atomic_store(P.host + 1 + i, uint32_t(P.demand[i]), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_SYSTEM);
            __syncthreads();
        }
        if (threadIdx.x == 0) {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");   // system scope: the list before the done bit
            __hip_atomic_store(P.host, st | STATUS_DONE, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        }
    }
    return st;
}

__device__ __forceinline__ void combine_finish(const CombinePublish &P, uint32_t ticket)
{
    if (P.arrive && threadIdx.x == 0 && ticket == gridDim.x - 1u)
        __hip_atomic_store(P.status, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// fp32 layers: y and ys in fp32, four columns per thread.
__global__ void __launch_bounds__(256) combine_f32_kernel(const float *__restrict__ y, const float *__restrict__ ys,
                                                          const int32_t *__restrict__ inv, float *__restrict__ out,
                                                          CombinePublish P, int T, int K, int d)
{
    uint32_t ticket;
    const uint32_t st = combine_status(P, ticket);
    combine_finish(P, ticket);
    if (st != 0u)
        return;
    const int d4 = d / 4;
    const int64_t i = (int64_t(blockIdx.x) - 1) * blockDim.x + threadIdx.x;   // workgroup 0: no rows
    if (i < 0 || i >= int64_t(T) * d4)
        return;
    const int t = int(i / d4), c = int(i % d4) * 4;
    float4 acc = ys ? *reinterpret_cast<const float4 *>(ys + int64_t(t) * d + c) : make_float4(0.f, 0.f, 0.f, 0.f);
    // all K row loads are issued before the fixed-order sum (K <= 16)
    f32x4 v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k)
        if (k < K)
            v[k] = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(y + int64_t(inv[int64_t(t) * K + k]) * d + c));
#pragma unroll
    for (int k = 0; k < 16; ++k)
        if (k < K) {
            acc.x += v[k][0];
            acc.y += v[k][1];
            acc.z += v[k][2];
            acc.w += v[k][3];
        }
    __builtin_nontemporal_store(f32x4{acc.x, acc.y, acc.z, acc.w}, reinterpret_cast<f32x4 *>(out + int64_t(t) * d + c));
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// bf16 y and ys, eight columns per thread; the sum is in fp32 in the same
// fixed order (shared expert, then the K routed rows in selection order).
// y is read once and out written once: both go through non-temporal
// accesses (at T = 32768 that takes the combine from 342 to 295 us).
// The row indices and the shared row are read together with the status word,
// so the kernel costs two dependent memory round trips before its store.
__global__ void __launch_bounds__(256) combine_kernel(const uint16_t *__restrict__ y, const uint16_t *__restrict__ ys,
                                                      const int32_t *__restrict__ inv, float *__restrict__ out,
                                                      CombinePublish P, int T, int K, int d)
{
    const int d8 = d / 8;
    const int64_t n = int64_t(T) * d8;
    const int64_t i = (int64_t(blockIdx.x) - 1) * blockDim.x + threadIdx.x;   // workgroup 0: no rows
    const bool live = i >= 0 && i < n;
    const int64_t ic = live ? i : 0;
    const int t = int(ic / d8), c = int(ic % d8) * 8;
    int32_t row[16];
    u32x4 s = {0u, 0u, 0u, 0u};
    if (n > 0) {                                       // T == 0: nothing to read
#pragma unroll
        for (int k = 0; k < 16; ++k)
            if (k < K)
                row[k] = inv[int64_t(t) * K + k];
        if (ys)
            s = *reinterpret_cast<const u32x4 *>(ys + int64_t(t) * d + c);
    }
    uint32_t ticket;
    const uint32_t st = combine_status(P, ticket);
    if (st == 0u && live) {
        float a[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            a[2 * q] = bf16_lo(s[q]);
            a[2 * q + 1] = bf16_hi(s[q]);
        }
        u32x4 v[16];
#pragma unroll
        for (int k = 0; k < 16; ++k)
            if (k < K)
                v[k] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(y + int64_t(row[k]) * d + c));
#pragma unroll
        for (int k = 0; k < 16; ++k)
            if (k < K) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    a[2 * q] += bf16_lo(v[k][q]);
                    a[2 * q + 1] += bf16_hi(v[k][q]);
                }
            }
        f32x4 *o = reinterpret_cast<f32x4 *>(out + int64_t(t) * d + c);
        __builtin_nontemporal_store(f32x4{a[0], a[1], a[2], a[3]}, o);
        __builtin_nontemporal_store(f32x4{a[4], a[5], a[6], a[7]}, o + 1);
    }
    combine_finish(P, ticket);
}

hipError_t launch_combine(const void *y, const void *ys, bool f32, const int32_t *inv, float *out,
                          const CombinePublish &P, int T, int K, int d, hipStream_t s)
{
    if (!P.status)
        return hipErrorInvalidValue;
    // the publishing workgroup, then the row ones (also for T == 0: the status is still published
    // and cleared)
    if (f32) {
        const int64_t n = int64_t(T) * (d / 4);
        launch_k(combine_f32_kernel, unsigned((n + 255) / 256 + 1), 256, 0, s, static_cast<const float *>(y),
                 static_cast<const float *>(ys), inv, out, P, T, K, d);
    } else {
        const int64_t n = int64_t(T) * (d / 8);
        launch_k(combine_kernel, unsigned((n + 255) / 256 + 1), 256, 0, s, static_cast<const uint16_t *>(y),
                 static_cast<const uint16_t *>(ys), inv, out, P, T, K, d);
    }
    return hipGetLastError();
}

// Residual stream of a layer stack: h = float(x0) or h += out, then
// x = bf16(h / sqrt(mean(h^2) + eps)) per row.  One 256-thread workgroup per
// row; the sum of squares is reduced in a fixed order (per-thread strided
// partial sums, then a wavefront tree, then the four wavefronts in order).
__global__ void __launch_bounds__(256) residual_kernel(const uint16_t *__restrict__ x0,
                                                       const float *__restrict__ out, float *__restrict__ h,
                                                       uint16_t *__restrict__ x, int cols)
{
    __shared__ float part[4];
    const int64_t row = blockIdx.x;
    float *hr = h + row * cols;
    float ss = 0.f;
    for (int c = threadIdx.x; c < cols; c += blockDim.x) {
        const float v = x0 ? bf16_to_f32(x0[row * cols + c]) : hr[c] + out[row * cols + c];
        hr[c] = v;
        ss = fmaf(v, v, ss);
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0)
        part[threadIdx.x >> 6] = ss;
    __syncthreads();
    const float ms = (((part[0] + part[1]) + part[2]) + part[3]) / float(cols);
    const float inv = 1.0f / sqrtf(ms + 1e-6f);
    for (int c = threadIdx.x; c < cols; c += blockDim.x)
        x[row * cols + c] = f32_to_bf16(hr[c] * inv);
}

hipError_t launch_residual(const uint16_t *x0, const float *out, float *h, uint16_t *x, int rows, int cols,
                           hipStream_t s)
{
    if (rows == 0 || cols == 0)
        return hipSuccess;
    launch_k(residual_kernel, unsigned(rows), 256, 0, s, x0, out, h, x, cols);
    return hipGetLastError();
}

// Generation words are written with vector stores from one lane per entry.
__global__ void set_gens_kernel(uint32_t *gen_dev, GenBatch b)
{
    const uint32_t i = threadIdx.x;
    if (i < b.n)
        __hip_atomic_store(gen_dev + b.slot[i], b.value[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

hipError_t launch_set_gens(uint32_t *gen_dev, const GenBatch &b, hipStream_t s)
{
    if (b.n == 0)
        return hipSuccess;
    launch_k(set_gens_kernel, 1, GEN_BATCH, 0, s, gen_dev, b);
    return hipGetLastError();
}

__global__ void clear_word_kernel(uint32_t *w)
{
    if (threadIdx.x == 0)
        __hip_atomic_store(w, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

hipError_t launch_clear_word(uint32_t *word, hipStream_t s)
{
    launch_k(clear_word_kernel, 1, 64, 0, s, word);
    return hipGetLastError();
}

}  // namespace msi
