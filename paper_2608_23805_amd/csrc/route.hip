// route.hip -- router (logits, top-K, restricted softmax) and the stable
// token-by-expert permutation, for gfx950.
//
// The routed set of each token is the layer's route event (the paper compares
// every recorded route event bit for bit, Section 2.2 and Section 5.4); here
// it is produced deterministically: fp32 logits (bf16 MFMA products, fp32
// accumulation, or fp32 FMA for fp32 layers), selection by (logit desc,
// expert id asc) with one wavefront per token, softmax restricted to the
// selection, and a counting-sort permutation whose rank computation is a
// population count over per-block token bitmasks (no atomics on ordering).
#include "common.h"
#include "gemm_tile.h"
#include "kernels.h"

namespace msi {

// ---------------------------------------------------------------- logits, fp32
// One thread per (token, expert): sequential fp32 FMA over d.
__global__ void __launch_bounds__(256) router_logits_f32_kernel(const float *__restrict__ x,
                                                                const float *__restrict__ wr,
                                                                const float *__restrict__ bias,
                                                                float *__restrict__ L, int T, int d, int E)
{
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= int64_t(T) * E)
        return;
    const int t = int(i / E), e = int(i % E);
    const float *xr = x + int64_t(t) * d;
    const float *wrow = wr + int64_t(e) * d;
    float acc = 0.f;
    for (int k = 0; k < d; k += 4) {
        const float4 a = *reinterpret_cast<const float4 *>(xr + k);
        const float4 b = *reinterpret_cast<const float4 *>(wrow + k);
        acc = fmaf(a.x, b.x, acc);
        acc = fmaf(a.y, b.y, acc);
        acc = fmaf(a.z, b.z, acc);
        acc = fmaf(a.w, b.w, acc);
    }
    L[i] = acc + (bias ? bias[e] : 0.f);
}

// ---------------------------------------------------------------- top-K
// One wavefront per token.  Lane l holds logits l, l+64, ...; each of the K
// rounds takes the wave-wide best (value desc, id asc) among untaken experts.
template <int PER_LANE>
__global__ void __launch_bounds__(256) topk_kernel(const float *__restrict__ L, int32_t *__restrict__ idx,
                                                   float *__restrict__ w, int T, int E, int K)
{
    const int lane = threadIdx.x & 63;
    const int t = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    if (t >= T)
        return;
    float v[PER_LANE];
    uint32_t taken = 0;
#pragma unroll
    for (int j = 0; j < PER_LANE; ++j) {
        const int e = lane + 64 * j;
        v[j] = e < E ? L[int64_t(t) * E + e] : 0.f;
        if (e >= E)
            taken |= 1u << j;
    }
    int sel_id[16];
    float sel_v[16];
    for (int k = 0; k < K; ++k) {
        float bv = 0.f;
        int bi = 0x7fffffff;
        bool have = false;
#pragma unroll
        for (int j = 0; j < PER_LANE; ++j) {
            if (taken & (1u << j))
                continue;
            const int e = lane + 64 * j;
            if (!have || v[j] > bv || (v[j] == bv && e < bi)) {
                bv = v[j];
                bi = e;
                have = true;
            }
        }
        if (!have) {
            bv = -INFINITY;
            bi = 0x7fffffff;
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            const float ov = __shfl_xor(bv, off, 64);
            const int oi = __shfl_xor(bi, off, 64);
            if (ov > bv || (ov == bv && oi < bi)) {
                bv = ov;
                bi = oi;
            }
        }
        sel_id[k] = bi;
        sel_v[k] = bv;
        if ((bi & 63) == lane)
            taken |= 1u << (bi >> 6);
    }
    // restricted softmax in fp32; the first selected logit is the maximum
    const float m = sel_v[0];
    float s = 0.f;
    float p[16];
    for (int k = 0; k < K; ++k) {
        p[k] = expf(sel_v[k] - m);
        s += p[k];
    }
    const float inv = 1.0f / s;
    // ascending expert ids (K <= 16, insertion sort, identical in every lane)
    for (int a = 1; a < K; ++a) {
        const int ki = sel_id[a];
        const float kp = p[a];
        int b = a - 1;
        while (b >= 0 && sel_id[b] > ki) {
            sel_id[b + 1] = sel_id[b];
            p[b + 1] = p[b];
            --b;
        }
        sel_id[b + 1] = ki;
        p[b + 1] = kp;
    }
    for (int k = 0; k < K; ++k)
        if (lane == k) {
            idx[int64_t(t) * K + k] = sel_id[k];
            w[int64_t(t) * K + k] = p[k] * inv;
        }
}

// ---------------------------------------------------------------- permutation
// Tokens are cut into blocks of PERM_BLOCK.  For block b, bit tl of row e of
// an LDS bitmask says token b*PERM_BLOCK + tl selected expert e.  The rank of
// (t, e) among the tokens of its expert is
//   offsets[e] + (tokens of e in earlier blocks) + popcount(row e below tl).

__device__ __forceinline__ void build_bits(uint32_t *bits, const int32_t *__restrict__ idx, int T, int K,
                                           int E, int t0)
{
    const int words = E * (PERM_BLOCK / 32);
    for (int i = threadIdx.x; i < words; i += blockDim.x)
        bits[i] = 0;
    __syncthreads();
    const int nt = min(PERM_BLOCK, T - t0);
    for (int a = threadIdx.x; a < nt * K; a += blockDim.x) {
        const int tl = a / K;
        const int e = idx[int64_t(t0 + tl) * K + (a % K)];
        atomicOr(&bits[e * (PERM_BLOCK / 32) + (tl >> 5)], 1u << (tl & 31));
    }
    __syncthreads();
}

__device__ __forceinline__ int row_popc(const uint32_t *row)
{
    int n = 0;
#pragma unroll
    for (int w = 0; w < PERM_BLOCK / 32; ++w)
        n += __popc(row[w]);
    return n;
}

__device__ __forceinline__ int rank_below(const uint32_t *row, int tl)
{
    int n = 0;
    for (int w = 0; w < (tl >> 5); ++w)
        n += __popc(row[w]);
    const uint32_t m = (tl & 31) ? ((1u << (tl & 31)) - 1u) : 0u;
    return n + __popc(row[tl >> 5] & m);
}

__global__ void __launch_bounds__(256) perm_hist_kernel(const int32_t *__restrict__ idx,
                                                        int32_t *__restrict__ blockhist, int T, int K, int E)
{
    extern __shared__ uint32_t bits[];
    const int b = blockIdx.x;
    build_bits(bits, idx, T, K, E, b * PERM_BLOCK);
    for (int e = threadIdx.x; e < E; e += blockDim.x)
        blockhist[int64_t(b) * E + e] = row_popc(bits + e * (PERM_BLOCK / 32));
}

// Single workgroup of 1024 threads: per-expert exclusive scan over blocks,
// then an exclusive scan over experts.
__global__ void __launch_bounds__(1024) perm_scan_kernel(int32_t *__restrict__ blockhist, int nblk, int E,
                                                         int32_t *__restrict__ counts,
                                                         int32_t *__restrict__ offsets)
{
    __shared__ int32_t part[1024];
    const int e = threadIdx.x;
    int run = 0;
    if (e < E) {
        for (int b = 0; b < nblk; ++b) {
            const int v = blockhist[int64_t(b) * E + e];
            blockhist[int64_t(b) * E + e] = run;
            run += v;
        }
        counts[e] = run;
    }
    part[e] = e < E ? run : 0;
    __syncthreads();
    // Hillis-Steele inclusive scan over 1024 entries
    for (int off = 1; off < 1024; off <<= 1) {
        const int v = e >= off ? part[e - off] : 0;
        __syncthreads();
        part[e] += v;
        __syncthreads();
    }
    if (e < E)
        offsets[e] = part[e] - run;
    if (e == E - 1)
        offsets[E] = part[e];
}

__global__ void __launch_bounds__(256) perm_scatter_kernel(const int32_t *__restrict__ idx,
                                                           const float *__restrict__ w,
                                                           const int32_t *__restrict__ blockbase,
                                                           const int32_t *__restrict__ offsets,
                                                           int32_t *__restrict__ perm, int32_t *__restrict__ inv,
                                                           float *__restrict__ row_weight, int T, int K, int E)
{
    extern __shared__ uint32_t bits[];
    const int b = blockIdx.x;
    const int t0 = b * PERM_BLOCK;
    build_bits(bits, idx, T, K, E, t0);
    const int nt = min(PERM_BLOCK, T - t0);
    for (int a = threadIdx.x; a < nt * K; a += blockDim.x) {
        const int tl = a / K;
        const int64_t tk = int64_t(t0 + tl) * K + (a % K);
        const int e = idx[tk];
        const int row = offsets[e] + blockbase[int64_t(b) * E + e] + rank_below(bits + e * (PERM_BLOCK / 32), tl);
        perm[row] = t0 + tl;
        inv[tk] = row;
        row_weight[row] = w[tk];
    }
}

// T <= PERM_BLOCK: histogram, scans and scatter in one workgroup.
__global__ void __launch_bounds__(1024) perm_small_kernel(const int32_t *__restrict__ idx,
                                                          const float *__restrict__ w,
                                                          int32_t *__restrict__ counts,
                                                          int32_t *__restrict__ offsets,
                                                          int32_t *__restrict__ perm, int32_t *__restrict__ inv,
                                                          float *__restrict__ row_weight, int T, int K, int E)
{
    extern __shared__ uint32_t bits[];
    __shared__ int32_t part[1024];
    build_bits(bits, idx, T, K, E, 0);
    const int e = threadIdx.x;
    const int c = e < E ? row_popc(bits + e * (PERM_BLOCK / 32)) : 0;
    part[e] = c;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
        const int v = e >= off ? part[e - off] : 0;
        __syncthreads();
        part[e] += v;
        __syncthreads();
    }
    if (e < E) {
        counts[e] = c;
        offsets[e] = part[e] - c;
    }
    if (e == E - 1)
        offsets[E] = part[e];
    __syncthreads();
    for (int a = threadIdx.x; a < T * K; a += blockDim.x) {
        const int tl = a / K;
        const int ee = idx[a];
        const int row = (part[ee] - row_popc(bits + ee * (PERM_BLOCK / 32))) +
                        rank_below(bits + ee * (PERM_BLOCK / 32), tl);
        perm[row] = tl;
        inv[a] = row;
        row_weight[row] = w[a];
    }
}

// ---------------------------------------------------------------- launchers

hipError_t launch_router_logits_f32(const float *x, const float *wr, const float *bias, float *L, int T,
                                    int d, int E, hipStream_t s)
{
    const int64_t n = int64_t(T) * E;
    if (n == 0)
        return hipSuccess;
    router_logits_f32_kernel<<<dim3(unsigned((n + 255) / 256)), dim3(256), 0, s>>>(x, wr, bias, L, T, d, E);
    return hipGetLastError();
}

hipError_t launch_topk(const float *L, int32_t *idx, float *w, int T, int E, int K, hipStream_t s)
{
    if (T == 0)
        return hipSuccess;
    const dim3 grid(unsigned((T + 3) / 4)), block(256);
    const int per = (E + 63) / 64;
    if (per <= 2)
        topk_kernel<2><<<grid, block, 0, s>>>(L, idx, w, T, E, K);
    else if (per <= 4)
        topk_kernel<4><<<grid, block, 0, s>>>(L, idx, w, T, E, K);
    else if (per <= 8)
        topk_kernel<8><<<grid, block, 0, s>>>(L, idx, w, T, E, K);
    else
        topk_kernel<16><<<grid, block, 0, s>>>(L, idx, w, T, E, K);
    return hipGetLastError();
}

hipError_t launch_permute(const int32_t *idx, const float *w, int32_t *counts, int32_t *offsets, int32_t *perm,
                          int32_t *inv, float *row_weight, int32_t *blockhist, int T, int K, int E,
                          hipStream_t s)
{
    const size_t lds = size_t(E) * (PERM_BLOCK / 32) * sizeof(uint32_t);
    if (T <= PERM_BLOCK) {
        perm_small_kernel<<<1, 1024, lds, s>>>(idx, w, counts, offsets, perm, inv, row_weight, T, K, E);
        return hipGetLastError();
    }
    const int nblk = (T + PERM_BLOCK - 1) / PERM_BLOCK;
    perm_hist_kernel<<<nblk, 256, lds, s>>>(idx, blockhist, T, K, E);
    perm_scan_kernel<<<1, 1024, 0, s>>>(blockhist, nblk, E, counts, offsets);
    perm_scatter_kernel<<<nblk, 256, lds, s>>>(idx, w, blockhist, offsets, perm, inv, row_weight, T, K, E);
    return hipGetLastError();
}

}  // namespace msi
