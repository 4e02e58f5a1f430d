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
//
// Top-K is a radix select on order-preserving integer keys: 32 passes of
// wavefront ballots find the K-th largest key, every larger key is selected,
// and keys equal to it are taken in ascending expert id until K are chosen.
// The selected experts come out in ascending id order from ballot prefix
// counts, so no sort and no per-round cross-lane argmax is needed.
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

// ---------------------------------------------------------------- logits, bf16, T <= 16
// Weight streaming: workgroup b owns experts 16b..16b+15; its four
// wavefronts take quarters of d with the router rows as the 16x16x32 MFMA A
// operand read straight from memory and the (<= 16) tokens as the B operand
// from LDS; the four partial sums are added in wavefront order through LDS.
__global__ void __launch_bounds__(256) router_stream_kernel(const uint16_t *__restrict__ x,
                                                            const uint16_t *__restrict__ wr,
                                                            const float *__restrict__ bias, float *__restrict__ L,
                                                            int T, int d, int E)
{
    extern __shared__ __attribute__((aligned(16))) uint16_t xs[];   // [16][d + 8]
    __shared__ float red[3][64][4];
    const int ldk = d + 8;
    const int chunks = d / 8, total = T * chunks;
    for (int c0 = threadIdx.x; c0 < total; c0 += 8 * blockDim.x) {   // loads batched 8 deep
        uint4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int c = c0 + u * int(blockDim.x);
            if (c < total)
                v[u] = *reinterpret_cast<const uint4 *>(x + int64_t(c / chunks) * d + (c % chunks) * 8);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int c = c0 + u * int(blockDim.x);
            if (c < total)
                *reinterpret_cast<uint4 *>(xs + (c / chunks) * ldk + (c % chunks) * 8) = v[u];
        }
    }
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int e0 = blockIdx.x * 16;
    const int row = e0 + (lane & 15);
    const int j = lane & 15, kg = (lane >> 4) * 8;
    const int kq = d / 4;
    const bool rvalid = row < E, live = j < T;
    const uint16_t *wp = wr + int64_t(rvalid ? row : 0) * d + wave * kq + kg;
    const uint16_t *xr = xs + j * ldk + wave * kq + kg;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < kq; k0 += 32 * 8) {
        u32x4 w[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            w[u] = (rvalid && k0 + 32 * u < kq) ? load_stream16(wp + k0 + 32 * u) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            if (k0 + 32 * u >= kq)
                break;
            const uint4 xv = live ? *reinterpret_cast<const uint4 *>(xr + k0 + 32 * u) : make_uint4(0, 0, 0, 0);
            acc = mfma16(as_bf16x8(w[u]), as_bf16x8(xv), acc);
        }
    }
    if (wave > 0)
        for (int r = 0; r < 4; ++r)
            red[wave - 1][lane][r] = acc[r];
    __syncthreads();
    if (wave == 0 && live) {
        for (int r = 0; r < 4; ++r) {
            const float v = ((acc[r] + red[0][lane][r]) + red[1][lane][r]) + red[2][lane][r];
            const int e = e0 + 4 * (lane >> 4) + r;
            if (e < E)
                L[int64_t(j) * E + e] = v + (bias ? bias[e] : 0.f);
        }
    }
}

// ---------------------------------------------------------------- top-K

// Order-preserving key: a > b as floats <=> key(a) > key(b); -0.0 folds onto +0.0.
__device__ __forceinline__ uint32_t order_key(float v)
{
    uint32_t u = __float_as_uint(v);
    if (u == 0x80000000u)
        u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Selection of one token by one wavefront.  Lane l holds logits of experts
// l + 64 j.  On return, sel_rank[j] is the output position (ascending id) of
// expert l + 64 j, or -1, and w[j] its gate weight.
template <int PER>
__device__ __forceinline__ void wave_select(const float *__restrict__ Lrow, int E, int K, int lane, int *sel_rank,
                                            float *w)
{
    float v[PER];
    uint32_t key[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int e = lane + 64 * j;
        v[j] = e < E ? Lrow[e] : -INFINITY;
        key[j] = e < E ? order_key(v[j]) : 0u;    // 0 is below every real key
    }
    // radix select the K-th largest key
    uint32_t prefix = 0u, mask = 0u;
    int need = K;
    for (int bit = 31; bit >= 0; --bit) {
        const uint32_t b = 1u << bit, mk = mask | b, want = prefix | b;
        int cnt = 0;
#pragma unroll
        for (int j = 0; j < PER; ++j)
            cnt += __popcll(__ballot((key[j] & mk) == want));
        if (cnt >= need)
            prefix = want;
        else
            need -= cnt;
        mask = mk;
    }
    // keys above the threshold, then equal keys in ascending id, in id order
    const uint64_t lt = lanemask_lt(lane);
    int base = 0, eq_taken = 0;
    float m = -INFINITY;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const bool gt = key[j] > prefix;
        const bool eq = key[j] == prefix;
        const uint64_t eqm = __ballot(eq);
        const bool sel = gt || (eq && eq_taken + __popcll(eqm & lt) < need);
        eq_taken += __popcll(eqm);
        const uint64_t selm = __ballot(sel);
        sel_rank[j] = sel ? base + __popcll(selm & lt) : -1;
        base += __popcll(selm);
        if (sel)
            m = fmaxf(m, v[j]);
    }
    m = wave_max(m);
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        w[j] = sel_rank[j] >= 0 ? expf(v[j] - m) : 0.f;
        s += w[j];
    }
    s = wave_sum(s);
    const float inv = 1.0f / s;
#pragma unroll
    for (int j = 0; j < PER; ++j)
        w[j] *= inv;
}

template <int PER>
__global__ void __launch_bounds__(256) topk_kernel(const float *__restrict__ L, int32_t *__restrict__ idx,
                                                   float *__restrict__ wout, int T, int E, int K)
{
    const int lane = threadIdx.x & 63;
    const int t = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    if (t >= T)
        return;
    int rank[PER];
    float w[PER];
    wave_select<PER>(L + int64_t(t) * E, E, K, lane, rank, w);
#pragma unroll
    for (int j = 0; j < PER; ++j)
        if (rank[j] >= 0) {
            idx[int64_t(t) * K + rank[j]] = lane + 64 * j;
            wout[int64_t(t) * K + rank[j]] = w[j];
        }
}

// ---------------------------------------------------------------- permutation
// Tokens are cut into blocks of PERM_BLOCK.  For block b, bit tl of row e of
// an LDS bitmask says token b*PERM_BLOCK + tl selected expert e.  The rank of
// (t, e) among the tokens of its expert is
//   offsets[e] + (tokens of e in earlier blocks) + popcount(row e below tl).

__device__ __forceinline__ void clear_bits(uint32_t *bits, int E)
{
    for (int i = threadIdx.x; i < E * (PERM_BLOCK / 32); i += blockDim.x)
        bits[i] = 0;
}

__device__ __forceinline__ void build_bits(uint32_t *bits, const int32_t *idx, int T, int K, int E, int t0)
{
    clear_bits(bits, E);
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

// Single workgroup of 1024 threads: per-expert exclusive scan over blocks
// (loads issued 16 at a time), then an exclusive scan over experts.
__global__ void __launch_bounds__(1024) perm_scan_kernel(int32_t *__restrict__ blockhist, int nblk, int E,
                                                         int32_t *__restrict__ counts,
                                                         int32_t *__restrict__ offsets)
{
    __shared__ int32_t part[1024];
    const int e = threadIdx.x;
    int run = 0;
    if (e < E) {
        for (int b0 = 0; b0 < nblk; b0 += 16) {
            int v[16];
#pragma unroll
            for (int i = 0; i < 16; ++i)
                v[i] = b0 + i < nblk ? blockhist[int64_t(b0 + i) * E + e] : 0;
#pragma unroll
            for (int i = 0; i < 16; ++i)
                if (b0 + i < nblk) {
                    blockhist[int64_t(b0 + i) * E + e] = run;
                    run += v[i];
                }
        }
        counts[e] = run;
    }
    part[e] = e < E ? run : 0;
    __syncthreads();
    block_scan_1024(part);
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

// T <= PERM_BLOCK: top-K of every token (one wavefront per token), then the
// histogram, scans and scatter, in one 1024-thread workgroup.  With
// L == nullptr the selection is read from idx / w instead.
template <int PER>
__global__ void __launch_bounds__(1024) route_small_kernel(const float *__restrict__ L, int32_t *__restrict__ idx,
                                                           float *__restrict__ w, int32_t *__restrict__ counts,
                                                           int32_t *__restrict__ offsets, int32_t *__restrict__ perm,
                                                           int32_t *__restrict__ inv, float *__restrict__ row_weight,
                                                           int T, int K, int E)
{
    extern __shared__ uint32_t bits[];          // [E][PERM_BLOCK / 32]
    __shared__ int32_t part[1024];
    __shared__ int32_t sidx[PERM_BLOCK * 16];   // this workgroup's selection (T * K <= 4096)
    __shared__ float sw[PERM_BLOCK * 16];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    clear_bits(bits, E);
    __syncthreads();
    if (L) {
        for (int t = wave; t < T; t += 16) {
            int rank[PER];
            float wv[PER];
            wave_select<PER>(L + int64_t(t) * E, E, K, lane, rank, wv);
#pragma unroll
            for (int j = 0; j < PER; ++j)
                if (rank[j] >= 0) {
                    const int e = lane + 64 * j;
                    idx[t * K + rank[j]] = e;
                    w[t * K + rank[j]] = wv[j];
                    sidx[t * K + rank[j]] = e;
                    sw[t * K + rank[j]] = wv[j];
                    atomicOr(&bits[e * (PERM_BLOCK / 32) + (t >> 5)], 1u << (t & 31));
                }
        }
    } else {
        for (int a = threadIdx.x; a < T * K; a += blockDim.x) {
            const int t = a / K, e = idx[a];
            sidx[a] = e;
            sw[a] = w[a];
            atomicOr(&bits[e * (PERM_BLOCK / 32) + (t >> 5)], 1u << (t & 31));
        }
    }
    __syncthreads();
    const int e = threadIdx.x;
    const int c = e < E ? row_popc(bits + e * (PERM_BLOCK / 32)) : 0;
    part[e] = c;
    __syncthreads();
    block_scan_1024(part);
    if (e < E) {
        counts[e] = c;
        offsets[e] = part[e] - c;
    }
    if (e == E - 1)
        offsets[E] = part[e];
    __syncthreads();
    for (int a = threadIdx.x; a < T * K; a += blockDim.x) {
        const int t = a / K;
        const int ee = sidx[a];
        const int row = (part[ee] - row_popc(bits + ee * (PERM_BLOCK / 32))) +
                        rank_below(bits + ee * (PERM_BLOCK / 32), t);
        perm[row] = t;
        inv[a] = row;
        row_weight[row] = sw[a];
    }
}

// ---------------------------------------------------------------- launchers

hipError_t init_route_attributes()
{
    hipError_t e = hipSuccess;
    auto set = [&](const void *f) {
        if (e == hipSuccess)
            e = allow_large_lds(f);
    };
    set(reinterpret_cast<const void *>(&router_stream_kernel));
    set(reinterpret_cast<const void *>(&route_small_kernel<2>));
    set(reinterpret_cast<const void *>(&route_small_kernel<4>));
    set(reinterpret_cast<const void *>(&route_small_kernel<8>));
    set(reinterpret_cast<const void *>(&route_small_kernel<16>));
    return e;
}

hipError_t launch_router_logits_f32(const float *x, const float *wr, const float *bias, float *L, int T,
                                    int d, int E, hipStream_t s)
{
    const int64_t n = int64_t(T) * E;
    if (n == 0)
        return hipSuccess;
    router_logits_f32_kernel<<<dim3(unsigned((n + 255) / 256)), dim3(256), 0, s>>>(x, wr, bias, L, T, d, E);
    return hipGetLastError();
}

hipError_t launch_router_stream(const uint16_t *x, const uint16_t *wr, const float *bias, float *L, int T, int d,
                                int E, hipStream_t s)
{
    const size_t lds = size_t(16) * (d + 8) * sizeof(uint16_t);
    router_stream_kernel<<<unsigned((E + 15) / 16), 256, lds, s>>>(x, wr, bias, L, T, d, E);
    return hipGetLastError();
}

template <int PER>
static void launch_route_small_t(const float *L, int32_t *idx, float *w, int32_t *counts, int32_t *offsets,
                                 int32_t *perm, int32_t *inv, float *row_weight, int T, int K, int E, hipStream_t s)
{
    const size_t lds = size_t(E) * (PERM_BLOCK / 32) * sizeof(uint32_t);
    route_small_kernel<PER><<<1, 1024, lds, s>>>(L, idx, w, counts, offsets, perm, inv, row_weight, T, K, E);
}

hipError_t launch_route_select(const float *L, int32_t *idx, float *w, int32_t *counts, int32_t *offsets,
                               int32_t *perm, int32_t *inv, float *row_weight, int32_t *blockhist, int T, int K,
                               int E, hipStream_t s)
{
    const int per = (E + 63) / 64;
    if (T <= PERM_BLOCK) {
        // T == 0 still writes zero counts and offsets
        if (per <= 2)
            launch_route_small_t<2>(T ? L : nullptr, idx, w, counts, offsets, perm, inv, row_weight, T, K, E, s);
        else if (per <= 4)
            launch_route_small_t<4>(T ? L : nullptr, idx, w, counts, offsets, perm, inv, row_weight, T, K, E, s);
        else if (per <= 8)
            launch_route_small_t<8>(T ? L : nullptr, idx, w, counts, offsets, perm, inv, row_weight, T, K, E, s);
        else
            launch_route_small_t<16>(T ? L : nullptr, idx, w, counts, offsets, perm, inv, row_weight, T, K, E, s);
        return hipGetLastError();
    }
    const dim3 grid(unsigned((T + 3) / 4)), block(256);
    if (per <= 2)
        topk_kernel<2><<<grid, block, 0, s>>>(L, idx, w, T, E, K);
    else if (per <= 4)
        topk_kernel<4><<<grid, block, 0, s>>>(L, idx, w, T, E, K);
    else if (per <= 8)
        topk_kernel<8><<<grid, block, 0, s>>>(L, idx, w, T, E, K);
    else
        topk_kernel<16><<<grid, block, 0, s>>>(L, idx, w, T, E, K);
    const size_t lds = size_t(E) * (PERM_BLOCK / 32) * sizeof(uint32_t);
    const int nblk = (T + PERM_BLOCK - 1) / PERM_BLOCK;
    perm_hist_kernel<<<nblk, 256, lds, s>>>(idx, blockhist, T, K, E);
    perm_scan_kernel<<<1, 1024, 0, s>>>(blockhist, nblk, E, counts, offsets);
    perm_scatter_kernel<<<nblk, 256, lds, s>>>(idx, w, blockhist, offsets, perm, inv, row_weight, T, K, E);
    return hipGetLastError();
}

}  // namespace msi
