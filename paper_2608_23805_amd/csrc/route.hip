// route.hip -- router (logits, top-K, restricted softmax) and the stable
// token-by-expert permutation, for gfx950.
//
// The routed set of each token is the layer's route event (the paper compares
// every recorded route event bit for bit: "Exactness Is Scoped by Identity
// and Horizon" and "Output-Exact Execution Beyond the Full-Residency
// Envelope"); here
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
#include <algorithm>

#include "common.h"
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

// Order-preserving key: a > b as floats <=> key(a) > key(b); -0.0 folds onto +0.0.
__device__ __forceinline__ uint32_t order_key(float v)
{
    uint32_t u = __float_as_uint(v);
    if (u == 0x80000000u)
        u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Radix select over PER keys per lane (absent entries hold key 0, below every
// real key).  On return the K largest keys are those with (key & mask) >
// prefix, plus the first `need` keys, in ascending id, with (key & mask) ==
// prefix.  The scan stops as soon as every key matching the prefix is needed.
template <int PER>
__device__ __forceinline__ void radix_threshold(const uint32_t (&key)[PER], int K, uint32_t &prefix,
                                                uint32_t &mask, int &need)
{
    prefix = 0u;
    mask = 0u;
    need = K;
    int cur = PER * 64;             // keys matching the prefix so far
    for (int bit = 31; bit >= 0 && cur != need; --bit) {
        const uint32_t b = 1u << bit, mk = mask | b, want = prefix | b;
        int cnt = 0;
#pragma unroll
        for (int j = 0; j < PER; ++j)
            cnt += __popcll(__ballot((key[j] & mk) == want));
        if (cnt >= need) {
            prefix = want;
            cur = cnt;
        } else {
            need -= cnt;
            cur -= cnt;
        }
        mask = mk;
    }
}

// Selection of one token by one wavefront.  Lane l holds the logits v[j] of
// experts l + 64 j (j < PER).  emit(rank, expert, weight) is called once per
// selected expert, rank = output position in ascending expert id.
//
// A threshold from the lane maxima comes first: every one of the K largest
// logits is at least the K-th largest lane maximum, so only entries whose
// masked key reaches that lane maximum's prefix are candidates.  When at most
// 64 remain they are compacted (ascending id) into the wavefront's LDS row
// and selected with one key per lane; otherwise all PER keys per lane are.
template <int PER, typename Emit>
__device__ __forceinline__ void wave_select(const float (&v)[PER], int E, int K, int lane, float *cand_v,
                                            int32_t *cand_e, Emit emit)
{
    uint32_t key[PER];
    uint32_t lm = 0u;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        key[j] = lane + 64 * j < E ? order_key(v[j]) : 0u;
        lm = max(lm, key[j]);
    }
    const uint64_t lt = lanemask_lt(lane);
    uint32_t tp, tm;
    int tn;
    {
        const uint32_t k1[1] = {lm};
        radix_threshold<1>(k1, K, tp, tm, tn);
    }
    int c = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j)
        c += __popcll(__ballot(lane + 64 * j < E && (key[j] & tm) >= tp));
    if (c <= 64) {
        int base = 0;
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const bool cd = lane + 64 * j < E && (key[j] & tm) >= tp;
            const uint64_t bm = __ballot(cd);
            if (cd) {
                const int pos = base + __popcll(bm & lt);
                cand_v[pos] = v[j];
                cand_e[pos] = lane + 64 * j;
            }
            base += __popcll(bm);
        }
        __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_wave_barrier();
        const float cv = lane < c ? cand_v[lane] : -INFINITY;
        const int ce = lane < c ? cand_e[lane] : 0;
        const uint32_t ck[1] = {lane < c ? order_key(cv) : 0u};
        __builtin_amdgcn_wave_barrier();
        uint32_t p, m;
        int need;
        radix_threshold<1>(ck, K, p, m, need);
        const bool eq = (ck[0] & m) == p;
        const bool sel = (ck[0] & m) > p || (eq && __popcll(__ballot(eq) & lt) < need);
        const uint64_t selm = __ballot(sel);
        const float mx = wave_max(sel ? cv : -INFINITY);
        float w = sel ? expf(cv - mx) : 0.f;
        const float sum = wave_sum(w);
        w *= 1.0f / sum;
        if (sel)
            emit(__popcll(selm & lt), ce, w);
        return;
    }
    uint32_t p, m;
    int need;
    radix_threshold<PER>(key, K, p, m, need);
    int base = 0, eq_taken = 0, rank[PER];
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const bool gt = (key[j] & m) > p;
        const bool eq = (key[j] & m) == p;
        const uint64_t eqm = __ballot(eq);
        const bool sel = gt || (eq && eq_taken + __popcll(eqm & lt) < need);
        eq_taken += __popcll(eqm);
        const uint64_t selm = __ballot(sel);
        rank[j] = sel ? base + __popcll(selm & lt) : -1;
        base += __popcll(selm);
        if (sel)
            mx = fmaxf(mx, v[j]);
    }
    mx = wave_max(mx);
    float w[PER], sum = 0.f;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        w[j] = rank[j] >= 0 ? expf(v[j] - mx) : 0.f;
        sum += w[j];
    }
    sum = wave_sum(sum);
    const float inv = 1.0f / sum;
#pragma unroll
    for (int j = 0; j < PER; ++j)
        if (rank[j] >= 0)
            emit(rank[j], lane + 64 * j, w[j] * inv);
}

// Logits of token t for lane's experts lane + 64 j (-inf past E).  Every load
// is issued, at a clamped index, before any is used, so the row costs one
// memory round trip.
template <int PER>
__device__ __forceinline__ void load_logits(float (&v)[PER], const float *L, int t, int E, int lane)
{
#pragma unroll
    for (int j = 0; j < PER; ++j)
        v[j] = L[int64_t(t) * E + min(lane + 64 * j, E - 1)];
#pragma unroll
    for (int j = 0; j < PER; ++j)
        if (lane + 64 * j >= E)
            v[j] = -INFINITY;
}

template <int PER>
__global__ void __launch_bounds__(256) topk_kernel(const float *__restrict__ L, int32_t *__restrict__ idx,
                                                   float *__restrict__ wout, int T, int E, int K)
{
    __shared__ float cand_v[4][64];
    __shared__ int32_t cand_e[4][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int t = blockIdx.x * (blockDim.x >> 6) + wave;
    if (t >= T)
        return;
    float v[PER];
    load_logits<PER>(v, L, t, E, lane);
    wave_select<PER>(v, E, K, lane, cand_v[wave], cand_e[wave], [&](int rank, int e, float w) {
        idx[int64_t(t) * K + rank] = e;
        wout[int64_t(t) * K + rank] = w;
    });
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
                                                         int32_t *__restrict__ offsets,
                                                         int32_t *__restrict__ demand)
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
    __syncthreads();
    part[e] = e < E && run > 0 ? 1 : 0;
    __syncthreads();
    block_scan_1024(part);
    if (e < E && run > 0)
        demand[part[e]] = e;                    // demanded experts, ascending, after the count
    if (e == E - 1)
        demand[0] = part[e];
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

// T <= TMAX (<= PERM_BLOCK): top-K of every token (one wavefront per token),
// then the histogram, scans and scatter, by one 1024-thread workgroup, with a
// bitmask of W = ceil(T / 32) words per expert (`bits`, E * W words of LDS).
// The logits are read from L (bias included).  With select == 0 the
// selection is read from o.idx / o.w instead.  CLEARED: the caller zeroed
// the bitmask before its last barrier.
template <int PER, int TMAX, bool CLEARED = false>
__device__ __forceinline__ void route_small_body(uint32_t *bits, const float *L, int select, const RouteOut &o,
                                                 int T, int K, int E)
{
    __shared__ int32_t excl[1024];              // first permuted row of each expert
    __shared__ int32_t wsum[16];
    __shared__ int32_t sidx[TMAX * 16];         // this workgroup's selection (K <= 16)
    __shared__ float sw[TMAX * 16];
    __shared__ float cand_v[16][64];
    __shared__ int32_t cand_e[16][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int W = (T + 31) >> 5;
    if constexpr (!CLEARED) {
        for (int i = threadIdx.x; i < E * W; i += blockDim.x)
            bits[i] = 0;
        __syncthreads();
    }
    if (select) {
        for (int t = wave; t < T; t += 16) {
            float v[PER];
            load_logits<PER>(v, L, t, E, lane);
            wave_select<PER>(v, E, K, lane, cand_v[wave], cand_e[wave], [&](int rank, int e, float wt) {
                o.idx[t * K + rank] = e;
                o.w[t * K + rank] = wt;
                sidx[t * K + rank] = e;
                sw[t * K + rank] = wt;
                atomicOr(&bits[e * W + (t >> 5)], 1u << (t & 31));
            });
        }
    } else {
        for (int a = threadIdx.x; a < T * K; a += blockDim.x) {
            const int t = a / K, e = o.idx[a];
            sidx[a] = e;
            sw[a] = o.w[a];
            atomicOr(&bits[e * W + (t >> 5)], 1u << (t & 31));
        }
    }
    __syncthreads();
    const int e = threadIdx.x;
    if (T == 1) {
        // one token: its K experts, ascending, are the demanded list and rows 0 .. K-1 of the permutation;
        // the first permuted row of expert e is the number of selected experts below e
        int below = 0;
        for (int k = 0; k < K; ++k)
            below += sidx[k] < e ? 1 : 0;
        if (e < E) {
            const bool mine = below < K && sidx[below] == e;
            o.counts[e] = mine ? 1 : 0;
            o.offsets[e] = below;
        }
        if (e < K) {
            o.demand[1 + e] = sidx[e];
            o.perm[e] = 0;
            o.inv[e] = e;
            o.row_weight[e] = sw[e];
        }
        if (e == 0) {
            o.offsets[E] = K;
            o.demand[0] = K;
        }
        return;
    }
    int c = 0;
    if (e < E)
        for (int q = 0; q < W; ++q)
            c += __popc(bits[e * W + q]);
    // one scan of (demanded << 16) + count: T * K <= 4096 keeps the halves apart
    const int packed = block_scan_incl_1024(c | (c > 0 ? 0x10000 : 0), wsum);
    const int incl = packed & 0xFFFF, nz = packed >> 16;
    excl[e] = incl - c;
    if (e < E) {
        o.counts[e] = c;
        o.offsets[e] = incl - c;
        if (c > 0)
            o.demand[nz] = e;                   // demanded experts, ascending, after the count
    }
    if (e == E - 1) {
        o.offsets[E] = incl;
        o.demand[0] = nz;
    }
    __syncthreads();
    for (int a = threadIdx.x; a < T * K; a += blockDim.x) {
        const int t = a / K;
        const int ee = sidx[a];
        const uint32_t *row = bits + ee * W;
        int r = excl[ee];
        for (int q = 0; q < (t >> 5); ++q)
            r += __popc(row[q]);
        r += __popc(row[t >> 5] & ((1u << (t & 31)) - 1u));
        o.perm[r] = t;
        o.inv[a] = r;
        o.row_weight[r] = sw[a];
    }
}

template <int PER>
__global__ void __launch_bounds__(1024) route_small_kernel(const float *__restrict__ L, int select, RouteOut o,
                                                           int T, int K, int E)
{
    extern __shared__ uint32_t bits[];          // [E][W]
    route_small_body<PER, PERM_BLOCK>(bits, L, select, o, T, K, E);
}

// ---------------------------------------------------------------- decode routing, bf16, T <= 16
// Logits, selection and permutation in one launch.  Workgroup g (16
// wavefronts) streams router rows 16 g .. 16 g + 15: its wavefronts take
// consecutive sixteenths of the K steps of 32, so each lane issues all of its
// loads at once (router rows as the 16x16x32 MFMA A operand, token rows as
// the B operand, both straight from memory).  The wavefront sums are added in
// a fixed order (four groups of four wavefronts, each group in wavefront
// order, then the groups in order, then the bias).  After storing its logits
// each workgroup releases them and counts itself in; the last to arrive (the
// counter wraps back to zero on its arrival) acquires every workgroup's
// logits and runs the selection and permutation of route_small_kernel.  No
// workgroup waits for another, so the launch completes in any schedule.
//
// STAGED (d <= 3584, at most 7 K steps per wavefront): the router rows are
// read with 16-byte loads that run along the rows (16 rows x 64 B per K step,
// 64 / (4 * steps) rows per load instruction) into the wavefront's own LDS
// region and the MFMA fragments are read back from there, as in the
// quantized stream kernels; loads in the fragment layout touch all 16 rows
// with every instruction.  A wavefront's LDS operations execute in order, so
// the region needs no barrier.  The regions (16 x 16 rows of 64 steps + 16
// bytes), the bitmask (up to 4 KiB) and the kernel's 30 KiB of static LDS
// must fit the workgroup's 160 KiB: 7 steps take 150 KiB, 8 would take 166.
constexpr int ROUTE_STAGE_MAX_STEPS = 7;

__host__ __device__ constexpr int route_stage_row_bytes(int steps) { return steps * 64 + 16; }

template <int PER, bool STAGED>
__global__ void __launch_bounds__(1024) route_decode_kernel(const uint16_t *__restrict__ x,
                                                            const uint16_t *__restrict__ wr,
                                                            const float *__restrict__ bias, float *L,
                                                            uint32_t *__restrict__ arrive, RouteOut o, int T, int d,
                                                            int K, int E)
{
    extern __shared__ uint32_t bits[];          // [E][1], then (STAGED) 16 wavefront regions
    __shared__ f32x4 red[16][64];
    __shared__ uint32_t last;
    constexpr int GROUPS = 4, WPG = 16 / GROUPS;   // summation groups, wavefronts per group
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nks = d / 32;
    const int per = (nks + 15) / 16;
    const int s0 = min(wave * per, nks), s1 = min(s0 + per, nks);
    const int e0 = int(blockIdx.x) * 16;
    const int j = lane & 15, kg = (lane >> 4) * 8;
    // issued before the router rows: the bias of this wavefront's output rows (wavefront 0) and the
    // selection's bitmask (one word per expert for T <= 32), which only the last workgroup uses
    float bv[4] = {0.f, 0.f, 0.f, 0.f};
    if (wave == 0 && bias) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
            bv[r] = bias[min(e0 + 4 * (lane >> 4) + r, E - 1)];
    }
    for (int i = threadIdx.x; i < E; i += blockDim.x)
        bits[i] = 0;
    // rows past E and tokens past T read a valid row; their sums are never stored
    const uint16_t *xp = x + int64_t(min(j, T - 1)) * d + kg;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    if constexpr (STAGED) {
        const int nst = s1 - s0, cpr = 4 * nst;        // K steps and 16-byte chunks per row
        const int RS = route_stage_row_bytes(per);
        uint8_t *wst = reinterpret_cast<uint8_t *>(bits + ((E + 3) & ~3)) + wave * 16 * RS;
        u32x4 v[ROUTE_STAGE_MAX_STEPS], xv[ROUTE_STAGE_MAX_STEPS];
#pragma unroll
        for (int k = 0; k < ROUTE_STAGE_MAX_STEPS; ++k)
            if (k < nst) {
                const int ci = 64 * k + lane, row = ci / cpr, ch = ci % cpr;
                v[k] = load_stream16(wr + int64_t(min(e0 + row, E - 1)) * d + s0 * 32 + 8 * ch);
                xv[k] = *reinterpret_cast<const u32x4 *>(xp + s0 * 32 + 32 * k);
            }
#pragma unroll
        for (int k = 0; k < ROUTE_STAGE_MAX_STEPS; ++k)
            if (k < nst) {
                const int ci = 64 * k + lane, row = ci / cpr, ch = ci % cpr;
                *reinterpret_cast<u32x4 *>(wst + row * RS + 16 * ch) = v[k];
            }
#pragma unroll
        for (int k = 0; k < ROUTE_STAGE_MAX_STEPS; ++k)
            if (k < nst) {
                const u32x4 wv = *reinterpret_cast<const u32x4 *>(wst + j * RS + 64 * k + 2 * kg);
                acc = mfma16(as_bf16x8(wv), as_bf16x8(xv[k]), acc);
            }
    } else {
        const uint16_t *wp = wr + int64_t(min(e0 + j, E - 1)) * d + kg;
        for (int st = s0; st < s1; st += 4) {
            u32x4 wv[4], xv[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int k = min(st + u, s1 - 1) * 32;       // clamped: no branch around the loads
                wv[u] = load_stream16(wp + k);
                xv[u] = *reinterpret_cast<const u32x4 *>(xp + k);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (st + u < s1)
                    acc = mfma16(as_bf16x8(wv[u]), as_bf16x8(xv[u]), acc);
        }
    }
    red[wave][lane] = acc;
    __syncthreads();
    if (wave == 0) {
        if (j < T) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int e = e0 + 4 * (lane >> 4) + r;
                float a = 0.f;
#pragma unroll
                for (int q = 0; q < GROUPS; ++q) {
                    float pq = red[q * WPG][lane][r];
#pragma unroll
                    for (int u = 1; u < WPG; ++u)
                        pq += red[q * WPG + u][lane][r];
                    a = q == 0 ? pq : a + pq;
                }
                if (e < E)
                    L[int64_t(j) * E + e] = a + bv[r];
            }
        }
        // release: only this wavefront stored logits
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        const bool is_last = atomicInc(arrive, gridDim.x - 1u) == gridDim.x - 1u;
        if (is_last)
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");   // every workgroup's logits
        last = is_last ? 1u : 0u;
    }
    __syncthreads();                            // orders this workgroup's reads after the acquire
    if (!last)
        return;
    route_small_body<PER, 16, true>(bits, L, 1, o, T, K, E);
}

// ---------------------------------------------------------------- launchers

hipError_t init_route_attributes()
{
    hipError_t e = hipSuccess;
    auto set = [&](const void *f) {
        if (e == hipSuccess)
            e = allow_large_lds(f);
    };
    set(reinterpret_cast<const void *>(&route_small_kernel<2>));
    set(reinterpret_cast<const void *>(&route_small_kernel<4>));
    set(reinterpret_cast<const void *>(&route_small_kernel<8>));
    set(reinterpret_cast<const void *>(&route_small_kernel<16>));
    set(reinterpret_cast<const void *>(&route_decode_kernel<2, true>));
    set(reinterpret_cast<const void *>(&route_decode_kernel<4, true>));
    set(reinterpret_cast<const void *>(&route_decode_kernel<8, true>));
    set(reinterpret_cast<const void *>(&route_decode_kernel<16, true>));
    return e;
}

hipError_t launch_router_logits_f32(const float *x, const float *wr, const float *bias, float *L, int T,
                                    int d, int E, hipStream_t s)
{
    const int64_t n = int64_t(T) * E;
    if (n == 0)
        return hipSuccess;
    launch_k(router_logits_f32_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, s, x, wr, bias, L, T, d, E);
    return hipGetLastError();
}

template <int PER>
static void launch_route_decode_t(const uint16_t *x, const uint16_t *wr, const float *bias, float *L,
                                  uint32_t *arrive, const RouteOut &o, int T, int d, int K, int E, hipStream_t s)
{
    const int per = (d / 32 + 15) / 16;
    const size_t bits = size_t((E + 3) & ~3) * sizeof(uint32_t);
    if (per <= ROUTE_STAGE_MAX_STEPS)
        launch_k(route_decode_kernel<PER, true>, unsigned((E + 15) / 16), 1024,
                 bits + size_t(16) * 16 * route_stage_row_bytes(per), s, x, wr, bias, L, arrive, o, T, d, K, E);
    else
        launch_k(route_decode_kernel<PER, false>, unsigned((E + 15) / 16), 1024, bits, s, x, wr, bias, L, arrive, o,
                 T, d, K, E);
}

hipError_t launch_route_decode(const uint16_t *x, const uint16_t *wr, const float *bias, float *L,
                               uint32_t *arrive, const RouteOut &o, int T, int d, int K, int E, hipStream_t s)
{
    if (T <= 0 || T > 16 || E <= 0 || E > 1024 || K <= 0 || K > 16 || d % 32 != 0 || !arrive)
        return hipErrorInvalidValue;
    const int per = (E + 63) / 64;
    if (per <= 2)
        launch_route_decode_t<2>(x, wr, bias, L, arrive, o, T, d, K, E, s);
    else if (per <= 4)
        launch_route_decode_t<4>(x, wr, bias, L, arrive, o, T, d, K, E, s);
    else if (per <= 8)
        launch_route_decode_t<8>(x, wr, bias, L, arrive, o, T, d, K, E, s);
    else
        launch_route_decode_t<16>(x, wr, bias, L, arrive, o, T, d, K, E, s);
    return hipGetLastError();
}

template <int PER>
static void launch_route_small_t(const float *L, const RouteOut &o, int T, int K, int E, hipStream_t s)
{
    const size_t lds = size_t(E) * std::max((T + 31) / 32, 1) * sizeof(uint32_t);
    launch_k(route_small_kernel<PER>, 1, 1024, lds, s, L, T > 0 ? 1 : 0, o, T, K, E);
}

hipError_t launch_route_select(const float *L, const RouteOut &o, int32_t *blockhist, int T, int K, int E,
                               hipStream_t s)
{
    const int per = (E + 63) / 64;
    if (T <= PERM_BLOCK) {
        // T == 0 still writes zero counts, offsets and demand
        if (per <= 2)
            launch_route_small_t<2>(L, o, T, K, E, s);
        else if (per <= 4)
            launch_route_small_t<4>(L, o, T, K, E, s);
        else if (per <= 8)
            launch_route_small_t<8>(L, o, T, K, E, s);
        else
            launch_route_small_t<16>(L, o, T, K, E, s);
        return hipGetLastError();
    }
    const dim3 grid(unsigned((T + 3) / 4)), block(256);
    if (per <= 2)
        launch_k(topk_kernel<2>, grid, block, 0, s, L, o.idx, o.w, T, E, K);
    else if (per <= 4)
        launch_k(topk_kernel<4>, grid, block, 0, s, L, o.idx, o.w, T, E, K);
    else if (per <= 8)
        launch_k(topk_kernel<8>, grid, block, 0, s, L, o.idx, o.w, T, E, K);
    else
        launch_k(topk_kernel<16>, grid, block, 0, s, L, o.idx, o.w, T, E, K);
    const size_t lds = size_t(E) * (PERM_BLOCK / 32) * sizeof(uint32_t);
    const int nblk = (T + PERM_BLOCK - 1) / PERM_BLOCK;
    launch_k(perm_hist_kernel, nblk, 256, lds, s, o.idx, blockhist, T, K, E);
    launch_k(perm_scan_kernel, 1, 1024, 0, s, blockhist, nblk, E, o.counts, o.offsets, o.demand);
    launch_k(perm_scatter_kernel, nblk, 256, lds, s, o.idx, o.w, blockhist, o.offsets, o.perm, o.inv, o.row_weight,
             T, K, E);
    return hipGetLastError();
}

}  // namespace msi
