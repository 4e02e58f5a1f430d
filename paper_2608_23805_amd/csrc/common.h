// common.h -- device helpers shared by the gfx950 kernels of the MoE layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

// s_waitcnt immediate (gfx9 encoding) that waits until at most n vector
// memory loads of the wavefront are outstanding; expcnt and lgkmcnt are left
// at their maxima, i.e. not waited for.
#define VMCNT_WAIT(n) ((((n) & 0xF) | (((n) >> 4) << 14)) | (0x7 << 4) | (0xF << 8))

namespace msi {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

// 16-byte streaming load (non-temporal: the data is read once)
__device__ __forceinline__ u32x4 load_stream16(const void *p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}

struct alignas(16) u16x8 {
    uint16_t v[8];
};

// tokens per block of the permutation's bitmask ranks
constexpr int PERM_BLOCK = 256;

// status word bits written by kernels that detect a problem
constexpr uint32_t STATUS_STALE = 1u;   // a tile saw a slot generation it did not expect
constexpr uint32_t STATUS_MISS = 2u;    // a demanded expert had no published slot (device work list)
constexpr uint32_t STATUS_DONE = 1u << 31;   // host copy only: the combine has published the status

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// binary32 -> bfloat16, round to nearest even (finite inputs; NaN stays NaN)
__device__ __forceinline__ uint16_t f32_to_bf16(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u)
        return uint16_t((u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u));
    u += 0x7FFFu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi)
{
    return uint32_t(f32_to_bf16(lo)) | (uint32_t(f32_to_bf16(hi)) << 16);
}

// SiLU(z) = z * sigmoid(z) = z / (1 + e^-z), with the device library's expf
__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

__device__ __forceinline__ f32x4 mfma16(const bf16x8 &a, const bf16x8 &b, const f32x4 &c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 mfma32(const bf16x8 &a, const bf16x8 &b, const f32x16 &c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

template <typename T>
__device__ __forceinline__ bf16x8 as_bf16x8(const T &v)
{
    return __builtin_bit_cast(bf16x8, v);
}

// Work item of one expert inside a launch: rows [row0, row0 + nrows) of the
// permuted order, weights at pool + slot * stride, expected generation gen.
// slot < 0 marks the shared expert (weights given directly, no generation).
struct WorkItem {
    int32_t expert;
    int32_t slot;      // global slot index (layer * pool_slots + s) or -1
    uint32_t gen;
    int32_t row0;
    int32_t nrows;
    int32_t tile0;     // first tile of this item in the launch's tile space
};

// Find the item owning tile `t` (items sorted by tile0, tile0[0] == 0).
__device__ __forceinline__ int find_item(const WorkItem *items, int n_items, int t)
{
    int lo = 0, hi = n_items - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (items[mid].tile0 <= t)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// Device-built work list of a decode forward: item i of a launch is the
// shared expert (i == 0, when there is one) or the (i - has_shared)-th
// demanded expert in ascending id, with its slot and generation from the
// layer's published residency table.  `demand` holds the number of demanded
// experts, then their ids ascending, as the routing wrote them.
struct DirectList {
    const int32_t *demand;       // [1 + E], or null: the launch has a host-built list
    const int32_t *slot_of;      // [E] published global slot of each expert of the layer, -1 if none
    const uint32_t *gen_of;      // [E] its published generation
    const int32_t *counts;       // [E] rows per expert
    const int32_t *offsets;      // [E + 1] first permuted row per expert
    int has_shared;
    int T;                       // rows of the shared expert
    int E;                       // experts of the layer (demand holds 1 + E words)
};

// Tile of workgroup b in a direct launch: the tiles of one item stay on one
// XCD (the hardware hands workgroup b to XCD b % 8) and items go round-robin
// over the XCDs, so the spread is even for any number of items.  The grid is
// a multiple of 8 * per_item.
__device__ __forceinline__ void direct_tile(int b, int per_item, int &item, int &local)
{
    const int q = b >> 3;
    item = (b & 7) + 8 * (q / per_item);
    local = q % per_item;
}

// Item i (tiles i * per_item ..) of a direct launch.  False past the last
// item.  A demanded expert without a published slot raises STATUS_MISS and
// comes back with nrows 0 (no work): the forward publishes nothing and is
// rescheduled by the host.  Every load is issued at a clamped, valid index
// before any branch (the empty asm statements keep the compiler from sinking
// them below one), so the lookup costs two dependent round trips.
__device__ __forceinline__ bool direct_item(const DirectList &D, int i, int per_item, uint32_t *status, WorkItem &it)
{
    const int j = i - D.has_shared;
    // (i is uniform: the values are kept in scalar registers)
    int n = __builtin_amdgcn_readfirstlane(D.demand[0]);
    int e = __builtin_amdgcn_readfirstlane(D.demand[1 + min(max(j, 0), D.E - 1)]);
    asm volatile("" : "+s"(n), "+s"(e));
    e = min(max(e, 0), D.E - 1);              // entries past n are stale: keep the reads in bounds
    int32_t s = __builtin_amdgcn_readfirstlane(D.slot_of[e]);
    int32_t r0 = __builtin_amdgcn_readfirstlane(D.offsets[e]);
    int32_t c = __builtin_amdgcn_readfirstlane(D.counts[e]);
    uint32_t g = __builtin_amdgcn_readfirstlane(D.gen_of[e]);
    asm volatile("" : "+s"(s), "+s"(r0), "+s"(c), "+s"(g));
    if (j >= n)
        return false;
    if (j < 0) {
        it = WorkItem{-1, -1, 0u, 0, D.T, 0};
        return true;
    }
    it = WorkItem{e, s, g, r0, s < 0 ? 0 : c, i * per_item};
    if (s < 0 && threadIdx.x == 0)
        atomicOr(status, STATUS_MISS);
    return true;
}

// Generation word of the tile's slot (read early, compared late).
__device__ __forceinline__ uint32_t slot_gen_now(const WorkItem &it, const uint32_t *gen_dev)
{
    return it.slot < 0 ? it.gen : __hip_atomic_load(gen_dev + it.slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ bool slot_gen_ok(const WorkItem &it, uint32_t g, uint32_t *status)
{
    asm volatile("" : "+v"(g));     // the compare stays here, after the work: the load's wait is not hoisted
    if (g == it.gen)
        return true;
    if (threadIdx.x == 0)
        atomicOr(status, STATUS_STALE);
    return false;
}

// Generation check done by every tile before it reads a slot: true if the
// slot denotes the version the host scheduled.  A mismatch raises the stale
// bit (vector atomic) and the tile must write nothing.
__device__ __forceinline__ bool slot_current(const WorkItem &it, const uint32_t *gen_dev, uint32_t *status)
{
    if (it.slot < 0)
        return true;
    uint32_t g = __hip_atomic_load(gen_dev + it.slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (g == it.gen)
        return true;
    if (threadIdx.x == 0)
        atomicOr(status, STATUS_STALE);
    return false;
}

// B-operand rows of one expert (n <= 16) staged into LDS [16][K + 8]:
// wavefront w handles rows w, w + 4, w + 8, w + 12, so each row's source
// index is wavefront-uniform; lane l takes 16-byte chunks l, l + 64, ...
// One pass covers 64 * CPL chunks of a row; rows longer than that take
// further passes.
template <int CPL>
struct StageRows {
    u32x4 v[4][CPL];

    __device__ __forceinline__ void load(const uint16_t *__restrict__ src, const int32_t *perm, int row0, int n,
                                         int K, int pass)
    {
        // the wavefront index is uniform: the row indices below are scalar
        const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
        const int lane = threadIdx.x & 63, cpr = K / 8;
        int64_t srow[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {             // all source rows first (clamped, no branch)
            const int r = min(wave + 4 * q, n - 1);
            srow[q] = perm ? int64_t(perm[row0 + r]) : int64_t(row0 + r);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (wave + 4 * q < n) {
#pragma unroll
                for (int c = 0; c < CPL; ++c) {
                    const int ch = lane + 64 * (pass * CPL + c);
                    if (ch < cpr)
                        v[q][c] = *reinterpret_cast<const u32x4 *>(src + srow[q] * K + ch * 8);
                }
            }
        }
    }

    __device__ __forceinline__ void store(uint16_t *xs, int n, int K, int pass) const
    {
        const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
        const int lane = threadIdx.x & 63, cpr = K / 8;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int r = wave + 4 * q;
            if (r < n) {
#pragma unroll
                for (int c = 0; c < CPL; ++c) {
                    const int ch = lane + 64 * (pass * CPL + c);
                    if (ch < cpr)
                        *reinterpret_cast<u32x4 *>(xs + r * (K + 8) + ch * 8) = v[q][c];
                }
            }
        }
    }

    // passes after the first (rows longer than 64 * CPL chunks)
    __device__ __forceinline__ void rest(const uint16_t *__restrict__ src, const int32_t *perm, int row0, int n,
                                         int K, uint16_t *xs)
    {
        for (int pass = 1; pass * 64 * CPL < K / 8; ++pass) {
            load(src, perm, row0, n, K, pass);
            store(xs, n, K, pass);
        }
    }
};

// ---- wavefront reductions and scans (64 lanes)
// Cross-lane moves without LDS: DPP (permutations and shifts within rows of
// 16 lanes, broadcasts of lanes 15 and 31) and the gfx950 lane swaps, which
// exchange lanes 16 or 32 apart.
namespace dpp {
constexpr int QUAD_1032 = 0xB1, QUAD_2301 = 0x4E;   // lanes l ^ 1, l ^ 2 within a quad
constexpr int ROW_SHR = 0x110;                      // + n: lane l - n of the same row
constexpr int ROW_MIRROR = 0x140, ROW_HALF_MIRROR = 0x141;
constexpr int ROW_BCAST15 = 0x142, ROW_BCAST31 = 0x143;
}  // namespace dpp

// v of the lane CTRL names, in the lanes the row and bank masks enable; 0 in
// the others and where the named lane lies outside the row.
template <int CTRL, int ROWS = 0xF, int BANKS = 0xF>
__device__ __forceinline__ uint32_t dpp_move(uint32_t v)
{
    return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), CTRL, ROWS, BANKS, true));
}

// op over all 64 lanes, the same value in every lane: each step combines lane
// l with a partner whose own step combines the same two values (commutative
// op, so all lanes agree bit for bit), in a fixed tree.
template <typename Op>
__device__ __forceinline__ float wave_reduce(float v, Op op)
{
    v = op(v, __uint_as_float(dpp_move<dpp::QUAD_1032>(__float_as_uint(v))));
    v = op(v, __uint_as_float(dpp_move<dpp::QUAD_2301>(__float_as_uint(v))));
    v = op(v, __uint_as_float(dpp_move<dpp::ROW_HALF_MIRROR>(__float_as_uint(v))));
    v = op(v, __uint_as_float(dpp_move<dpp::ROW_MIRROR>(__float_as_uint(v))));
    const auto s16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = op(__uint_as_float(s16[0]), __uint_as_float(s16[1]));
    const auto s32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return op(__uint_as_float(s32[0]), __uint_as_float(s32[1]));
}

__device__ __forceinline__ float wave_max(float v)
{
    return wave_reduce(v, [](float a, float b) { return fmaxf(a, b); });
}

__device__ __forceinline__ float wave_sum(float v)
{
    return wave_reduce(v, [](float a, float b) { return a + b; });
}

// Inclusive prefix sum over the 64 lanes: within each row the sums of up to
// 4, 8 and 16 preceding lanes, then the totals of rows 0 and 1 broadcast
// into the rows after them.
__device__ __forceinline__ int wave_scan_incl(int v)
{
    const uint32_t u = uint32_t(v);
    uint32_t s = u + dpp_move<dpp::ROW_SHR + 1>(u);
    s += dpp_move<dpp::ROW_SHR + 2>(u);
    s += dpp_move<dpp::ROW_SHR + 3>(u);
    s += dpp_move<dpp::ROW_SHR + 4, 0xF, 0xE>(s);
    s += dpp_move<dpp::ROW_SHR + 8, 0xF, 0xC>(s);
    s += dpp_move<dpp::ROW_BCAST15, 0xA, 0xF>(s);
    s += dpp_move<dpp::ROW_BCAST31, 0xC, 0xF>(s);
    return int(s);
}

__device__ __forceinline__ uint64_t lanemask_lt(int lane) { return (uint64_t(1) << lane) - 1; }

// Inclusive scan of one value per thread of a 1024-thread workgroup (wsum:
// 16 words of LDS): wavefront scans, then the totals of the earlier
// wavefronts (integers, so the grouping does not change the result).  The
// caller separates consecutive uses of wsum with a barrier.
__device__ __forceinline__ int block_scan_incl_1024(int v, int32_t *wsum)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int x = wave_scan_incl(v);
    if (lane == 63)
        wsum[wave] = x;
    __syncthreads();
    int base = 0;
    for (int w = 0; w < wave; ++w)
        base += wsum[w];
    return x + base;
}

// Inclusive scan of part[0..1023] in place by a 1024-thread workgroup.
__device__ __forceinline__ void block_scan_1024(int32_t *part)
{
    __shared__ int32_t wsum[16];
    const int e = threadIdx.x;
    const int x = block_scan_incl_1024(part[e], wsum);
    __syncthreads();
    part[e] = x;
    __syncthreads();
}

// Work counts of a launch whose work list was built on the device: the grid
// is an upper bound and each workgroup reads the list's length.
struct DevCount {
    int32_t n_items;
    int32_t n_tiles;
};

// Tile of workgroup b when n tiles exist and the grid may be larger: XCD x
// (b % 8) walks tiles [x per, (x + 1) per), per = ceil(n / 8), so the real
// tiles spread over every XCD however large the grid; -1 past the end.
__device__ __forceinline__ int xcd_tile(int b, int n)
{
    const int per = (n + 7) >> 3;
    const int q = b >> 3, t = (b & 7) * per + q;
    return (q < per && t < n) ? t : -1;
}

// Logical tile index with consecutive tiles kept on one XCD: hardware hands
// workgroup b to XCD b % 8, so XCD x walks tiles [x*per, (x+1)*per).
__device__ __forceinline__ int xcd_swizzle(int b, int n)
{
    const int per = n / 8;
    const int full = per * 8;
    if (b >= full)
        return b;
    return (b % 8) * per + (b / 8);
}

// Stream-path weight staging.  A wavefront's weights are 16 rows of W bytes
// each (its share of one row); per-lane 4-byte loads of the MFMA layout would
// touch 16 rows per load instruction, so the wavefront instead reads them with
// 16-byte loads that run along the rows (each instruction covers 64 / (W / 16)
// rows), writes them to its own LDS region, and reads the MFMA words back.
// Rows are padded by 16 bytes there, which puts the 64 lanes' word reads on
// distinct banks.  The region is the wavefront's alone, so no workgroup
// barrier is needed, and no wait either: a wavefront's LDS operations execute
// in order (a read after a write to the same address returns the written
// value, a write after a read cannot overtake it), and the compiler keeps the
// program order of these accesses because it cannot prove that the stored and
// the read addresses differ.  (An explicit lgkmcnt(0) wait around the writes
// made the kq decode gate/up kernel 65% slower.)
template <int W>
struct WaveRows {
    static constexpr int RS = W + 16;                  // LDS bytes per row
    static constexpr int CPR = W / 16;                 // 16-byte chunks per row
    static constexpr int NL = (16 * CPR + 63) / 64;    // load instructions
    u32x4 v[NL];

    // rows row0 .. row0 + 15 of stride `stride` bytes, W bytes from `src` on
    __device__ __forceinline__ void load(const uint8_t *src, int64_t stride, int lane)
    {
#pragma unroll
        for (int k = 0; k < NL; ++k) {
            const int ci = 64 * k + lane, row = ci / CPR, ch = ci % CPR;
            if (row < 16)
                v[k] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(src + row * stride + 16 * ch));
        }
    }
    // write the rows to the wavefront's region (see below for why no wait follows)
    __device__ __forceinline__ void store(uint8_t *lds, int lane) const
    {
#pragma unroll
        for (int k = 0; k < NL; ++k) {
            const int ci = 64 * k + lane, row = ci / CPR, ch = ci % CPR;
            if (row < 16)
                *reinterpret_cast<u32x4 *>(lds + row * RS + 16 * ch) = v[k];
        }
    }
};

}  // namespace msi
