// gemm_ring.h -- gate/up (SiLU-gated) and down projections of the routed
// experts on the tile path (experts with more than 16 routed rows), gfx950.
//
// The complete gate, up and down projections of every selected expert are
// computed ("Output-Exact Execution Beyond the Full-Residency Envelope"); outputs are the same per-row quantities as the
// stream path: act[row, I] = silu(x Wg^T) * (x Wu^T) and
// y[row, d] = row_weight * (act Wd^T), rows in permuted order, bf16.
//
// Tile: 256 routed rows x 256 weight rows (gate/up: 128 gate + the 128
// matching up rows; down: 256 output features), 8 wavefronts as 4 (rows) x 2
// (features), each 64 rows x 128 weight rows as 4 x 8 blocks of
// v_mfma_f32_16x16x32_bf16 with the weights as the A operand, so a lane ends
// with 4 consecutive output features of one row (SiLU(gate) * up formed in
// registers).  Two wavefronts per SIMD, fp32
// accumulators in VGPRs.
//
// K advances in stages of 32 elements.  A stage (256 A rows and 256 B rows of
// 64 bytes, 32 KiB) is copied from memory straight into LDS by buffer loads
// (no register staging), into a ring of four stage buffers: while stage s is
// multiplied, stages s+1 .. s+3 are in flight.  Each 16-byte chunk c of a
// stage row r sits at slot c ^ ring_swz(r) of the row (ring_swz below), so
// the fragment reads (16 rows x 16 bytes per 16 lanes) spread over all LDS
// banks whether the banks serve 16 lanes of 16 bytes or 8 lanes per cycle;
// the copies write 16 rows x 64 bytes per instruction.  The fragments of
// stage s+1 are read while stage s is multiplied (weight fragments double
// buffered, each row fragment right after its last use), two reads per eight
// MFMAs.  The loop has no branches: stages past the end are loaded through a
// buffer resource with no records (the loads touch no memory and write
// zeros to their LDS destination), so every step waits on the same counts.  Row blocks past the
// tile's valid rows are loaded the same way, and a wavefront whose 64 rows
// are all past the end keeps its share of the copies and the barriers but
// skips the MFMAs.
//
// A rows are gathered through the permutation (row r of expert e's tile is
// token perm[row0 + r]) while being copied, so the permuted copy of x is
// never materialised.  Every tile first checks the generation word of the
// slot it reads and writes nothing when the slot no longer denotes the
// scheduled version.  Rows of one expert are always cut into tiles from the
// expert's first row with the same K order, and an MFMA output element
// depends only on its own row and feature, so an expert's result for a token
// never depends on which other experts share the launch.
#pragma once

#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace msi {

// Slot permutation of the four 16-byte chunks of a 64-byte stage row, by the row's position within its
// 16-row block.  A fragment read has 16 lanes read chunk c of 16 consecutive rows: rows 4 apart share their
// 64-byte position modulo 256 bytes and rows 2 apart modulo 128 bytes, so the permutation gives distinct
// slots to rows {a, a+4, a+8, a+12} (16 lanes per 256-byte bank cycle) and to rows of equal parity within
// each half of 8 (8 lanes per 128-byte cycle).
__device__ __forceinline__ int ring_swz(int r) { return (((r >> 1) ^ (r >> 3)) & 1) | (((r >> 2) & 1) << 1); }

namespace ring {
constexpr int SK = 32;                       // K elements per stage
constexpr int ROWB = SK * 2;                 // bytes per stage row
constexpr int TM = 256;                      // routed rows per tile
constexpr int TN = 256;                      // weight rows per tile
constexpr int NBUF = 4;                      // stage buffers in the ring
constexpr int STAGE = (TM + TN) * ROWB;      // 32 KiB
constexpr int THREADS = 512;
constexpr int WAVES = THREADS / 64;
constexpr int LA = TM / 16 / WAVES;          // A copy instructions per wavefront per stage
constexpr int LB = TN / 16 / WAVES;          // B copy instructions per wavefront per stage
constexpr int LPS = LA + LB;
constexpr uint32_t RSRC_FLAGS = 0x00020000u; // raw buffer, 32-bit data format
}  // namespace ring

enum class RingMode : int { GateUp = 0, Down = 1, Router = 2 };

typedef __attribute__((address_space(3))) void lds_void_t;

// 64 lanes x 16 bytes from a buffer into LDS: lane i's bytes land at dst + 16 i.
// (The address-space cast is only meaningful in the device pass.)
__device__ __forceinline__ void dma16_lds(__amdgpu_buffer_rsrc_t r, void *dst, uint32_t voff, int soff)
{
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t *)dst, 16, voff, soff, 0, 0);
#else
    (void)r, (void)dst, (void)voff, (void)soff;
#endif
}

// SiLU(z) = z / (1 + e^-z) with the hardware base-2 exponential and reciprocal
__device__ __forceinline__ float silu_hw(float z)
{
    return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * z));
}

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_hw_t;

// two fp32 values -> packed bf16 pair, rounded to nearest even by the gfx950
// conversion instruction (identical to f32_to_bf16 for every non-NaN input)
__device__ __forceinline__ uint32_t pack_bf16x2_hw(float lo, float hi)
{
    const bf16x2_hw_t v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
    return __builtin_bit_cast(uint32_t, v);
}

// Output rows leave the MFMA tiles as 4-feature pieces: lane (i, j) (i = lane % 16, j = lane / 16) holds
// features 16 a + 4 j .. 16 a + 4 j + 3 of row i for every 16-feature block a, two bf16 per dword (lo: the
// first two, hi: the last two).  For two consecutive blocks a0, a0 + 1 this regroups the pieces so that
// lane (i, j) holds the 16 contiguous bytes 16 j .. 16 j + 15 of the 64 bytes the two blocks cover (lanes
// of rows j = 0, 1: block a0; j = 2, 3: block a0 + 1), and each store writes 64 contiguous bytes per row
// instead of four 8-byte pieces 32 bytes apart.  The 32-lane swap exchanges lanes 32 apart, the 16-lane
// swap lanes 16 apart (gfx950 lane permutes; every lane takes part, so they run outside row predicates).
__device__ __forceinline__ uint4 gather16(uint32_t lo0, uint32_t hi0, uint32_t lo1, uint32_t hi1)
{
    const auto l32 = __builtin_amdgcn_permlane32_swap(lo0, lo1, false, false);
    const auto h32 = __builtin_amdgcn_permlane32_swap(hi0, hi1, false, false);
    const auto l16 = __builtin_amdgcn_permlane16_swap(l32[0], l32[1], false, false);
    const auto h16 = __builtin_amdgcn_permlane16_swap(h32[0], h32[1], false, false);
    uint4 v;
    v.x = l16[0];
    v.y = h16[0];
    v.z = l16[1];
    v.w = h16[1];
    return v;
}

// Tile epilogue: lane holds row 16 q + lane % 16 of the wavefront's 64 rows and
// features 16 a + 4 (lane / 16) + j of its 128 weight rows.  Gate/up stores
// act = silu(gate) * up; down stores y = row_weight * acc; bf16, regrouped so
// each lane stores 16 contiguous bytes.  Addresses: a uniform tile base plus
// 32-bit lane offsets.
template <RingMode MODE>
__device__ __forceinline__ void ring_store(const ExpertLaunch &L, const f32x4 (&acc)[8][4], int64_t rowbase, int nt,
                                           int valid, bool sh, int wm, int wn, int lane_in)
{
    // (the lane index is made opaque so the store offsets are computed here, not kept live across the K loop)
    int lane = lane_in;
    asm volatile("" : "+v"(lane));
    if constexpr (MODE == RingMode::GateUp) {
        const int I = L.I;
        uint8_t *base = reinterpret_cast<uint8_t *>(static_cast<uint16_t *>(sh ? L.act_s : L.act) + rowbase * I +
                                                    nt * 128 + wn * 64);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            uint32_t lo[4], hi[4];
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                lo[a] = pack_bf16x2_hw(silu_hw(acc[a][q][0]) * acc[a + 4][q][0], silu_hw(acc[a][q][1]) * acc[a + 4][q][1]);
                hi[a] = pack_bf16x2_hw(silu_hw(acc[a][q][2]) * acc[a + 4][q][2], silu_hw(acc[a][q][3]) * acc[a + 4][q][3]);
            }
            const int row = wm * 64 + q * 16 + (lane & 15);
            const uint32_t off = uint32_t(row * I) * 2u + uint32_t(16 * (lane >> 4));
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const uint4 v = gather16(lo[2 * k], hi[2 * k], lo[2 * k + 1], hi[2 * k + 1]);
                if (row < valid)
                    *reinterpret_cast<uint4 *>(base + (off + uint32_t(64 * k))) = v;
            }
        }
    } else if constexpr (MODE == RingMode::Router) {
        const int E = L.E;
        float *base = L.logits + rowbase * E;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int row = wm * 64 + q * 16 + (lane & 15);
            if (row < valid) {
#pragma unroll
                for (int a = 0; a < 8; ++a) {
                    const int c = nt * ring::TN + wn * 128 + a * 16 + 4 * (lane >> 4);
                    float *dst = base + (row * E + c);
                    if (c + 3 < E) {
                        f32x4 v = acc[a][q];
                        if (L.bias) {
                            v[0] += L.bias[c];
                            v[1] += L.bias[c + 1];
                            v[2] += L.bias[c + 2];
                            v[3] += L.bias[c + 3];
                        }
                        *reinterpret_cast<f32x4 *>(dst) = v;
                    } else {
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            if (c + j < E)
                                dst[j] = acc[a][q][j] + (L.bias ? L.bias[c + j] : 0.0f);
                    }
                }
            }
        }
    } else {
        const int d = L.d;
        uint8_t *base = reinterpret_cast<uint8_t *>(static_cast<uint16_t *>(sh ? L.ys : L.y) + rowbase * d +
                                                    nt * ring::TN + wn * 128);
        const float *rw = (sh || !L.row_weight) ? nullptr : L.row_weight + rowbase;
        // all four row weights first, so one wait covers them (the stores below never wait on each other)
        float wq[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int row = wm * 64 + q * 16 + (lane & 15);
            wq[q] = (rw && row < valid) ? rw[row] : 1.0f;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int row = wm * 64 + q * 16 + (lane & 15);
            const float wgt = wq[q];
            uint32_t lo[8], hi[8];
#pragma unroll
            for (int a = 0; a < 8; ++a) {
                lo[a] = pack_bf16x2_hw(acc[a][q][0] * wgt, acc[a][q][1] * wgt);
                hi[a] = pack_bf16x2_hw(acc[a][q][2] * wgt, acc[a][q][3] * wgt);
            }
            const uint32_t off = uint32_t(row * d) * 2u + uint32_t(16 * (lane >> 4));
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint4 v = gather16(lo[2 * k], hi[2 * k], lo[2 * k + 1], hi[2 * k + 1]);
                if (row < valid)
                    *reinterpret_cast<uint4 *>(base + (off + uint32_t(64 * k))) = v;
            }
        }
    }
}

inline int ring_tiles_gateup(int nrows, int I) { return ((nrows + ring::TM - 1) / ring::TM) * (I / 128); }
inline int ring_tiles_down(int nrows, int d) { return ((nrows + ring::TM - 1) / ring::TM) * (d / ring::TN); }

template <RingMode MODE>
__global__ void __launch_bounds__(ring::THREADS, 1) ring_gemm_kernel(ExpertLaunch L)
{
    using namespace ring;
    constexpr bool GU = MODE == RingMode::GateUp;
    constexpr bool RT = MODE == RingMode::Router;     // router logits: one item of T token rows, E router rows
    __shared__ __attribute__((aligned(1024))) uint8_t lds[NBUF * STAGE];

    int n_items = 1, n_tiles = 0;
    const int t = RT ? xcd_swizzle(int(blockIdx.x), int(gridDim.x)) : launch_tile(L, n_items, n_tiles);
    if (t < 0)
        return;                                   // past the device-built list's tiles
    const WorkItem it = RT ? WorkItem{-1, -1, 0u, 0, L.T, 0} : L.items[find_item(L.items, n_items, t)];
    if (!RT && !slot_current(it, L.gen_dev, L.status))
        return;
    const int d = L.d, I = L.I;
    const int K = (GU || RT) ? d : I;
    const int ntn = RT ? (L.E + TN - 1) / TN : GU ? I / 128 : d / TN;
    const int local = t - it.tile0;
    const int m0 = (local / ntn) * TM;
    const int nt = local % ntn;
    const int valid = min(TM, it.nrows - m0);
    const bool sh = it.slot < 0;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);   // (uniform: scalar selects, no waterfall loops)

    // ---- copy addressing: instruction i of this wavefront covers stage rows
    // 16 (i WAVES + wave) + lane / 4; lane % 4 is the 16-byte slot it fills
    const int rl = lane >> 2;
    const uint32_t cw = uint32_t(((lane & 3) ^ ring_swz(rl & 15)) << 4);
    // A rows: gate/up and router gather token rows of x by their row index (the caller keeps x under 2^31
    // bytes); down reads the tile's own act rows, addressed from the tile's first row so the offsets stay
    // small for any number of rows
    const void *abase = (GU || RT) ? L.x
                                   : static_cast<const uint8_t *>(sh ? L.act_s : L.act) +
                                         (int64_t(it.row0) + m0) * int64_t(I) * 2;
    uint32_t aoff[LA];
    bool areal[LA];
#pragma unroll
    for (int i = 0; i < LA; ++i) {
        const int blk = i * WAVES + wave;
        areal[i] = blk * 16 < valid;
        const int r = blk * 16 + rl;
        const int m = m0 + (r < valid ? r : 0);
        const uint32_t src = !(GU || RT) ? uint32_t(m - m0) : !sh && GU ? uint32_t(L.perm[it.row0 + m])
                                                                         : uint32_t(it.row0 + m);
        aoff[i] = src * uint32_t(K * 2) + cw;
    }
    const uint8_t *wobj = RT ? L.wbase : sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const uint8_t *bbase = (GU || RT) ? wobj : wobj + uint64_t(2) * I * d * 2;   // Wd follows Wg, Wu
    uint32_t boff[LB];
    bool breal[LB];
#pragma unroll
    for (int i = 0; i < LB; ++i) {
        const int r = (i * WAVES + wave) * 16 + rl;   // stage B row
        int src = GU ? (r < 128 ? nt * 128 + r : I + nt * 128 + (r - 128)) : nt * TN + r;
        // router rows past E: whole 16-row blocks load zeros, a partial block reads row E - 1 (never stored)
        breal[i] = !RT || nt * TN + (i * WAVES + wave) * 16 < L.E;
        if (RT && src >= L.E)
            src = L.E - 1;
        boff[i] = uint32_t(src) * uint32_t(K * 2) + cw;
    }
    const int nstage = K / SK;
    const __amdgpu_buffer_rsrc_t none = __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(abase), 0, 0, RSRC_FLAGS);
    auto issue = [&](int stage) {
        const bool real = stage < nstage;
        const __amdgpu_buffer_rsrc_t ar =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(abase), 0, real ? 0x7fffffff : 0, RSRC_FLAGS);
        const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint8_t *>(bbase), 0, real ? 0x7fffffff : 0, RSRC_FLAGS);
        uint8_t *buf = lds + (stage % NBUF) * STAGE;
        const int kb = stage * ROWB;
#pragma unroll
        for (int i = 0; i < LA; ++i)
            dma16_lds(areal[i] ? ar : none, buf + (i * WAVES + wave) * 1024, aoff[i], kb);
#pragma unroll
        for (int i = 0; i < LB; ++i)
            dma16_lds(breal[i] ? br : none, buf + TM * ROWB + (i * WAVES + wave) * 1024, boff[i], kb);
    };
    auto sync_stage = [&](auto waitn) {
        __builtin_amdgcn_s_waitcnt(VMCNT_WAIT(decltype(waitn)::value));
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };
    using W_STEADY = std::integral_constant<int, LPS * (NBUF - 3)>;   // stage s+1 landed, s+2 in flight
    using W_FIRST = std::integral_constant<int, LPS * (NBUF - 2)>;    // stage 0 landed, 1 and 2 in flight

    // ---- fragment addressing: row lane % 16 of a 16-row block, chunk lane / 16
    const int wm = wave >> 1, wn = wave & 1;
    const uint32_t fofs = uint32_t((lane & 15) * ROWB + (((lane >> 4) ^ ring_swz(lane & 15)) << 4));
    auto wrow = [&](int a) { return GU ? (a < 4 ? wn * 64 + a * 16 : 128 + wn * 64 + (a - 4) * 16) : wn * 128 + a * 16; };

#pragma unroll
    for (int s = 0; s < NBUF - 1; ++s)
        issue(s);
    sync_stage(W_FIRST{});

    if (wm * 64 >= valid) {
        // every row of this wavefront is past the end: copies and barriers only
        for (int s = 0; s < nstage; ++s) {
            sync_stage(W_STEADY{});
            issue(s + NBUF - 1);
        }
        return;
    }

    f32x4 acc[8][4];   // [weight block][row block]
#pragma unroll
    for (int a = 0; a < 8; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
            acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    u32x4 fw[2][8], fx[4];
    {
        const uint8_t *b0 = lds + fofs;
#pragma unroll
        for (int a = 0; a < 8; ++a)
            fw[0][a] = *reinterpret_cast<const u32x4 *>(b0 + TM * ROWB + wrow(a) * ROWB);
#pragma unroll
        for (int b = 0; b < 4; ++b)
            fx[b] = *reinterpret_cast<const u32x4 *>(b0 + (wm * 64 + b * 16) * ROWB);
    }
    // one K step: MFMAs of stage s from fw[H] / fx, reading stage s+1's fragments
    // (the last step reads a stale buffer; those values are never used)
    auto step = [&](int s, auto h) {
        constexpr int H = decltype(h)::value;
        const uint8_t *nb = lds + ((s + 1) % NBUF) * STAGE + fofs;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
#pragma unroll
            for (int a = 0; a < 8; ++a)
                acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(fw[H][a]), as_bf16x8(fx[b]), acc[a][b],
                                                                    0, 0, 0);
#pragma unroll
            for (int q = 0; q < 2; ++q)
                fw[H ^ 1][b * 2 + q] = *reinterpret_cast<const u32x4 *>(nb + TM * ROWB + wrow(b * 2 + q) * ROWB);
            fx[b] = *reinterpret_cast<const u32x4 *>(nb + (wm * 64 + b * 16) * ROWB);
        }
        // four MFMAs, two fragment reads, four MFMAs, one read
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
    };
    // step s: stage s+1 has landed (s+2 may be in flight), stage s+3 goes into
    // the buffer of stage s-1, which every wavefront has finished reading
    for (int s = 0; s < nstage; s += 2) {
        sync_stage(W_STEADY{});
        issue(s + NBUF - 1);
        step(s, std::integral_constant<int, 0>{});
        sync_stage(W_STEADY{});
        issue(s + NBUF);
        step(s + 1, std::integral_constant<int, 1>{});
    }

    ring_store<MODE>(L, acc, int64_t(it.row0) + m0, nt, valid, sh, wm, wn, lane);
}


// ---------------------------------------------------------------- persistent form
//
// One workgroup per CU walks a sequence of tiles: XCD x (workgroup b runs on
// XCD b % 8) owns the contiguous tile range [x per, (x + 1) per) and its
// workgroups interleave over it, so the tiles that share rows and weights run
// together in one L2.  The stage stream runs on across tiles: the last three
// steps of a tile already copy the first three stages of the next one, so the
// pipeline never drains and the epilogue's stores overlap the next tile's
// copies.  The next tile's item is found after each epilogue by walking
// forward from the current item (scalar loads); for gate/up its 256 gather
// indices reach LDS through one extra copy per wavefront per step (zero
// records, into a spare LDS area, except at step 2, so every step still waits
// on the same count) and
// are turned into copy offsets at step nstage - 4.  Requires K / 32 >= 8.

struct RingTile {
    int ii;             // item index
    int row0, m0, nt, valid, slot;
    uint32_t gen;
    int sh;             // shared expert (an int: a struct without padding copies as plain registers)
    const uint8_t *bbase;
    const uint8_t *abase;   // A rows: x (gate/up, gathered) or the tile's first act row (down)
};

// The work list and the slot generations, read through the constant address space so the persistent
// kernel's per-tile lookups are scalar loads: those wait on their own counter, not behind the tile copies
// and output stores in flight.  (Generations are read once per tile, as a plain load would read them.)
#if defined(__HIP_DEVICE_COMPILE__)
#define MSI_SCALAR_AS __attribute__((address_space(4)))
#else
#define MSI_SCALAR_AS
#endif
template <class T>
__device__ __forceinline__ const MSI_SCALAR_AS T *scalar_view(const T *p)
{
    return (const MSI_SCALAR_AS T *)p;
}

template <RingMode MODE>
__device__ __forceinline__ RingTile ring_tile_at(const ExpertLaunch &L, int t, int ii, int n_items)
{
    const auto *items = scalar_view(L.items);
    while (ii + 1 < n_items && items[ii + 1].tile0 <= t)   // items are sorted by tile0
        ++ii;
    const WorkItem w = items[ii];
    constexpr bool GU = MODE == RingMode::GateUp;
    const int ntn = GU ? L.I / 128 : L.d / ring::TN;
    RingTile r;
    r.ii = ii;
    const int local = t - w.tile0;
    r.row0 = w.row0;
    r.m0 = (local / ntn) * ring::TM;
    r.nt = local % ntn;
    r.valid = min(ring::TM, w.nrows - r.m0);
    r.slot = w.slot;
    r.gen = w.gen;
    r.sh = w.slot < 0;
    const uint8_t *wobj = r.sh ? L.shared_w : L.wbase + uint64_t(w.slot) * L.wstride;
    r.bbase = GU ? wobj + uint64_t(r.nt) * 128 * L.d * 2
                 : wobj + (uint64_t(2) * L.I * L.d + uint64_t(r.nt) * ring::TN * L.I) * 2;
    r.abase = GU ? static_cast<const uint8_t *>(L.x)
                 : static_cast<const uint8_t *>(r.sh ? L.act_s : L.act) + (int64_t(w.row0) + r.m0) * int64_t(L.I) * 2;
    return r;
}

template <RingMode MODE>
__global__ void __launch_bounds__(ring::THREADS, 1) ring_gemm_persistent(ExpertLaunch L)
{
    using namespace ring;
    constexpr bool GU = MODE == RingMode::GateUp;
    constexpr int XP = GU ? 1 : 0;                          // extra copies per wavefront per step
    constexpr int LP = LPS + XP;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[NBUF * STAGE];
    // next tile's gather indices; the second half takes the extra copies that carry nothing (a copy through a
    // zero-record resource still writes its zeros to LDS)
    __shared__ __attribute__((aligned(256))) int32_t permlds[2 * WAVES * 64];

    const int d = L.d, I = L.I;
    const int K = GU ? d : I;
    const int nstage = K / SK;
    const int n = L.dev_n ? __builtin_amdgcn_readfirstlane(L.dev_n->n_tiles) : L.n_tiles;
    const int n_items = L.dev_n ? __builtin_amdgcn_readfirstlane(L.dev_n->n_items) : L.n_items;
    const int nwg = int(gridDim.x), b = int(blockIdx.x);
    int t, tend, tstep;
    if (nwg % 8 == 0) {
        const int per = (n + 7) / 8, x = b % 8;
        t = x * per + b / 8;
        tend = min(n, (x + 1) * per);
        tstep = nwg / 8;
    } else {
        t = b;
        tend = n;
        tstep = nwg;
    }
    if (t >= tend)
        return;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);   // (uniform: scalar selects, no waterfall loops)
    const int wm = wave >> 1, wn = wave & 1;
    const int rl = lane >> 2;
    const uint32_t cw = uint32_t(((lane & 3) ^ ring_swz(rl & 15)) << 4);
    uint32_t boff[LB];   // B rows of this lane's copies, relative to the tile's weight base
#pragma unroll
    for (int i = 0; i < LB; ++i) {
        const int r = (i * WAVES + wave) * 16 + rl;
        const int src = GU ? (r < 128 ? r : I + (r - 128)) : r;
        boff[i] = uint32_t(src) * uint32_t(K * 2) + cw;
    }
    const __amdgpu_buffer_rsrc_t none = __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(L.x), 0, 0, RSRC_FLAGS);
    const uint32_t fofs = uint32_t((lane & 15) * ROWB + (((lane >> 4) ^ ring_swz(lane & 15)) << 4));
    auto wrow = [&](int a) { return GU ? (a < 4 ? wn * 64 + a * 16 : 128 + wn * 64 + (a - 4) * 16) : wn * 128 + a * 16; };
    auto sync_stage = [&](auto waitn) {
        __builtin_amdgcn_s_waitcnt(VMCNT_WAIT(decltype(waitn)::value));
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };
    // row index within the tile of this lane's copy i (rows past the end read the tile's first row); the
    // lane index is made opaque so this is recomputed where used rather than kept live across the K loop
    auto arow = [&](const RingTile &T, int i) {
        int l = lane;
        asm volatile("" : "+v"(l));
        const int r = (i * WAVES + wave) * 16 + (l >> 2);
        return r < T.valid ? r : 0;
    };
    // stage copies: tile T's stage st into ring buffer B; !real (or past the tile's rows): zero-record loads
    auto issue = [&](const RingTile &T, const uint32_t (&ao)[LA], auto bufc, int st, bool real) {
        constexpr int B = decltype(bufc)::value;
        const __amdgpu_buffer_rsrc_t ar =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(T.abase), 0, real ? 0x7fffffff : 0, RSRC_FLAGS);
        const __amdgpu_buffer_rsrc_t br =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(T.bbase), 0, real ? 0x7fffffff : 0, RSRC_FLAGS);
        uint8_t *buf = lds + B * STAGE;
        const int kb = st * ROWB;
#pragma unroll
        for (int i = 0; i < LA; ++i)
            dma16_lds(((i * WAVES + wave) * 16 < T.valid) ? ar : none, buf + (i * WAVES + wave) * 1024, ao[i], kb);
#pragma unroll
        for (int i = 0; i < LB; ++i)
            dma16_lds(br, buf + TM * ROWB + (i * WAVES + wave) * 1024, boff[i], kb);
    };
    // the extra copy: at step 2 wavefront w brings the next tile's gather indices of rows 32 w .. 32 w + 31
    // (lanes 32..63 repeat them) into permlds[64 w ..]; zero records otherwise
    auto extra = [&](const RingTile &N, bool real) {
        if constexpr (GU) {
            const __amdgpu_buffer_rsrc_t pr =
                __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t *>(L.perm), 0, real ? 0x7fffffff : 0, RSRC_FLAGS);
            int l = lane;
            asm volatile("" : "+v"(l));
            const int r = 32 * wave + (l & 31);
            const uint32_t off = uint32_t(N.row0 + N.m0 + (r < N.valid ? r : 0)) * 4u;
#if defined(__HIP_DEVICE_COMPILE__)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(pr, (lds_void_t *)(permlds + (real ? 0 : WAVES * 64) + 64 * wave), 4,
                                                     off, 0, 0, 0);
#else
            (void)pr, (void)off;
#endif
        }
    };
    auto a_offsets = [&](const RingTile &T, uint32_t (&ao)[LA], bool from_lds) {
#pragma unroll
        for (int i = 0; i < LA; ++i) {
            const int r = arow(T, i);
            uint32_t src;
            if (GU)
                src = T.sh ? uint32_t(T.m0 + r) : (from_lds ? uint32_t(permlds[64 * (r >> 5) + (r & 31)])
                                                            : uint32_t(L.perm[T.row0 + T.m0 + r]));
            else
                src = uint32_t(r);                      // (down: rows relative to the tile's first row)
            int l = lane;                               // (opaque: the chunk offset is recomputed here too)
            asm volatile("" : "+v"(l));
            ao[i] = src * uint32_t(K * 2) + uint32_t(((l & 3) ^ ring_swz((l >> 2) & 15)) << 4);
        }
    };
    using W_STEADY = std::integral_constant<int, LP * (NBUF - 3)>;   // stage s+1 landed, s+2 in flight

    // ---- first tile (blocking)
    RingTile cur = ring_tile_at<MODE>(L, t, find_item(L.items, n_items, t), n_items);
    bool cur_ok = cur.sh || scalar_view(L.gen_dev)[cur.slot] == cur.gen;
    uint32_t aoff[LA];
    a_offsets(cur, aoff, false);
    issue(cur, aoff, std::integral_constant<int, 0>{}, 0, true);
    extra(cur, false);
    issue(cur, aoff, std::integral_constant<int, 1>{}, 1, true);
    extra(cur, false);
    issue(cur, aoff, std::integral_constant<int, 2>{}, 2, true);
    extra(cur, false);
    sync_stage(std::integral_constant<int, LP * (NBUF - 2)>{});

    u32x4 fw[8], fx[2][4];
    f32x4 acc[8][4];
    auto load_frags0 = [&]() {
        const uint8_t *b0 = lds + fofs;
#pragma unroll
        for (int a = 0; a < 8; ++a)
            fw[a] = *reinterpret_cast<const u32x4 *>(b0 + TM * ROWB + wrow(a) * ROWB);
#pragma unroll
        for (int q = 0; q < 4; ++q)
            fx[0][q] = *reinterpret_cast<const u32x4 *>(b0 + (wm * 64 + q * 16) * ROWB);
    };
    // MFMAs of step s (fragments in fw / fx[H]), weight block by weight block; with PREF the fragments of
    // stage s+1 are read in between: each weight fragment right after its last use, the row fragments into
    // the other buffer
    auto mma = [&](auto sbc, auto pref) {
        constexpr int SB = decltype(sbc)::value;          // step index mod 4 (K / 32 is a multiple of 4)
        constexpr int H = SB & 1;
        constexpr bool PREF = decltype(pref)::value;
        const uint8_t *nb = lds + ((SB + 1) % NBUF) * STAGE + fofs;
#pragma unroll
        for (int a = 0; a < 8; ++a) {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                acc[a][q] =
                    __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(fw[a]), as_bf16x8(fx[H][q]), acc[a][q], 0, 0, 0);
            if (PREF) {
                fw[a] = *reinterpret_cast<const u32x4 *>(nb + TM * ROWB + wrow(a) * ROWB);
                if (a & 1)
                    fx[H ^ 1][a >> 1] = *reinterpret_cast<const u32x4 *>(nb + (wm * 64 + (a >> 1) * 16) * ROWB);
            }
        }
        if (PREF) {
            // per weight block: four MFMAs, then its read (and every second block a row fragment read)
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
            }
        }
    };
    using PF = std::true_type;
    using NP = std::false_type;

    load_frags0();
    for (;;) {
#pragma unroll
        for (int a = 0; a < 8; ++a)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                acc[a][q] = f32x4{0.f, 0.f, 0.f, 0.f};
        // the next tile's item (scalar loads; first used by step 2's extra copy)
        const int tn = t + tstep;
        const bool has_next = tn < tend;
        const RingTile nxt = has_next ? ring_tile_at<MODE>(L, tn, cur.ii, n_items) : cur;
        const bool nxt_ok = nxt.sh || !has_next || scalar_view(L.gen_dev)[nxt.slot] == nxt.gen;

        using S0 = std::integral_constant<int, 0>;
        using S1 = std::integral_constant<int, 1>;
        using S2 = std::integral_constant<int, 2>;
        using S3 = std::integral_constant<int, 3>;
        // steps 0 .. nstage-5 (four per pass): copies of this tile's stages 3 .. nstage-2
        for (int s = 0; s < nstage - 4; s += 4) {
            sync_stage(W_STEADY{});
            issue(cur, aoff, S3{}, s + 3, true);
            extra(nxt, false);
            mma(S0{}, PF{});
            sync_stage(W_STEADY{});
            issue(cur, aoff, S0{}, s + 4, true);
            extra(nxt, false);
            mma(S1{}, PF{});
            sync_stage(W_STEADY{});
            issue(cur, aoff, S1{}, s + 5, true);
            extra(nxt, has_next && s == 0);
            mma(S2{}, PF{});
            sync_stage(W_STEADY{});
            issue(cur, aoff, S2{}, s + 6, true);
            extra(nxt, false);
            mma(S3{}, PF{});
        }
        // steps nstage-4 .. nstage-1: the last stage of this tile, then the next tile's stages 0 .. 2
        uint32_t naoff[LA];
        sync_stage(W_STEADY{});
        a_offsets(nxt, naoff, true);                // (the indices landed by step 4's barrier)
        issue(cur, aoff, S3{}, nstage - 1, true);
        extra(nxt, false);
        mma(S0{}, PF{});
        sync_stage(W_STEADY{});
        issue(nxt, naoff, S0{}, 0, has_next);
        extra(nxt, false);
        mma(S1{}, PF{});
        sync_stage(W_STEADY{});
        issue(nxt, naoff, S1{}, 1, has_next);
        extra(nxt, false);
        mma(S2{}, PF{});
        sync_stage(W_STEADY{});
        issue(nxt, naoff, S2{}, 2, has_next);
        extra(nxt, false);
        mma(S3{}, NP{});

        // ---- epilogue of this tile (the next tile's first stages are in flight)
        if (!cur_ok) {
            if (threadIdx.x == 0)
                atomicOr(L.status, STATUS_STALE);
        } else {
            ring_store<MODE>(L, acc, int64_t(cur.row0) + cur.m0, cur.nt, cur.valid, cur.sh, wm, wn, lane);
        }
        if (!has_next)
            break;
        t = tn;
        cur = nxt;
        cur_ok = nxt_ok;
#pragma unroll
        for (int i = 0; i < LA; ++i)
            aoff[i] = naoff[i];
        load_frags0();                               // stage 0 of the new tile (landed by the last barrier)
    }
}

}  // namespace msi
