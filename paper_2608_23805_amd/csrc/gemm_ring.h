// gemm_ring.h -- gate/up (SiLU-gated) and down projections of the routed
// experts on the tile path (experts with more than 16 routed rows), gfx950.
//
// The complete gate, up and down projections of every selected expert are
// computed (Section 5.4); outputs are the same per-row quantities as the
// stream path: act[row, I] = silu(x Wg^T) * (x Wu^T) and
// y[row, d] = row_weight * (act Wd^T), rows in permuted order, bf16.
//
// Tile: 256 routed rows x 256 weight rows (gate/up: 128 gate + the 128
// matching up rows; down: 256 output features), 8 wavefronts as 4 (rows) x 2
// (features), each 64 rows x 128 weight rows as 4 x 8 blocks of
// v_mfma_f32_16x16x32_bf16 with the weights as the A operand, so a lane ends
// with 4 consecutive output features of one row (8-byte packed stores, and
// SiLU(gate) * up formed in registers).  Two wavefronts per SIMD, fp32
// accumulators in VGPRs.
//
// K advances in stages of 32 elements.  A stage (256 A rows and 256 B rows of
// 64 bytes, 32 KiB) is copied from memory straight into LDS by buffer loads
// (no register staging), into a ring of four stage buffers: while stage s is
// multiplied, stages s+1 .. s+3 are in flight.  Each 16-byte chunk c of a
// stage row r sits at slot c ^ ((r >> 2) & 3) of the row, so both the copies
// (16 rows x 64 bytes per instruction) and the fragment reads (16 rows x 16
// bytes per 16 lanes) are free of LDS bank conflicts.  The fragments of
// stage s+1 are read while stage s is multiplied (weight fragments double
// buffered, each row fragment right after its last use), two reads per eight
// MFMAs.  The loop has no branches: stages past the end are loaded through a
// buffer resource with no records (the loads return zeros and touch no
// memory), so every step waits on the same counts.  Row blocks past the
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

enum class RingMode : int { GateUp = 0, Down = 1 };

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

inline int ring_tiles_gateup(int nrows, int I) { return ((nrows + ring::TM - 1) / ring::TM) * (I / 128); }
inline int ring_tiles_down(int nrows, int d) { return ((nrows + ring::TM - 1) / ring::TM) * (d / ring::TN); }

template <RingMode MODE>
__global__ void __launch_bounds__(ring::THREADS, 1) ring_gemm_kernel(ExpertLaunch L)
{
    using namespace ring;
    constexpr bool GU = MODE == RingMode::GateUp;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[NBUF * STAGE];

    const int t = xcd_swizzle(int(blockIdx.x), int(gridDim.x));
    const WorkItem it = L.items[find_item(L.items, L.n_items, t)];
    if (!slot_current(it, L.gen_dev, L.status))
        return;
    const int d = L.d, I = L.I;
    const int K = GU ? d : I;
    const int ntn = GU ? I / 128 : d / TN;
    const int local = t - it.tile0;
    const int m0 = (local / ntn) * TM;
    const int nt = local % ntn;
    const int valid = min(TM, it.nrows - m0);
    const bool sh = it.slot < 0;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;

    // ---- copy addressing: instruction i of this wavefront covers stage rows
    // 16 (i WAVES + wave) + lane / 4; lane % 4 is the 16-byte slot it fills
    const int rl = lane >> 2;
    const uint32_t cw = uint32_t(((lane & 3) ^ ((rl >> 2) & 3)) << 4);
    const void *abase = GU ? L.x : (sh ? L.act_s : L.act);
    uint32_t aoff[LA];
    bool areal[LA];
#pragma unroll
    for (int i = 0; i < LA; ++i) {
        const int blk = i * WAVES + wave;
        areal[i] = blk * 16 < valid;
        const int r = blk * 16 + rl;
        const int m = m0 + (r < valid ? r : 0);
        const uint32_t src = GU ? uint32_t(sh ? m : L.perm[it.row0 + m]) : uint32_t(it.row0 + m);
        aoff[i] = src * uint32_t(K * 2) + cw;
    }
    const uint8_t *wobj = sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const uint8_t *bbase = GU ? wobj : wobj + uint64_t(2) * I * d * 2;   // Wd follows Wg, Wu
    uint32_t boff[LB];
#pragma unroll
    for (int i = 0; i < LB; ++i) {
        const int r = (i * WAVES + wave) * 16 + rl;   // stage B row
        const int src = GU ? (r < 128 ? nt * 128 + r : I + nt * 128 + (r - 128)) : nt * TN + r;
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
            dma16_lds(br, buf + TM * ROWB + (i * WAVES + wave) * 1024, boff[i], kb);
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
    const uint32_t fofs = uint32_t((lane & 15) * ROWB + (((lane >> 4) ^ ((lane >> 2) & 3)) << 4));
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

    // ---- epilogue: lane holds row 16 b + lane % 16, features 16 a + 4 (lane / 16) + j
    const int64_t rowbase = int64_t(it.row0) + m0;
    if constexpr (GU) {
        uint16_t *out = static_cast<uint16_t *>(sh ? L.act_s : L.act);
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int row = wm * 64 + b * 16 + (lane & 15);
            if (row < valid) {
                uint16_t *dst = out + (rowbase + row) * I + nt * 128 + wn * 64 + 4 * (lane >> 4);
#pragma unroll
                for (int a = 0; a < 4; ++a) {
                    uint2 v;
                    v.x = pack_bf16x2(silu_hw(acc[a][b][0]) * acc[a + 4][b][0], silu_hw(acc[a][b][1]) * acc[a + 4][b][1]);
                    v.y = pack_bf16x2(silu_hw(acc[a][b][2]) * acc[a + 4][b][2], silu_hw(acc[a][b][3]) * acc[a + 4][b][3]);
                    *reinterpret_cast<uint2 *>(dst + a * 16) = v;
                }
            }
        }
    } else {
        uint16_t *out = static_cast<uint16_t *>(sh ? L.ys : L.y);
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int row = wm * 64 + b * 16 + (lane & 15);
            if (row < valid) {
                const float wgt = (sh || !L.row_weight) ? 1.0f : L.row_weight[rowbase + row];
                uint16_t *dst = out + (rowbase + row) * d + nt * TN + wn * 128 + 4 * (lane >> 4);
#pragma unroll
                for (int a = 0; a < 8; ++a) {
                    uint2 v;
                    v.x = pack_bf16x2(acc[a][b][0] * wgt, acc[a][b][1] * wgt);
                    v.y = pack_bf16x2(acc[a][b][2] * wgt, acc[a][b][3] * wgt);
                    *reinterpret_cast<uint2 *>(dst + a * 16) = v;
                }
            }
        }
    }
}

}  // namespace msi
