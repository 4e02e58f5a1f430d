// gemm_tile.h -- LDS-staged bf16 MFMA tile (gfx950, v_mfma_f32_32x32x16_bf16)
// for the router logits and the per-expert gate/up and down projections.
//
// C[m, n] = sum_k A[m, k] * B[n, k]: both operands have the reduction axis
// contiguous (x and act rows; router / expert weight rows).  A workgroup of
// 256 threads (4 wavefronts, 2 x 2) computes a BM x BN = 128 x 256 tile; each
// wavefront owns 64 x 128 as 2 x 4 blocks of 32 x 32.  K advances in BK = 32
// steps through a double-buffered LDS stage (60 KiB per workgroup, so two
// workgroups share a CU and each SIMD interleaves two wavefronts); the next
// stage's global loads are in flight while the current stage is computed.
//
// A rows are gathered through the permutation (row r of expert e's tile reads
// token perm[row0 + r]), so the permuted copy of x is never materialised.
// Every tile first checks the generation word of the slot it reads and writes
// nothing when the slot no longer denotes the scheduled version.
//
// Rows of one expert are always cut into tiles from the expert's first row
// with the same K order, and an MFMA output element depends only on its own
// A row and B column, so an expert's result for a token never depends on
// which other experts share the launch (capacity-independent outputs).
#pragma once

#include "common.h"

namespace msi {

namespace tile {
constexpr int BM = 128;
constexpr int BN = 256;
constexpr int BK = 32;
constexpr int LDK = BK + 8;   // 80-byte LDS row pitch: conflict-free 16-byte fragment reads
constexpr int THREADS = 256;
constexpr int A_LOADS = BM * (BK / 8) / THREADS;   // 16-byte loads per thread per stage
constexpr int B_LOADS = BN * (BK / 8) / THREADS;
constexpr size_t LDS_BYTES = size_t(2) * (BM + BN) * LDK * sizeof(uint16_t);
}  // namespace tile

enum class TileMode : int { Router = 0, GateUp = 1, Down = 2 };

struct TileArgs {
    const uint16_t *a;          // A rows (x or act), bf16
    int64_t lda;                // elements per A row
    const int32_t *perm;        // gather map (A row = perm[row0 + m]) or null (A row = row0 + m)
    const uint8_t *wbase;       // slot pool, shared object or router weight
    uint64_t wstride;           // bytes between slots
    int K;                      // reduction length (d or I)
    int n_valid;                // valid B rows (router: E) for masking
    int n_tiles_n;              // N tiles per item
    int d, I;
    const WorkItem *items;      // device list, or null to use `single`
    int n_items;
    WorkItem single;
    const uint32_t *gen_dev;
    uint32_t *status;
    void *out;                  // L (fp32), act (bf16) or Y (bf16)
    int64_t ldo;                // elements per output row
    const float *bias;          // router bias or null
    const float *row_weight;    // gate weight per permuted row (down) or null (1.0)
    // items with slot < 0 (gate/up, down) are the shared expert: weights at
    // shared_w, A rows are tokens (gate/up) or rows of a_s (down), output to out_s
    const uint8_t *shared_w;
    const uint16_t *a_s;
    void *out_s;
};

// Stage helpers: row i of a thread's share sits THREADS / (BK / 8) rows below row i-1.
template <int N>
__device__ __forceinline__ void tile_load_rows(u32x4 (&r)[N], const uint16_t *base, const uint32_t (&off)[N],
                                               uint32_t k0)
{
#pragma unroll
    for (int i = 0; i < N; ++i)
        r[i] = *reinterpret_cast<const u32x4 *>(base + (off[i] + k0));
}

template <int N>
__device__ __forceinline__ void tile_store_rows(const u32x4 (&r)[N], uint16_t *dst)
{
#pragma unroll
    for (int i = 0; i < N; ++i)
        *reinterpret_cast<u32x4 *>(dst + (tile::THREADS / (tile::BK / 8)) * i * tile::LDK) = r[i];
}

template <TileMode MODE>
__device__ __forceinline__ int wave_col_block(int wn, int nb)
{
    if constexpr (MODE == TileMode::GateUp)
        return nb < 2 ? wn * 64 + nb * 32 : 128 + wn * 64 + (nb - 2) * 32;
    else
        return wn * 128 + nb * 32;
}

template <TileMode MODE>
__global__ void __launch_bounds__(tile::THREADS, 2) tile_gemm_kernel(TileArgs p)
{
    using namespace tile;
    extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
    uint16_t *As = lds;                         // [2][BM][LDK]
    uint16_t *Bs = lds + 2 * BM * LDK;          // [2][BN][LDK]

    const int t = xcd_swizzle(int(blockIdx.x), int(gridDim.x));
    const WorkItem it = p.items ? p.items[find_item(p.items, p.n_items, t)] : p.single;
    if (!slot_current(it, p.gen_dev, p.status))
        return;
    const int local = t - it.tile0;
    const int m0 = (local / p.n_tiles_n) * BM;
    const int nt = local % p.n_tiles_n;

    const bool sh = MODE != TileMode::Router && it.slot < 0;
    const uint16_t *abase = (MODE == TileMode::Down && sh) ? p.a_s : p.a;
    const int32_t *perm = sh ? nullptr : p.perm;
    void *outp = sh ? p.out_s : p.out;
    const float *rweight = sh ? nullptr : p.row_weight;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    constexpr int CPR = BK / 8;       // 16-byte chunks per stage row
    const int chunk = tid % CPR;
    const int rsub = tid / CPR;       // first row of this thread's share

    // ---- per-thread A / B row offsets (fixed over K): 32-bit element offsets
    // from uniform bases, so the loads use the scalar-base addressing form.
    // Rows past the tile's valid rows (or past the router's E columns) read
    // row 0 unmasked: an MFMA output element depends only on its own A row and
    // B column, and those outputs are never stored.  (Masking the loads would
    // put a divergent branch, and a full memory wait, behind every load.)
    uint32_t aoff[A_LOADS];
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i) {
        const int r = rsub + (THREADS / CPR) * i;
        int64_t src = 0;
        if (m0 + r < it.nrows)
            src = perm ? int64_t(perm[it.row0 + m0 + r]) : int64_t(it.row0 + m0 + r);
        aoff[i] = uint32_t(src * p.lda) + chunk * 8;
    }
    static_assert(THREADS / CPR * A_LOADS == BM && THREADS / CPR * B_LOADS == BN, "stage rows per thread");
    const uint8_t *base = MODE == TileMode::Router ? p.wbase
                          : sh                     ? p.shared_w
                                                   : p.wbase + uint64_t(it.slot) * p.wstride;
    const uint16_t *bbase = reinterpret_cast<const uint16_t *>(base) +
                            (MODE == TileMode::Down ? int64_t(2) * p.I * p.d : int64_t(0));
    uint32_t boff[B_LOADS];
#pragma unroll
    for (int j = 0; j < B_LOADS; ++j) {
        const int c = rsub + (THREADS / CPR) * j;
        int64_t brow;
        if constexpr (MODE == TileMode::GateUp)
            brow = (c < 128 ? int64_t(0) : int64_t(p.I)) + int64_t(nt) * 128 + (c & 127);   // Wu follows Wg
        else
            brow = int64_t(nt) * BN + c;
        if (MODE == TileMode::Router && brow >= p.n_valid)
            brow = 0;
        boff[j] = uint32_t(brow * p.K) + chunk * 8;
    }

    u32x4 ra0[A_LOADS], rb0[B_LOADS];
#define MSI_LOAD_STAGE(RA, RB, K0)                  \
    do {                                            \
        tile_load_rows(RA, abase, aoff, uint32_t(K0)); \
        tile_load_rows(RB, bbase, boff, uint32_t(K0)); \
    } while (0)
#define MSI_STORE_STAGE(RA, RB, BUF)                                     \
    do {                                                                 \
        tile_store_rows(RA, As + (BUF) * BM * LDK + rsub * LDK + chunk * 8); \
        tile_store_rows(RB, Bs + (BUF) * BN * LDK + rsub * LDK + chunk * 8); \
    } while (0)

    f32x16 acc[2][4];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[mb][nb][r] = 0.f;

    const int frow = lane & 31;
    const int fk = (lane >> 5) * 8;
    auto compute = [&](int buf) {
        const uint16_t *a = As + buf * BM * LDK;
        const uint16_t *b = Bs + buf * BN * LDK;
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            bf16x8 af[2], bfr[4];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
                af[mb] = as_bf16x8(*reinterpret_cast<const uint4 *>(a + (wm * 64 + mb * 32 + frow) * LDK + ks * 16 + fk));
#pragma unroll
            for (int nb = 0; nb < 4; ++nb)
                bfr[nb] = as_bf16x8(
                    *reinterpret_cast<const uint4 *>(b + (wave_col_block<MODE>(wn, nb) + frow) * LDK + ks * 16 + fk));
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int nb = 0; nb < 4; ++nb)
                    acc[mb][nb] = mfma32(af[mb], bfr[nb], acc[mb][nb]);
        }
    };

    // One register set: stage kt+1 is loaded while stage kt feeds the MFMAs
    // and written to the other LDS buffer afterwards.  Two workgroups per CU
    // (two wavefronts per SIMD) cover each other's load and barrier waits.
    const int nk = p.K / BK;
    MSI_LOAD_STAGE(ra0, rb0, 0);
    MSI_STORE_STAGE(ra0, rb0, 0);
    if (nk > 1)
        MSI_LOAD_STAGE(ra0, rb0, BK);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        compute(buf);
        if (kt + 1 < nk)
            MSI_STORE_STAGE(ra0, rb0, buf ^ 1);
        if (kt + 2 < nk)
            MSI_LOAD_STAGE(ra0, rb0, (kt + 2) * BK);
        __syncthreads();
    }
#undef MSI_LOAD_STAGE
#undef MSI_STORE_STAGE

    // ---- epilogue: lane holds rows 8*(r/4) + 4*(lane/32) + r%4, column lane%32 of each block
    const int col_l = lane & 31;
    if constexpr (MODE == TileMode::GateUp) {
        // act = silu(gate) * up in bf16, transposed through LDS (the main loop
        // is done with it) so that each lane stores 16 contiguous bytes
        constexpr int EP = 64 + 8;                     // per-wave [64 rows][64 cols] bf16, padded
        uint16_t *ep = lds + wave * 64 * EP;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int rl = mb * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
                    ep[rl * EP + nb * 32 + col_l] = f32_to_bf16(silu(acc[mb][nb][r]) * acc[mb][nb + 2][r]);
            }
        __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_wave_barrier();
        uint16_t *act = reinterpret_cast<uint16_t *>(outp);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int c = lane + 64 * i;                // 512 chunks of 8 bf16
            const int rl = c >> 3, q = c & 7;
            const int row = wm * 64 + rl;
            if (m0 + row < it.nrows)
                *reinterpret_cast<uint4 *>(act + (int64_t(it.row0) + m0 + row) * p.ldo + nt * 128 + wn * 64 + q * 8) =
                    *reinterpret_cast<const uint4 *>(ep + rl * EP + q * 8);
        }
        return;
    }
    if constexpr (MODE == TileMode::Down) {
        // y = row_weight * acc in bf16, transposed through LDS in two halves
        // of 64 columns so that each lane stores 16 contiguous bytes
        constexpr int EP = 64 + 8;
        uint16_t *ep = lds + wave * 64 * EP;
        uint16_t *y = reinterpret_cast<uint16_t *>(outp);
        float wrow[2][16];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = wm * 64 + mb * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                wrow[mb][r] = !rweight ? 1.0f : (m0 + row < it.nrows ? rweight[int64_t(it.row0) + m0 + row] : 0.f);
            }
#pragma unroll
        for (int half = 0; half < 2; ++half) {
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int rl = mb * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
#pragma unroll
                    for (int nb = 0; nb < 2; ++nb)
                        ep[rl * EP + nb * 32 + col_l] = f32_to_bf16(acc[mb][half * 2 + nb][r] * wrow[mb][r]);
                }
            __builtin_amdgcn_s_waitcnt(0);
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int c = lane + 64 * i;            // 512 chunks of 8 bf16
                const int rl = c >> 3, q = c & 7;
                const int row = wm * 64 + rl;
                if (m0 + row < it.nrows)
                    *reinterpret_cast<uint4 *>(y + (int64_t(it.row0) + m0 + row) * p.ldo + nt * BN + wn * 128 +
                                               half * 64 + q * 8) =
                        *reinterpret_cast<const uint4 *>(ep + rl * EP + q * 8);
            }
            __builtin_amdgcn_s_waitcnt(0);
            __builtin_amdgcn_wave_barrier();
        }
        return;
    }
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = wm * 64 + mb * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (m0 + row >= it.nrows)
                continue;
            const int64_t orow = int64_t(it.row0) + m0 + row;
            float *L = reinterpret_cast<float *>(p.out) + orow * p.ldo;
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                const int col = nt * BN + wn * 128 + nb * 32 + col_l;
                if (col < p.n_valid)
                    L[col] = acc[mb][nb][r] + (p.bias ? p.bias[col] : 0.f);
            }
        }
    }
}

}  // namespace msi
