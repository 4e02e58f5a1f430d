// gemm_tile.h -- LDS-staged bf16 MFMA tile (gfx950, v_mfma_f32_32x32x16_bf16)
// for the router logits and the per-expert gate/up and down projections.
//
// C[m, n] = sum_k A[m, k] * B[n, k]: both operands have the reduction axis
// contiguous (x and act rows; router / expert weight rows).  A workgroup of
// 256 threads (4 wavefronts, 2 x 2) computes a BM x BN = 128 x 256 tile; each
// wavefront owns 64 x 128 as 2 x 4 blocks of 32 x 32.  K advances in BK = 64
// steps through a double-buffered LDS stage, the next stage's global loads
// held in registers while the current stage feeds the MFMAs.
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
constexpr int BK = 64;
constexpr int LDK = BK + 8;   // 144-byte LDS row pitch: conflict-free 16-byte fragment reads
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
    void *out;                  // L (fp32), act (bf16) or Y (fp32)
    int64_t ldo;                // elements per output row
    const float *bias;          // router bias or null
    const float *row_weight;    // gate weight per permuted row (down) or null (1.0)
    // items with slot < 0 (gate/up, down) are the shared expert: weights at
    // shared_w, A rows are tokens (gate/up) or rows of a_s (down), output to out_s
    const uint8_t *shared_w;
    const uint16_t *a_s;
    void *out_s;
};

template <TileMode MODE>
__device__ __forceinline__ int wave_col_block(int wn, int nb)
{
    if constexpr (MODE == TileMode::GateUp)
        return nb < 2 ? wn * 64 + nb * 32 : 128 + wn * 64 + (nb - 2) * 32;
    else
        return wn * 128 + nb * 32;
}

template <TileMode MODE>
__global__ void __launch_bounds__(tile::THREADS, 1) tile_gemm_kernel(TileArgs p)
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
    const int chunk = tid & 7;        // 16-byte chunk of a 128-byte stage row
    const int rsub = tid >> 3;        // 0..31

    // ---- per-thread A / B row pointers (fixed over K)
    const uint16_t *aptr[A_LOADS];
    bool aval[A_LOADS];
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i) {
        const int r = rsub + 32 * i;
        aval[i] = m0 + r < it.nrows;
        int64_t src = 0;
        if (aval[i])
            src = perm ? int64_t(perm[it.row0 + m0 + r]) : int64_t(it.row0 + m0 + r);
        aptr[i] = abase + src * p.lda + chunk * 8;
    }
    const uint8_t *base = MODE == TileMode::Router ? p.wbase
                          : sh                     ? p.shared_w
                                                   : p.wbase + uint64_t(it.slot) * p.wstride;
    const uint16_t *bptr[B_LOADS];
    bool bval[B_LOADS];
#pragma unroll
    for (int j = 0; j < B_LOADS; ++j) {
        const int c = rsub + 32 * j;
        int64_t brow;
        const uint16_t *mat;
        if constexpr (MODE == TileMode::GateUp) {
            const uint16_t *wg = reinterpret_cast<const uint16_t *>(base);
            mat = c < 128 ? wg : wg + int64_t(p.I) * p.d;
            brow = int64_t(nt) * 128 + (c & 127);
            bval[j] = true;
        } else if constexpr (MODE == TileMode::Down) {
            mat = reinterpret_cast<const uint16_t *>(base) + int64_t(2) * p.I * p.d;
            brow = int64_t(nt) * BN + c;
            bval[j] = true;
        } else {
            mat = reinterpret_cast<const uint16_t *>(base);
            brow = int64_t(nt) * BN + c;
            bval[j] = brow < p.n_valid;
            if (!bval[j])
                brow = 0;
        }
        bptr[j] = mat + brow * p.K + chunk * 8;
    }

    uint4 ra[A_LOADS], rb[B_LOADS];
    auto load_stage = [&](int k0) {
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i)
            ra[i] = aval[i] ? *reinterpret_cast<const uint4 *>(aptr[i] + k0) : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int j = 0; j < B_LOADS; ++j)
            rb[j] = bval[j] ? *reinterpret_cast<const uint4 *>(bptr[j] + k0) : make_uint4(0, 0, 0, 0);
    };
    auto store_stage = [&](int buf) {
        uint16_t *a = As + buf * BM * LDK;
        uint16_t *b = Bs + buf * BN * LDK;
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i)
            *reinterpret_cast<uint4 *>(a + (rsub + 32 * i) * LDK + chunk * 8) = ra[i];
#pragma unroll
        for (int j = 0; j < B_LOADS; ++j)
            *reinterpret_cast<uint4 *>(b + (rsub + 32 * j) * LDK + chunk * 8) = rb[j];
    };

    f32x16 acc[2][4];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[mb][nb][r] = 0.f;

    const int nk = p.K / BK;
    load_stage(0);
    store_stage(0);
    if (nk > 1)
        load_stage(BK);
    __syncthreads();

    const int frow = lane & 31;
    const int fk = (lane >> 5) * 8;
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
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
        if (kt + 1 < nk)
            store_stage(buf ^ 1);
        if (kt + 2 < nk)
            load_stage((kt + 2) * BK);
        __syncthreads();
    }

    // ---- epilogue: lane holds rows 8*(r/4) + 4*(lane/32) + r%4, column lane%32 of each block
    const int col_l = lane & 31;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = wm * 64 + mb * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (m0 + row >= it.nrows)
                continue;
            const int64_t orow = int64_t(it.row0) + m0 + row;
            if constexpr (MODE == TileMode::GateUp) {
                uint16_t *act = reinterpret_cast<uint16_t *>(outp) + orow * p.ldo;
#pragma unroll
                for (int nb = 0; nb < 2; ++nb) {
                    const int col = nt * 128 + wn * 64 + nb * 32 + col_l;
                    act[col] = f32_to_bf16(silu(acc[mb][nb][r]) * acc[mb][nb + 2][r]);
                }
            } else if constexpr (MODE == TileMode::Down) {
                float *y = reinterpret_cast<float *>(outp) + orow * p.ldo;
                const float w = rweight ? rweight[orow] : 1.0f;
#pragma unroll
                for (int nb = 0; nb < 4; ++nb)
                    y[nt * BN + wn * 128 + nb * 32 + col_l] = acc[mb][nb][r] * w;
            } else {
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
}

}  // namespace msi
