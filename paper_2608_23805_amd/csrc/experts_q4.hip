// experts_q4.hip -- 4-bit block-quantized expert projections for gfx950.
//
// Storage (per matrix [rows, cols]): nibbles [rows, cols/2] (element 2j in the
// low nibble of byte j, 4-bit two's complement) then fp16 scales
// [rows, cols/32]; value = scale * q.  Dequantization is exact: q in [-8, 7]
// is exact in bf16, every 16x16x32 MFMA spans exactly one 32-element scale
// block, so it returns the block's partial dot product (C = 0) and the scale
// is applied in fp32: acc += scale * partial.
//
//  * stream path (<= 16 tokens per expert): weights as the A operand read
//    straight from memory, tokens as the B operand from LDS (as the bf16
//    stream path).
//  * tile path: 128 tokens x 128 weight rows per workgroup, packed nibbles and
//    scales staged in LDS (a quarter of the bf16 staging traffic), unpacked
//    to bf16 while the MFMA fragments are built.
#include "common.h"
#include "kernels.h"

namespace msi {

__device__ __forceinline__ uint32_t q4_matrix_bytes(int rows, int cols)
{
    return uint32_t(rows) * uint32_t(cols / 2) + uint32_t(rows) * uint32_t(cols / 32) * 2u;
}

// 8 nibbles (element e at bits 4e..4e+3) -> 8 exact bf16 values
__device__ __forceinline__ bf16x8 unpack_q4(uint32_t q)
{
    u32x4 r;
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        const int lo = int(q << (28 - 8 * h)) >> 28;          // element 2h
        const int hi = int(q << (24 - 8 * h)) >> 28;          // element 2h + 1
        r[h] = (__float_as_uint(float(lo)) >> 16) | (__float_as_uint(float(hi)) & 0xFFFF0000u);
    }
    return __builtin_bit_cast(bf16x8, r);
}

__device__ __forceinline__ float half_to_float(uint16_t h) { return float(__builtin_bit_cast(_Float16, h)); }

// ============================================================== stream path

namespace q4s {
constexpr int WAVES = 4, ROWS = 16;
}

int tiles_gateup_q4_stream(int nrows, int d, int I)
{
    (void)nrows;
    (void)d;
    return I / q4s::ROWS;
}

int tiles_down_q4_stream(int nrows, int d, int I)
{
    (void)nrows;
    (void)I;
    return d / (q4s::WAVES * q4s::ROWS);
}

// Tile t of a stream launch and its item: from the device-built list (the
// grid is then an upper bound) or the host list.
__device__ __forceinline__ bool q4_tile(const ExpertLaunch &L, int per_item, int &t, WorkItem &it)
{
    if (L.direct.demand) {
        int i, local;
        direct_tile(int(blockIdx.x), per_item, i, local);
        t = i * per_item + local;
        return direct_item(L.direct, i, per_item, L.status, it);
    }
    int n_items, n_tiles;
    t = launch_tile(L, n_items, n_tiles);
    if (t < 0)
        return false;
    it = L.items[find_item(L.items, n_items, t)];
    return true;
}

// CH consecutive fp16 block scales of one row, in one vector load (the row's
// scales start 16-byte aligned and CH divides the blocks of a quarter of d).
template <int CH>
__device__ __forceinline__ void load_scales(uint32_t (&w)[CH / 2], const uint16_t *p)
{
    if constexpr (CH == 16) {
        const u32x4 a = reinterpret_cast<const u32x4 *>(p)[0], b = reinterpret_cast<const u32x4 *>(p)[1];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            w[i] = a[i];
            w[4 + i] = b[i];
        }
    } else if constexpr (CH == 8) {
        const u32x4 a = *reinterpret_cast<const u32x4 *>(p);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            w[i] = a[i];
    } else if constexpr (CH == 4) {
        const uint2 a = *reinterpret_cast<const uint2 *>(p);
        w[0] = a.x;
        w[1] = a.y;
    } else {
        w[0] = *reinterpret_cast<const uint32_t *>(p);
    }
}

__device__ __forceinline__ float scale_at(const uint32_t *w, int b)
{
    return half_to_float(uint16_t(w[b >> 1] >> (16 * (b & 1))));
}

// Gate/up, 4-bit stream path: a workgroup owns 16 rows of Wg and of Wu; its
// four wavefronts take the four quarters of d and add their fp32 partial sums
// in wavefront order before SiLU(g) * u, so an item is I / 16 workgroups.
// Within a quarter, blocks go in chunks of CH: every nibble word and block
// scale of a chunk, for both matrices, is issued before its first MFMA.
// Lane (row r = lane % 16, group g = lane / 16) holds elements 8g .. 8g + 7 of
// each block of row r; the output lane (rows 4g .. 4g + 3, token lane % 16)
// applies those rows' block scales to each block's exact partial sum.
template <int CH>
__global__ void __launch_bounds__(256, 2) stream_gateup_q4_kernel(ExpertLaunch L)
{
    extern __shared__ __attribute__((aligned(16))) uint16_t xs[];
    __shared__ f32x4 red[3][2][64];
    int t;
    WorkItem it;
    if (!q4_tile(L, L.I / q4s::ROWS, t, it) || it.nrows == 0 ||
        !slot_current(it, L.gen_dev, L.status))      // nrows 0: unpublished expert, no work
        return;
    const int n = it.nrows, d = L.d, I = L.I, ldk = d + 8, nblk = d / 32, nq = nblk / q4s::WAVES;
    const bool sh = it.slot < 0;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int i0 = (t - it.tile0) * q4s::ROWS;
    const int r = lane & 15, g = lane >> 4;
    const int bq = wave * nq;                          // this wavefront's first block
    const uint8_t *base = sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const uint32_t mb = q4_matrix_bytes(I, d);
    const uint32_t *qp[2];
    const uint16_t *sp[2];
#pragma unroll
    for (int m = 0; m < 2; ++m) {
        const uint8_t *mat = base + m * mb;
        qp[m] = reinterpret_cast<const uint32_t *>(mat + int64_t(i0 + r) * (d / 2)) + 4 * bq + g;
        sp[m] = reinterpret_cast<const uint16_t *>(mat + int64_t(I) * (d / 2)) + int64_t(i0 + 4 * g) * nblk + bq;
    }
    uint32_t q[2][CH], sc[2][4][CH / 2];
    auto issue = [&](int c0) {
#pragma unroll
        for (int m = 0; m < 2; ++m) {
#pragma unroll
            for (int u = 0; u < CH; ++u)
                q[m][u] = __builtin_nontemporal_load(qp[m] + 4 * (c0 + u));
#pragma unroll
            for (int rr = 0; rr < 4; ++rr)
                load_scales<CH>(sc[m][rr], sp[m] + rr * nblk + c0);
        }
    };
    issue(0);                                          // the first chunk goes out before the token rows
    {
        const uint16_t *xsrc = reinterpret_cast<const uint16_t *>(L.x);
        const int32_t *xperm = sh ? nullptr : L.perm;
        StageRows<4> sr;                               // one pass for d <= 2048
        sr.load(xsrc, xperm, it.row0, n, d, 0);
        sr.store(xs, n, d, 0);
        sr.rest(xsrc, xperm, it.row0, n, d, xs);
    }
    __syncthreads();
    const uint16_t *xrow = xs + r * ldk + 8 * g + 32 * bq;   // rows past n hold stale data: not stored
    f32x4 ag = {0.f, 0.f, 0.f, 0.f}, au = {0.f, 0.f, 0.f, 0.f};
    for (int c0 = 0; c0 < nq; c0 += CH) {
        if (c0 > 0)
            issue(c0);
#pragma unroll
        for (int u = 0; u < CH; ++u) {
            const bf16x8 xb = as_bf16x8(*reinterpret_cast<const u32x4 *>(xrow + 32 * (c0 + u)));
            const f32x4 pg = mfma16(unpack_q4(q[0][u]), xb, f32x4{0.f, 0.f, 0.f, 0.f});
            const f32x4 pu = mfma16(unpack_q4(q[1][u]), xb, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                ag[rr] = fmaf(scale_at(sc[0][rr], u), pg[rr], ag[rr]);
                au[rr] = fmaf(scale_at(sc[1][rr], u), pu[rr], au[rr]);
            }
        }
    }
    // quarters of d added in wavefront order
    if (wave > 0) {
        red[wave - 1][0][lane] = ag;
        red[wave - 1][1][lane] = au;
    }
    __syncthreads();
    if (wave != 0)
        return;
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
        ag[rr] = ((ag[rr] + red[0][0][lane][rr]) + red[1][0][lane][rr]) + red[2][0][lane][rr];
        au[rr] = ((au[rr] + red[0][1][lane][rr]) + red[1][1][lane][rr]) + red[2][1][lane][rr];
    }
    const int j = lane & 15;
    if (j < n) {
        uint2 v;
        v.x = pack_bf16x2(silu(ag[0]) * au[0], silu(ag[1]) * au[1]);
        v.y = pack_bf16x2(silu(ag[2]) * au[2], silu(ag[3]) * au[3]);
        uint16_t *act = reinterpret_cast<uint16_t *>(sh ? L.act_s : L.act) + int64_t(it.row0 + j) * I + i0 + 4 * g;
        *reinterpret_cast<uint2 *>(act) = v;
    }
}

// Down, 4-bit stream path: a workgroup owns 64 output columns (16 per
// wavefront) over all of I, in chunks of CH blocks; the first chunk's nibble
// words and block scales are issued before the act rows are staged.
template <int CH>
__global__ void __launch_bounds__(256, 2) stream_down_q4_kernel(ExpertLaunch L)
{
    extern __shared__ __attribute__((aligned(16))) uint16_t as[];
    int t;
    WorkItem it;
    if (!q4_tile(L, L.d / (q4s::WAVES * q4s::ROWS), t, it) || it.nrows == 0 ||
        !slot_current(it, L.gen_dev, L.status))      // nrows 0: unpublished expert, no work
        return;
    const int n = it.nrows, d = L.d, I = L.I, ldk = I + 8, nblk = I / 32;
    const bool sh = it.slot < 0;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int c0 = ((t - it.tile0) * q4s::WAVES + wave) * q4s::ROWS;
    const int r = lane & 15, g = lane >> 4;
    const uint8_t *base = sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const uint8_t *wd = base + 2 * q4_matrix_bytes(I, d);
    const uint32_t *qp = reinterpret_cast<const uint32_t *>(wd + int64_t(c0 + r) * (I / 2)) + g;
    const uint16_t *sp = reinterpret_cast<const uint16_t *>(wd + int64_t(d) * (I / 2)) + int64_t(c0 + 4 * g) * nblk;
    uint32_t q[CH], sc[4][CH / 2];
    auto issue = [&](int b0) {
#pragma unroll
        for (int u = 0; u < CH; ++u)
            q[u] = __builtin_nontemporal_load(qp + 4 * (b0 + u));
#pragma unroll
        for (int rr = 0; rr < 4; ++rr)
            load_scales<CH>(sc[rr], sp + rr * nblk + b0);
    };
    issue(0);
    {
        const uint16_t *asrc = reinterpret_cast<const uint16_t *>(sh ? L.act_s : L.act);
        StageRows<1> sr;                               // one pass for I <= 512
        sr.load(asrc, nullptr, it.row0, n, I, 0);
        sr.store(as, n, I, 0);
        sr.rest(asrc, nullptr, it.row0, n, I, as);
    }
    __syncthreads();
    const uint16_t *arow = as + r * ldk + 8 * g;       // rows past n hold stale data: not stored
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int b0 = 0; b0 < nblk; b0 += CH) {
        if (b0 > 0)
            issue(b0);
#pragma unroll
        for (int u = 0; u < CH; ++u) {
            const bf16x8 ab = as_bf16x8(*reinterpret_cast<const u32x4 *>(arow + 32 * (b0 + u)));
            const f32x4 part = mfma16(unpack_q4(q[u]), ab, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
            for (int rr = 0; rr < 4; ++rr)
                acc[rr] = fmaf(scale_at(sc[rr], u), part[rr], acc[rr]);
        }
    }
    const int j = lane & 15;
    if (j < n) {
        const int64_t row = it.row0 + j;
        const float w = sh ? 1.0f : L.row_weight[row];
        *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(sh ? L.ys : L.y) + row * d + c0 + 4 * g) =
            make_uint2(pack_bf16x2(acc[0] * w, acc[1] * w), pack_bf16x2(acc[2] * w, acc[3] * w));
    }
}

hipError_t launch_gateup_q4_stream(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    // chunk: the largest of 16, 8, 4, 2 blocks dividing a quarter of d (d % 256 == 0)
    const int nq = L.d / 128;
    const size_t lds = size_t(16) * (L.d + 8) * 2;
    if (nq % 16 == 0)
        launch_k(stream_gateup_q4_kernel<16>, L.n_tiles, 256, lds, s, L);
    else if (nq % 8 == 0)
        launch_k(stream_gateup_q4_kernel<8>, L.n_tiles, 256, lds, s, L);
    else if (nq % 4 == 0)
        launch_k(stream_gateup_q4_kernel<4>, L.n_tiles, 256, lds, s, L);
    else
        launch_k(stream_gateup_q4_kernel<2>, L.n_tiles, 256, lds, s, L);
    return hipGetLastError();
}

hipError_t launch_down_q4_stream(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    // chunk: the largest of 16, 8, 4 blocks dividing I / 32 (I % 128 == 0)
    const int nblk = L.I / 32;
    const size_t lds = size_t(16) * (L.I + 8) * 2;
    if (nblk % 16 == 0)
        launch_k(stream_down_q4_kernel<16>, L.n_tiles, 256, lds, s, L);
    else if (nblk % 8 == 0)
        launch_k(stream_down_q4_kernel<8>, L.n_tiles, 256, lds, s, L);
    else
        launch_k(stream_down_q4_kernel<4>, L.n_tiles, 256, lds, s, L);
    return hipGetLastError();
}

// ============================================================== tile path

namespace q4t {
constexpr int BM = 128, BN = 128, BK = 64, THREADS = 256;
constexpr int LDA = BK + 8;                 // bf16 elements per staged A row
constexpr int LDQ = BK / 2 + 4;             // bytes per staged nibble row (36: conflict-spread)
constexpr int A_BYTES = BM * LDA * 2;
constexpr int Q_BYTES = BN * LDQ;
constexpr int S_BYTES = BN * (BK / 32) * 2;
constexpr int STAGE = A_BYTES + Q_BYTES + S_BYTES;
constexpr size_t LDS_BYTES = size_t(2) * STAGE;
}  // namespace q4t

int tiles_gateup_q4_tile(int nrows, int d, int I)
{
    (void)d;
    return ((nrows + q4t::BM - 1) / q4t::BM) * (I / 64);
}

int tiles_down_q4_tile(int nrows, int d, int I)
{
    (void)I;
    return ((nrows + q4t::BM - 1) / q4t::BM) * (d / q4t::BN);
}

TileGeom geom_gateup_q4_tile(int d, int I)
{
    (void)d;
    return TileGeom{q4t::BM, I / 64};
}

TileGeom geom_down_q4_tile(int d, int I)
{
    (void)I;
    return TileGeom{q4t::BM, d / q4t::BN};
}

// GATEUP: tile columns 0..63 are gate rows nt*64 .. nt*64+63, columns 64..127 the
// matching up rows; wavefront (wm, wn) owns rows wm*64.., gate columns
// wn*32.. and the matching up columns, so SiLU * up forms in registers.
template <bool GATEUP>
__global__ void __launch_bounds__(q4t::THREADS, 2) tile_q4_kernel(ExpertLaunch L)
{
    using namespace q4t;
    extern __shared__ __attribute__((aligned(16))) uint8_t lds8[];
    int n_items, n_tiles;
    const int t = launch_tile(L, n_items, n_tiles);
    if (t < 0)
        return;                                   // past the device-built list's tiles
    const WorkItem it = L.items[find_item(L.items, n_items, t)];
    if (!slot_current(it, L.gen_dev, L.status))
        return;
    const bool sh = it.slot < 0;
    const int d = L.d, I = L.I;
    const int K = GATEUP ? d : I;
    const int ntn = GATEUP ? I / 64 : d / BN;
    const int local = t - it.tile0;
    const int m0 = (local / ntn) * BM;
    const int nt = local % ntn;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    const uint16_t *abase = reinterpret_cast<const uint16_t *>(GATEUP ? L.x : (sh ? L.act_s : L.act));
    const int32_t *perm = (GATEUP && !sh) ? L.perm : nullptr;
    const uint8_t *obj = sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const uint32_t mbytes = q4_matrix_bytes(I, d);

    // A: 128 rows x 64 bf16 per stage = 8 chunks of 16 B per row; 4 per thread
    uint32_t aoff[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = (tid >> 3) + 32 * i;
        int64_t src = 0;
        if (m0 + r < it.nrows)
            src = perm ? int64_t(perm[it.row0 + m0 + r]) : int64_t(it.row0 + m0 + r);
        aoff[i] = uint32_t(src * K) + (tid & 7) * 8;
    }
    // B: 128 weight rows x 32 nibble bytes per stage: 2 chunks of 16 B per row, 1 per thread;
    // scales: 128 rows x 2 fp16 per stage, one 4-byte word per thread for tid < 128
    const int brow_l = tid >> 1, bchunk = tid & 1;
    auto weight_row = [&](int c) -> int {          // tile column -> matrix row
        if (GATEUP)
            return (c < 64 ? 0 : I) + nt * 64 + (c & 63);
        return nt * BN + c;
    };
    const int wr_b = weight_row(brow_l);
    const uint8_t *qmat = GATEUP ? obj + (wr_b >= I ? mbytes : 0u) : obj + 2 * mbytes;
    const int wr_local = GATEUP ? (wr_b >= I ? wr_b - I : wr_b) : wr_b;
    const int qrows = GATEUP ? I : d;
    const uint8_t *qrow = qmat + int64_t(wr_local) * (K / 2) + bchunk * 16;
    const int wr_s = weight_row(tid & 127);
    const uint8_t *smat = GATEUP ? obj + (wr_s >= I ? mbytes : 0u) : obj + 2 * mbytes;
    const int ws_local = GATEUP ? (wr_s >= I ? wr_s - I : wr_s) : wr_s;
    const uint16_t *srow = reinterpret_cast<const uint16_t *>(smat + uint32_t(qrows) * uint32_t(K / 2)) +
                           int64_t(ws_local) * (K / 32);

    u32x4 ra[4], rq;
    uint32_t rs = 0;
    auto load = [&](int k0) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            ra[i] = *reinterpret_cast<const u32x4 *>(abase + (aoff[i] + uint32_t(k0)));
        rq = *reinterpret_cast<const u32x4 *>(qrow + k0 / 2);
        if (tid < 128)
            rs = *reinterpret_cast<const uint32_t *>(srow + k0 / 32);
    };
    auto store = [&](int buf) {
        uint8_t *st = lds8 + buf * STAGE;
        uint16_t *a = reinterpret_cast<uint16_t *>(st);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            *reinterpret_cast<u32x4 *>(a + ((tid >> 3) + 32 * i) * LDA + (tid & 7) * 8) = ra[i];
        uint32_t *q = reinterpret_cast<uint32_t *>(st + A_BYTES + brow_l * LDQ + bchunk * 16);
#pragma unroll
        for (int w = 0; w < 4; ++w)
            q[w] = rq[w];
        if (tid < 128)
            *reinterpret_cast<uint32_t *>(st + A_BYTES + Q_BYTES + (tid & 127) * 4) = rs;
    };

    f32x4 acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
            acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int r16 = lane & 15, g = lane >> 4;
    auto col_of = [&](int nb) -> int {              // tile column block of this wavefront
        if (GATEUP)
            return nb < 2 ? wn * 32 + nb * 16 : 64 + wn * 32 + (nb - 2) * 16;
        return wn * 64 + nb * 16;
    };
    auto compute = [&](int buf) {
        const uint8_t *st = lds8 + buf * STAGE;
        const uint16_t *a = reinterpret_cast<const uint16_t *>(st);
        const uint8_t *q = st + A_BYTES;
        const uint16_t *sc = reinterpret_cast<const uint16_t *>(st + A_BYTES + Q_BYTES);
#pragma unroll
        for (int kb = 0; kb < BK / 32; ++kb) {
            bf16x8 af[4];
#pragma unroll
            for (int mb = 0; mb < 4; ++mb)
                af[mb] = as_bf16x8(*reinterpret_cast<const u32x4 *>(a + (wm * 64 + mb * 16 + r16) * LDA + kb * 32 + g * 8));
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                const int c = col_of(nb) + r16;                    // B fragment: weight row c
                const bf16x8 bq = unpack_q4(*reinterpret_cast<const uint32_t *>(q + c * LDQ + kb * 16 + g * 4));
                const float s = half_to_float(sc[c * 2 + kb]);    // output column of this lane = c
#pragma unroll
                for (int mb = 0; mb < 4; ++mb) {
                    const f32x4 part = mfma16(af[mb], bq, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr)
                        acc[mb][nb][rr] = fmaf(s, part[rr], acc[mb][nb][rr]);
                }
            }
        }
    };

    const int nk = K / BK;
    load(0);
    store(0);
    if (nk > 1)
        load(BK);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        compute(kt & 1);
        if (kt + 1 < nk)
            store((kt + 1) & 1);
        if (kt + 2 < nk)
            load((kt + 2) * BK);
        __syncthreads();
    }

    // lane holds rows 4g + rr of each 16x16 block, column r16
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
            const int row = wm * 64 + mb * 16 + 4 * g + rr;
            if (m0 + row >= it.nrows)
                continue;
            const int64_t orow = int64_t(it.row0) + m0 + row;
            if (GATEUP) {
                uint16_t *act = reinterpret_cast<uint16_t *>(sh ? L.act_s : L.act) + orow * I;
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
                    act[nt * 64 + wn * 32 + nb * 16 + r16] =
                        f32_to_bf16(silu(acc[mb][nb][rr]) * acc[mb][nb + 2][rr]);
            } else {
                uint16_t *y = static_cast<uint16_t *>(sh ? L.ys : L.y) + orow * d;
                const float w = sh ? 1.0f : L.row_weight[orow];
#pragma unroll
                for (int nb = 0; nb < 4; ++nb)
                    y[nt * BN + wn * 64 + nb * 16 + r16] = f32_to_bf16(acc[mb][nb][rr] * w);
            }
        }
}

hipError_t launch_gateup_q4_tile(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    launch_k(tile_q4_kernel<true>, L.n_tiles, q4t::THREADS, q4t::LDS_BYTES, s, L);
    return hipGetLastError();
}

hipError_t launch_down_q4_tile(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    launch_k(tile_q4_kernel<false>, L.n_tiles, q4t::THREADS, q4t::LDS_BYTES, s, L);
    return hipGetLastError();
}

hipError_t init_q4_attributes()
{
    hipError_t e = allow_large_lds(reinterpret_cast<const void *>(&stream_gateup_q4_kernel<16>));
    if (e == hipSuccess)
        e = allow_large_lds(reinterpret_cast<const void *>(&stream_gateup_q4_kernel<8>));
    if (e == hipSuccess)
        e = allow_large_lds(reinterpret_cast<const void *>(&stream_gateup_q4_kernel<4>));
    if (e == hipSuccess)
        e = allow_large_lds(reinterpret_cast<const void *>(&stream_gateup_q4_kernel<2>));
    if (e == hipSuccess)
        e = allow_large_lds(reinterpret_cast<const void *>(&stream_down_q4_kernel<16>));
    if (e == hipSuccess)
        e = allow_large_lds(reinterpret_cast<const void *>(&stream_down_q4_kernel<8>));
    if (e == hipSuccess)
        e = allow_large_lds(reinterpret_cast<const void *>(&stream_down_q4_kernel<4>));
    if (e == hipSuccess)
        e = allow_large_lds(reinterpret_cast<const void *>(&tile_q4_kernel<true>));
    if (e == hipSuccess)
        e = allow_large_lds(reinterpret_cast<const void *>(&tile_q4_kernel<false>));
    return e;
}

}  // namespace msi
