// experts_q4.hip -- 4-bit block-quantized expert projections for gfx950.
//
// Storage (per matrix [rows, cols]): nibbles [rows, cols/2] (element 2j in the
// low nibble of byte j, 4-bit two's complement) then fp16 scales
// [rows, cols/32]; value = scale * q.  Every 16x16x32 MFMA spans exactly one
// 32-element scale block, so it returns the block's partial dot product and
// the scale is applied in fp32: acc += scale * partial.
//
//  * stream path (<= 16 tokens per expert): tokens as the A operand and
//    weights as the B operand, tokens read straight from memory and the
//    nibbles through row-contiguous loads rearranged in LDS (WaveRows); the
//    codes unpacked to exact bf16 q (C = 0).
//  * tile path: 128 tokens x 128 weight rows per workgroup; A rows, packed
//    nibbles and scales copied from memory straight into two LDS stage
//    buffers (three workgroups per CU); the codes enter the MFMA as the exact
//    bf16 136 + q, and the offset leaves through the C input (-136 times the
//    A row's block sum, from one more MFMA per A fragment).
#include "common.h"
#include "kernels.h"

namespace msi {

typedef __attribute__((address_space(3))) void lds_void_t;

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

// 8 nibbles (element e at bits 4e..4e+3, two's complement q) -> 8 exact bf16
// values 136 + q: the bits 0x4300 | u are the bf16 128 + u, u = q + 8 = the
// nibble with its top bit flipped.  Byte permutes place the nibbles (even
// elements from the low halves of the bytes, odd ones from the high halves)
// under the 0x43 bytes: nine operations per 8 values.
__device__ __forceinline__ bf16x8 unpack_q4_136(uint32_t w)
{
    const uint32_t e = (w ^ 0x08080808u) & 0x0F0F0F0Fu;           // u of elements 0, 2, 4, 6
    const uint32_t o = ((w >> 4) ^ 0x08080808u) & 0x0F0F0F0Fu;    // u of elements 1, 3, 5, 7
    const uint32_t lo = __builtin_amdgcn_perm(o, e, 0x05010400u);  // bytes u0 u1 u2 u3
    const uint32_t hi = __builtin_amdgcn_perm(o, e, 0x07030602u);  // bytes u4 u5 u6 u7
    u32x4 r;
    r[0] = __builtin_amdgcn_perm(0x43434343u, lo, 0x04010400u);
    r[1] = __builtin_amdgcn_perm(0x43434343u, lo, 0x04030402u);
    r[2] = __builtin_amdgcn_perm(0x43434343u, hi, 0x04010400u);
    r[3] = __builtin_amdgcn_perm(0x43434343u, hi, 0x04030402u);
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

// CH consecutive fp16 block scales of one row, in one vector load (the
// row's scales start 16-byte aligned and CH divides the blocks of a quarter
// of d, or of I).
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
// Tokens are the A operand and weights the B operand: lane (r = lane % 16,
// g = lane / 16) holds elements 8g .. 8g + 7 of each block of token r and of
// weight row i0 + r, and its outputs are tokens 4g .. 4g + 3 of that weight
// row, so each lane applies one row's block scales.  Token fragments come
// straight from global memory (lanes past the item's rows repeat its last
// row and are not stored); the nibbles go through WaveRows (row-contiguous
// 16-byte loads, rearranged in the wavefront's own LDS region).  Blocks go
// in chunks of CH, each chunk's loads issued before its first MFMA.
template <int CH>
__global__ void __launch_bounds__(256, 2) stream_gateup_q4_kernel(ExpertLaunch L)
{
    using Rows = WaveRows<16 * CH>;
    __shared__ __attribute__((aligned(16))) uint8_t wst[q4s::WAVES][2][16 * Rows::RS];
    __shared__ f32x4 red[3][2][64];
    const int d = L.d, I = L.I, nblk = d / 32, nq = nblk / q4s::WAVES;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int bq = wave * nq;                          // this wavefront's first block
    // One token (a device-built decode list of T = 1): every row is token 0, so the token fragments of the
    // first chunk are requested before the item is known, and the generation is compared after the work
    // (before the stores), so the weights are requested as soon as the slot is known.
    const bool one = L.direct.demand && L.direct.T == 1;
    u32x4 xv[CH];
    if (one) {
#pragma unroll
        for (int u = 0; u < CH; ++u)
            xv[u] = *reinterpret_cast<const u32x4 *>(reinterpret_cast<const uint16_t *>(L.x) + 8 * g + 32 * (bq + u));
    }
    int t;
    WorkItem it;
    if (!q4_tile(L, L.I / q4s::ROWS, t, it) || it.nrows == 0)   // nrows 0: unpublished expert, no work
        return;
    const uint32_t gnow = slot_gen_now(it, L.gen_dev);
    const int n = it.nrows;
    const bool sh = it.slot < 0;
    const int i0 = (t - it.tile0) * q4s::ROWS;
    const uint8_t *base = sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const uint32_t mb = q4_matrix_bytes(I, d);
    const uint8_t *qrows[2];
    const uint16_t *sp[2];
#pragma unroll
    for (int m = 0; m < 2; ++m) {
        const uint8_t *mat = base + m * mb;
        qrows[m] = mat + int64_t(i0) * (d / 2) + 16 * bq;
        sp[m] = reinterpret_cast<const uint16_t *>(mat + int64_t(I) * (d / 2)) + int64_t(i0 + r) * nblk + bq;
    }
    const int tr = min(r, n - 1);
    const int64_t xrow = one ? 0 : sh ? int64_t(it.row0 + tr) : int64_t(L.perm[it.row0 + tr]);
    const uint16_t *xp = reinterpret_cast<const uint16_t *>(L.x) + xrow * d + 8 * g + 32 * bq;
    Rows wr[2];
    uint32_t sc[2][CH / 2];
    auto issue = [&](int c0) {
#pragma unroll
        for (int m = 0; m < 2; ++m)
            wr[m].load(qrows[m] + 16 * c0, d / 2, lane);
        if (!(one && c0 == 0)) {
#pragma unroll
            for (int u = 0; u < CH; ++u)
                xv[u] = *reinterpret_cast<const u32x4 *>(xp + 32 * (c0 + u));
        }
#pragma unroll
        for (int m = 0; m < 2; ++m)
            load_scales<CH>(sc[m], sp[m] + c0);
    };
    f32x4 ag = {0.f, 0.f, 0.f, 0.f}, au = {0.f, 0.f, 0.f, 0.f};
    for (int c0 = 0; c0 < nq; c0 += CH) {
        issue(c0);
        wr[0].store(wst[wave][0], lane);
        wr[1].store(wst[wave][1], lane);
        const uint8_t *q0 = wst[wave][0] + r * Rows::RS + 4 * g, *q1 = wst[wave][1] + r * Rows::RS + 4 * g;
#pragma unroll
        for (int u = 0; u < CH; ++u) {
            const bf16x8 xb = as_bf16x8(xv[u]);
            const f32x4 pg = mfma16(xb, unpack_q4(*reinterpret_cast<const uint32_t *>(q0 + 16 * u)),
                                    f32x4{0.f, 0.f, 0.f, 0.f});
            const f32x4 pu = mfma16(xb, unpack_q4(*reinterpret_cast<const uint32_t *>(q1 + 16 * u)),
                                    f32x4{0.f, 0.f, 0.f, 0.f});
            const float s_g = scale_at(sc[0], u), s_u = scale_at(sc[1], u);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                ag[k] = fmaf(s_g, pg[k], ag[k]);
                au[k] = fmaf(s_u, pu[k], au[k]);
            }
        }
    }
    // quarters of d added in wavefront order
    if (wave > 0) {
        red[wave - 1][0][lane] = ag;
        red[wave - 1][1][lane] = au;
    }
    __syncthreads();
    if (wave != 0 || !slot_gen_ok(it, gnow, L.status))
        return;
    uint16_t *act = reinterpret_cast<uint16_t *>(sh ? L.act_s : L.act) + int64_t(it.row0) * I + i0 + r;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const float gv = ((ag[k] + red[0][0][lane][k]) + red[1][0][lane][k]) + red[2][0][lane][k];
        const float uv = ((au[k] + red[0][1][lane][k]) + red[1][1][lane][k]) + red[2][1][lane][k];
        if (4 * g + k < n)
            act[int64_t(4 * g + k) * I] = f32_to_bf16(silu(gv) * uv);
    }
}

// Down, 4-bit stream path: a workgroup owns 64 output columns (16 per
// wavefront) over all of I, in chunks of CH blocks whose nibbles (through
// WaveRows), act fragments and this lane's block scales are issued together.
// Act rows are the A operand, read straight from global memory (lanes past
// the item's rows repeat its last row), and weights the B operand (outputs:
// tokens 4g .. 4g + 3 of column c0 + r).
template <int CH>
__global__ void __launch_bounds__(256, 2) stream_down_q4_kernel(ExpertLaunch L)
{
    using Rows = WaveRows<16 * CH>;
    __shared__ __attribute__((aligned(16))) uint8_t wst[q4s::WAVES][16 * Rows::RS];
    int t;
    WorkItem it;
    if (!q4_tile(L, L.d / (q4s::WAVES * q4s::ROWS), t, it) || it.nrows == 0)   // nrows 0: unpublished expert
        return;
    // the generation is read here and compared before the stores, and the row weights are read with the
    // first weights, so nothing waits between the item lookup and the weight loads
    const uint32_t gnow = slot_gen_now(it, L.gen_dev);
    const int n = it.nrows, d = L.d, I = L.I, nblk = I / 32;
    const bool sh = it.slot < 0;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int c0 = ((t - it.tile0) * q4s::WAVES + wave) * q4s::ROWS;
    const int r = lane & 15, g = lane >> 4;
    const uint8_t *base = sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const uint8_t *wd = base + 2 * q4_matrix_bytes(I, d);
    const uint8_t *qrows = wd + int64_t(c0) * (I / 2);
    const uint16_t *sp = reinterpret_cast<const uint16_t *>(wd + int64_t(d) * (I / 2)) + int64_t(c0 + r) * nblk;
    const uint16_t *ap = reinterpret_cast<const uint16_t *>(sh ? L.act_s : L.act) +
                         int64_t(it.row0 + min(r, n - 1)) * I + 8 * g;
    Rows wr;
    u32x4 av[CH];
    uint32_t sc[CH / 2];
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    float rw[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
        rw[k] = (sh || 4 * g + k >= n) ? 1.0f : L.row_weight[it.row0 + 4 * g + k];
    for (int b0 = 0; b0 < nblk; b0 += CH) {
        wr.load(qrows + 16 * b0, I / 2, lane);
#pragma unroll
        for (int u = 0; u < CH; ++u)
            av[u] = *reinterpret_cast<const u32x4 *>(ap + 32 * (b0 + u));
        load_scales<CH>(sc, sp + b0);
        wr.store(wst[wave], lane);
        const uint8_t *q = wst[wave] + r * Rows::RS + 4 * g;
#pragma unroll
        for (int u = 0; u < CH; ++u) {
            const f32x4 part = mfma16(as_bf16x8(av[u]), unpack_q4(*reinterpret_cast<const uint32_t *>(q + 16 * u)),
                                      f32x4{0.f, 0.f, 0.f, 0.f});
            const float sv = scale_at(sc, u);
#pragma unroll
            for (int k = 0; k < 4; ++k)
                acc[k] = fmaf(sv, part[k], acc[k]);
        }
    }
    if (!slot_gen_ok(it, gnow, L.status))
        return;
    uint16_t *y = static_cast<uint16_t *>(sh ? L.ys : L.y) + int64_t(it.row0) * d + c0 + r;
#pragma unroll
    for (int k = 0; k < 4; ++k)
        if (4 * g + k < n)
            y[int64_t(4 * g + k) * d] = f32_to_bf16(acc[k] * rw[k]);
}

hipError_t launch_gateup_q4_stream(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    // chunk: the largest of 16, 8, 4, 2 blocks dividing a quarter of d (d % 256 == 0)
    const int nq = L.d / 128;
    if (nq % 16 == 0)
        launch_k(stream_gateup_q4_kernel<16>, L.n_tiles, 256, 0, s, L);
    else if (nq % 8 == 0)
        launch_k(stream_gateup_q4_kernel<8>, L.n_tiles, 256, 0, s, L);
    else if (nq % 4 == 0)
        launch_k(stream_gateup_q4_kernel<4>, L.n_tiles, 256, 0, s, L);
    else
        launch_k(stream_gateup_q4_kernel<2>, L.n_tiles, 256, 0, s, L);
    return hipGetLastError();
}

hipError_t launch_down_q4_stream(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    // chunk: the largest of 16, 8, 4 blocks dividing I / 32 (I % 128 == 0)
    const int nblk = L.I / 32;
    if (nblk % 16 == 0)
        launch_k(stream_down_q4_kernel<16>, L.n_tiles, 256, 0, s, L);
    else if (nblk % 8 == 0)
        launch_k(stream_down_q4_kernel<8>, L.n_tiles, 256, 0, s, L);
    else
        launch_k(stream_down_q4_kernel<4>, L.n_tiles, 256, 0, s, L);
    return hipGetLastError();
}

// ============================================================== tile path

namespace q4t {
constexpr int BM = 128, BN = 128, BK = 64, THREADS = 256, NBUF = 2;
constexpr int A_ROWB = BK * 2;              // bytes of bf16 per staged A row
constexpr int Q_ROWB = BK / 2;              // bytes of codes per staged weight row
constexpr int A_BYTES = BM * A_ROWB;        // 16 KiB
constexpr int Q_BYTES = BN * Q_ROWB;        // 4 KiB
constexpr int S_BYTES = 2 * BN * (BK / 32) * 2;   // the 512 bytes of scales, then a spare 512 for idle copies
constexpr int STAGE = A_BYTES + Q_BYTES + S_BYTES;
constexpr int COPIES = 6;                   // copy instructions per wavefront per stage
constexpr size_t LDS_BYTES = size_t(NBUF) * STAGE;
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
__global__ void __launch_bounds__(q4t::THREADS, 3) tile_q4_kernel(ExpertLaunch L)
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
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // (uniform: copy destinations and resources)
    const int wm = wave >> 1, wn = wave & 1;

    const uint16_t *abase = reinterpret_cast<const uint16_t *>(GATEUP ? L.x : (sh ? L.act_s : L.act));
    const int32_t *perm = (GATEUP && !sh) ? L.perm : nullptr;
    const uint8_t *obj = sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const uint32_t mbytes = q4_matrix_bytes(I, d);

    // Stage copies go from memory straight into two LDS stage buffers (buffer loads with an
    // LDS destination, no register staging).  Per stage and wavefront: four 1 KiB copies of A rows (lane l
    // of copy i brings row 8 (4 i + w) + l / 8 into slot l % 8 of its 128-byte LDS row, the 16-byte chunk
    // (l % 8) ^ aswz(row) of the row's 64 elements), one of weight codes (row 32 w + l / 2, slot l % 2 =
    // chunk (l % 2) ^ bit 3 of the row) and one of scales (4 bytes: row 64 w + l; wavefronts 2 and 3 copy
    // nothing into a spare region, so every wavefront waits on the same counts).  The slot permutations put
    // the 16 rows of each fragment read on distinct banks.
    auto aswz = [](int r) { return (r >> 1) & 7; };
    const __amdgpu_buffer_rsrc_t ar =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(abase), 0, 0x7fffffff, 0x00020000u);
    const __amdgpu_buffer_rsrc_t wr_ = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(obj), 0, 0x7fffffff,
                                                                         0x00020000u);
    const __amdgpu_buffer_rsrc_t sr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(obj), 0,
                                                                        wave < 2 ? 0x7fffffff : 0, 0x00020000u);
    uint32_t aoff[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = 8 * (4 * i + wave) + (lane >> 3);
        int64_t src = 0;
        if (m0 + r < it.nrows)
            src = perm ? int64_t(perm[it.row0 + m0 + r]) : int64_t(it.row0 + m0 + r);
        aoff[i] = uint32_t(src * K) * 2u + uint32_t(16 * ((lane & 7) ^ aswz(r)));
    }
    auto weight_row = [&](int c) -> int {          // tile column -> matrix row
        if (GATEUP)
            return (c < 64 ? 0 : I) + nt * 64 + (c & 63);
        return nt * BN + c;
    };
    // (a tile column's matrix: gate rows, then up rows, for gate/up; the down matrix for down)
    auto row_base = [&](int c) -> uint32_t {
        const int wrw = weight_row(c);
        const uint32_t mat = GATEUP ? (wrw >= I ? mbytes : 0u) : 2u * mbytes;
        return mat + uint32_t(GATEUP ? (wrw >= I ? wrw - I : wrw) : wrw) * uint32_t(K / 2);
    };
    auto scale_base = [&](int c) -> uint32_t {
        const int wrw = weight_row(c);
        const uint32_t mat = GATEUP ? (wrw >= I ? mbytes : 0u) : 2u * mbytes;
        const int rows = GATEUP ? I : d;
        return mat + uint32_t(rows) * uint32_t(K / 2) + uint32_t(GATEUP ? (wrw >= I ? wrw - I : wrw) : wrw) *
                                                            uint32_t(K / 32) * 2u;
    };
    const int qr = 32 * wave + (lane >> 1);
    const uint32_t qoff = row_base(qr) + uint32_t(16 * ((lane & 1) ^ ((qr >> 3) & 1)));
    const uint32_t soff = wave < 2 ? scale_base(64 * wave + lane) : 0u;
    auto issue = [&](int k0, int buf, bool real) {
        uint8_t *st = lds8 + buf * STAGE;
        const __amdgpu_buffer_rsrc_t none = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(obj), 0, 0,
                                                                              0x00020000u);
#if defined(__HIP_DEVICE_COMPILE__)
#pragma unroll
        for (int i = 0; i < 4; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(real ? ar : none, (lds_void_t *)(st + (4 * i + wave) * 1024), 16,
                                                     aoff[i], k0 * 2, 0, 0);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(real ? wr_ : none, (lds_void_t *)(st + A_BYTES + wave * 1024), 16,
                                                 qoff, k0 / 2, 0, 0);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(real ? sr : none, (lds_void_t *)(st + A_BYTES + Q_BYTES + wave * 256),
                                                 4, soff, k0 / 16, 0, 0);
#else
        (void)st, (void)none, (void)k0, (void)real;
#endif
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
    // The codes enter the MFMA as 136 + q; the -136 * (block sum of the A row) that takes the offset back
    // out comes from one more MFMA per A fragment, against a fragment of -136, and is the C input of that
    // fragment's four block partials.
    const bf16x8 neg136 = __builtin_bit_cast(bf16x8, u32x4{0xC308C308u, 0xC308C308u, 0xC308C308u, 0xC308C308u});
    auto compute = [&](int buf) {
        const uint8_t *st = lds8 + buf * STAGE;
        const uint8_t *q = st + A_BYTES;
        const uint16_t *sc = reinterpret_cast<const uint16_t *>(st + A_BYTES + Q_BYTES);
#pragma unroll
        for (int kb = 0; kb < BK / 32; ++kb) {
            uint32_t cw[4];
            uint16_t sr16[4];
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                const int c = col_of(nb) + r16;                    // B fragment: weight row c
                cw[nb] = *reinterpret_cast<const uint32_t *>(q + c * Q_ROWB + 16 * (kb ^ ((c >> 3) & 1)) + 4 * g);
                sr16[nb] = sc[c * 2 + kb];
            }
            bf16x8 af[4];
            f32x4 corr[4];
#pragma unroll
            for (int mb = 0; mb < 4; ++mb) {
                const int r = wm * 64 + mb * 16 + r16;
                af[mb] = as_bf16x8(*reinterpret_cast<const u32x4 *>(st + r * A_ROWB + 16 * ((4 * kb + g) ^ aswz(r))));
                corr[mb] = mfma16(af[mb], neg136, f32x4{0.f, 0.f, 0.f, 0.f});
            }
            bf16x8 bq[4];
#pragma unroll
            for (int nb = 0; nb < 4; ++nb)
                bq[nb] = unpack_q4_136(cw[nb]);
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                const float s = half_to_float(sr16[nb]);          // output column of this lane = c
                f32x4 part[4];
#pragma unroll
                for (int mb = 0; mb < 4; ++mb)
                    part[mb] = mfma16(af[mb], bq[nb], corr[mb]);
#pragma unroll
                for (int mb = 0; mb < 4; ++mb)
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr)
                        acc[mb][nb][rr] = fmaf(s, part[mb][rr], acc[mb][nb][rr]);
            }
        }
    };

    const int nk = K / BK;
    constexpr int AHEAD = NBUF - 1;                            // stages in flight beside the one computed
#pragma unroll
    for (int j = 0; j < AHEAD; ++j)
        issue(j * BK, j, j < nk);
    for (int kt = 0; kt < nk; ++kt) {
        __builtin_amdgcn_s_waitcnt(VMCNT_WAIT(COPIES * (AHEAD - 1)));   // this stage landed
        __builtin_amdgcn_s_barrier();                          // ... for every wavefront; the buffer refilled
        asm volatile("" ::: "memory");                         //     next was last read one stage ago
        issue((kt + AHEAD) * BK, (kt + AHEAD) % NBUF, kt + AHEAD < nk);
        compute(kt % NBUF);
    }

    // Epilogue through LDS (the stage buffers are free once every wavefront has left the K loop): each lane
    // writes its outputs, rows 4g + rr of each 16x16 block in column r16, as bf16 into a [128][OUTW + 8]
    // tile, then every thread stores whole 16-byte pieces of the tile's rows.  The row weights of the
    // lane's 16 rows are read first, all at once.
    constexpr int OUTW = GATEUP ? 64 : BN;         // output columns of the tile
    constexpr int LDO = OUTW + 8;                  // bf16 per LDS output row (16 bytes of padding)
    float rwv[4][4];
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
            const int row = wm * 64 + mb * 16 + 4 * g + rr;
            rwv[mb][rr] = (GATEUP || sh || m0 + row >= it.nrows) ? 1.0f : L.row_weight[int64_t(it.row0) + m0 + row];
        }
    static_assert(size_t(BM) * LDO * 2 <= LDS_BYTES, "output tile fits the stage buffers");
    __builtin_amdgcn_s_waitcnt(VMCNT_WAIT(0));    // the last (idle) stage copies have written LDS too
    __syncthreads();
    uint16_t *ot = reinterpret_cast<uint16_t *>(lds8);
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
            uint16_t *orow_l = ot + (wm * 64 + mb * 16 + 4 * g + rr) * LDO;
            if (GATEUP) {
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
                    orow_l[wn * 32 + nb * 16 + r16] = f32_to_bf16(silu(acc[mb][nb][rr]) * acc[mb][nb + 2][rr]);
            } else {
#pragma unroll
                for (int nb = 0; nb < 4; ++nb)
                    orow_l[wn * 64 + nb * 16 + r16] = f32_to_bf16(acc[mb][nb][rr] * rwv[mb][rr]);
            }
        }
    __syncthreads();
    constexpr int PPR = OUTW / 8;                  // 16-byte pieces per tile row
    uint16_t *obase = GATEUP ? reinterpret_cast<uint16_t *>(sh ? L.act_s : L.act) + nt * 64
                             : static_cast<uint16_t *>(sh ? L.ys : L.y) + nt * BN;
    const int ostride = GATEUP ? I : d;
#pragma unroll
    for (int k = 0; k < BM * PPR / THREADS; ++k) {
        const int pidx = k * THREADS + tid, row = pidx / PPR, pc = pidx % PPR;
        if (m0 + row < it.nrows)
            *reinterpret_cast<u32x4 *>(obase + (int64_t(it.row0) + m0 + row) * ostride + pc * 8) =
                *reinterpret_cast<const u32x4 *>(ot + row * LDO + pc * 8);
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
    hipError_t e = allow_large_lds(reinterpret_cast<const void *>(&tile_q4_kernel<true>));
    if (e == hipSuccess)
        e = allow_large_lds(reinterpret_cast<const void *>(&tile_q4_kernel<false>));
    return e;
}

}  // namespace msi
