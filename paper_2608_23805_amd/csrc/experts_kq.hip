// experts_kq.hip -- expert projections of the quantized-expert mix (the
// paper's 4.5 / 6.5625 bits-per-weight representation, "Implementation" and
// "Output-Exact Execution Beyond the Full-Residency Envelope"), gfx950.
//
// Formats (per matrix [rows, cols], 256-element super-blocks along a row):
//  * k4 (Wg, Wu): nibbles [rows, cols/2] (unsigned 0..15, element 2j in the
//    low nibble of byte j), then a 16-byte header per (row, super-block):
//    fp16 d, fp16 dmin, eight 6-bit sub-block scales, eight 6-bit sub-block
//    mins (48-bit little-endian fields); value = d sc_j q - dmin m_j for the
//    j-th 32-element sub-block.
//  * k6 (Wd): low nibbles [rows, cols/2], high 2-bit parts [rows, cols/4]
//    (element 4j + t at bits 2t of byte j), int8 scales [rows, cols/16], fp16
//    d [rows, cols/256]; q = low | high << 4 and value = d sc_j (q - 32) for
//    the j-th 16-element sub-block.
//
// The k6 integers q - 32 and the k4 integers 128 + q are exact in bf16, so
// every MFMA partial over a sub-block is a sum of exact products in fp32; the
// sub-block's scale is then applied in fp32.  The k4 min term takes the
// tokens' sums over the sub-block (one more MFMA, against a fragment of ones)
// times dmin m_j + 128 d sc_j, which also removes the 128 of the operands.  A
// 16x16x32 MFMA spans one k4 sub-block, or two k6 sub-blocks: those are split
// by zeroing the weight lanes of the other half (lanes 0..31 carry elements
// 0..15 of the 32).
//
//  * stream path (<= 16 tokens per expert): tokens as the A operand and
//    weights as the B operand, both read straight from memory, so each output
//    lane holds one weight row (and that row's coefficients) for four tokens;
//  * tile path: 128 tokens x 128 weight rows per workgroup, packed weights,
//    headers and scales staged in LDS (the coefficients decoded once per
//    stage into fp32), unpacked while the fragments are built.
#include "common.h"
#include "kernels.h"

namespace msi {

namespace {

constexpr uint32_t BF16_ONE2 = 0x3F803F80u;        // two bf16 1.0

__device__ __forceinline__ float h2f(uint16_t h) { return float(__builtin_bit_cast(_Float16, h)); }

// 8 unsigned nibbles (element e at bits 4e) -> 8 bf16 values 128 + q, exact
// (bf16 numbers in [128, 256) are the integers: bits 0x4300 | q).  A partial
// sum over these is the partial over q plus 128 times the sum of the other
// operand, which the callers subtract with the sub-block's min term.
__device__ __forceinline__ bf16x8 unpack_u4_128(uint32_t q)
{
    const uint32_t ev = q & 0x0F0F0F0Fu;               // elements 0, 2, 4, 6 in bytes 0..3
    const uint32_t od = (q >> 4) & 0x0F0F0F0Fu;        // elements 1, 3, 5, 7
    u32x4 r;
    r[0] = (ev & 0xFFu) | ((od & 0xFFu) << 16) | 0x43004300u;
    r[1] = ((ev >> 8) & 0xFFu) | ((od << 8) & 0xFF0000u) | 0x43004300u;
    r[2] = ((ev >> 16) & 0xFFu) | (od & 0xFF0000u) | 0x43004300u;
    r[3] = (ev >> 24) | ((od >> 8) & 0xFF0000u) | 0x43004300u;
    return __builtin_bit_cast(bf16x8, r);
}

// 8 k6 elements: low nibbles (element e at bits 4e of lo) and 2-bit high
// parts (element e at bits 2e of hi) -> 8 exact bf16 values q - 32.  The
// codes are assembled one per byte (even and odd elements in two words), each
// byte converted to binary32 by the byte-to-float instructions and 32
// subtracted: q - 32 exactly, and that integer (at most 6 significant bits) is
// exact in the top half of its binary32.
__device__ __forceinline__ bf16x8 unpack_k6(uint32_t lo, uint32_t hi)
{
    // spread the four 4-bit groups of hi (two elements each) to bytes 0..3
    uint32_t t = (hi | (hi << 8)) & 0x00FF00FFu;
    t = (t | (t << 4)) & 0x0F0F0F0Fu;
    const uint32_t ev = (lo & 0x0F0F0F0Fu) | ((t & 0x03030303u) << 4);          // elements 0, 2, 4, 6
    const uint32_t od = ((lo >> 4) & 0x0F0F0F0Fu) | ((t & 0x0C0C0C0Cu) << 2);   // elements 1, 3, 5, 7
    u32x4 r;
    float c32 = 32.0f;
    asm("" : "+v"(c32));        // (kept a register: the byte conversions then stay v_cvt_f32_ubyte)
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        const float fe = float((ev >> (8 * h)) & 0xFFu) - c32;
        const float fo = float((od >> (8 * h)) & 0xFFu) - c32;
        r[h] = __builtin_amdgcn_perm(__float_as_uint(fo), __float_as_uint(fe), 0x07060302u);
    }
    return __builtin_bit_cast(bf16x8, r);
}

// k4 header (16 bytes as four words): sub-block j's scale d sc_j and offset dmin m_j
__device__ __forceinline__ void k4_coef(const u32x4 &h, int j, float &a, float &b)
{
    const uint64_t sc = uint64_t(h[1]) | (uint64_t(h[2] & 0xFFFFu) << 32);
    const uint64_t mn = uint64_t(h[2] >> 16) | (uint64_t(h[3]) << 16);
    a = h2f(uint16_t(h[0])) * float(uint32_t(sc >> (6 * j)) & 63u);
    b = h2f(uint16_t(h[0] >> 16)) * float(uint32_t(mn >> (6 * j)) & 63u);
}

// the same with the min coefficient taken against partials over 128 + q:
// a (P + 128 S) - (b + 128 a) S = a P - b S
__device__ __forceinline__ void k4_coef128(const u32x4 &h, int j, float &a, float &b)
{
    k4_coef(h, j, a, b);
    b = fmaf(128.0f, a, b);
}

__host__ __device__ __forceinline__ uint32_t k4_bytes(uint32_t rows, uint32_t cols)
{
    return rows * (cols / 2) + rows * (cols / 256) * 16u;
}

// k6 planes of a [rows, cols] matrix at m: low nibbles, high parts, scales, d
struct K6Planes {
    const uint8_t *ql, *qh;
    const int8_t *sc;
    const uint16_t *d;
};
__device__ __forceinline__ K6Planes k6_planes(const uint8_t *m, uint32_t rows, uint32_t cols)
{
    K6Planes p;
    p.ql = m;
    p.qh = m + rows * (cols / 2);
    p.sc = reinterpret_cast<const int8_t *>(p.qh + rows * (cols / 4));
    p.d = reinterpret_cast<const uint16_t *>(reinterpret_cast<const uint8_t *>(p.sc) + rows * (cols / 16));
    return p;
}

// Tile of a launch and its item (device-built decode list, device-built
// prefill list, or host list), as the 4-bit kernels find theirs.
__device__ __forceinline__ bool kq_tile(const ExpertLaunch &L, int per_item, int &t, WorkItem &it)
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

}  // namespace

// ============================================================== stream path

namespace kqs {
constexpr int WAVES = 4, ROWS = 16;
}

int tiles_gateup_kq_stream(int nrows, int d, int I)
{
    (void)nrows;
    (void)d;
    return I / kqs::ROWS;
}

int tiles_down_kq_stream(int nrows, int d, int I)
{
    (void)nrows;
    (void)I;
    return d / (kqs::WAVES * kqs::ROWS);
}

// Gate/up, k4 stream path: a workgroup owns 16 rows of Wg and of Wu; its four
// wavefronts take the quarters of d and add their partial sums in wavefront
// order.  Tokens are the A operand and weights the B operand, so lane
// (r = lane % 16, g = lane / 16) holds elements 8g .. 8g + 7 of each block of
// token r and of weight row i0 + r, and its outputs are tokens 4g .. 4g + 3
// of weight row i0 + r: one row's sub-block coefficients per lane.  Token
// fragments come straight from global memory (the few rows of a decode step
// stay in cache; lanes past the item's rows repeat its last row and are not
// stored); weights go through WaveRows.  Blocks go in chunks of CH (CH
// divides 8: at most one super-block), each chunk's loads issued before its
// first MFMA.  The four lanes of a weight row share the decoding of its
// sub-block coefficients: lane (r, g) decodes those of blocks g, g + 4 of
// the chunk into the wavefront's LDS table, and every lane reads the block's
// four coefficients back.  Chunks of 8 and the table keep the kernel at 80
// registers, three workgroups per CU.
template <int CH>
__global__ void __launch_bounds__(256, 3) stream_gateup_kq_kernel(ExpertLaunch L)
{
    using Rows = WaveRows<16 * CH>;
    __shared__ __attribute__((aligned(16))) uint8_t wst[kqs::WAVES][2][16 * Rows::RS];
    // the coefficient table of the chunks, then the cross-wavefront sums (after a barrier)
    __shared__ f32x4 cbuf[kqs::WAVES * CH * 16 > 3 * 2 * 64 ? kqs::WAVES * CH * 16 : 3 * 2 * 64];
    f32x4 (*coef)[CH][16] = reinterpret_cast<f32x4 (*)[CH][16]>(cbuf);   // {a_g, b_g, a_u, b_u} of block u, row r
    f32x4 (*red)[2][64] = reinterpret_cast<f32x4 (*)[2][64]>(cbuf);
    int t;
    WorkItem it;
    if (!kq_tile(L, L.I / kqs::ROWS, t, it) || it.nrows == 0 ||
        !slot_current(it, L.gen_dev, L.status))      // nrows 0: unpublished expert, no work
        return;
    static_assert(CH <= 8, "a chunk stays within one super-block");
    const int n = it.nrows, d = L.d, I = L.I, nsb = d / 256, nq = d / 32 / kqs::WAVES;
    const bool sh = it.slot < 0;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int i0 = (t - it.tile0) * kqs::ROWS;
    const int r = lane & 15, g = lane >> 4;
    const int bq = wave * nq;                          // this wavefront's first block
    const uint8_t *base = sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const uint32_t mb = k4_bytes(I, d);
    const uint8_t *qrows[2];
    const u32x4 *hp[2];
#pragma unroll
    for (int m = 0; m < 2; ++m) {
        const uint8_t *mat = base + m * mb;
        qrows[m] = mat + int64_t(i0) * (d / 2) + 16 * bq;
        hp[m] = reinterpret_cast<const u32x4 *>(mat + uint32_t(I) * uint32_t(d / 2)) + int64_t(i0 + r) * nsb;
    }
    const int tr = min(r, n - 1);
    const int64_t xrow = sh ? int64_t(it.row0 + tr) : int64_t(L.perm[it.row0 + tr]);
    const uint16_t *xp = reinterpret_cast<const uint16_t *>(L.x) + xrow * d + 8 * g + 32 * bq;
    Rows wr[2];
    u32x4 xv[CH], hd[2];                               // token fragments; the chunk's super-block headers
    auto issue = [&](int c0) {
#pragma unroll
        for (int m = 0; m < 2; ++m)
            wr[m].load(qrows[m] + 16 * c0, d / 2, lane);
#pragma unroll
        for (int u = 0; u < CH; ++u)
            xv[u] = *reinterpret_cast<const u32x4 *>(xp + 32 * (c0 + u));
#pragma unroll
        for (int m = 0; m < 2; ++m)
            hd[m] = hp[m][(bq + c0) >> 3];
    };
    const bf16x8 ones = __builtin_bit_cast(bf16x8, u32x4{BF16_ONE2, BF16_ONE2, BF16_ONE2, BF16_ONE2});
    f32x4 ag = {0.f, 0.f, 0.f, 0.f}, au = {0.f, 0.f, 0.f, 0.f};
    for (int c0 = 0; c0 < nq; c0 += CH) {
        issue(c0);
        wr[0].store(wst[wave][0], lane);
        wr[1].store(wst[wave][1], lane);
        const uint8_t *q0 = wst[wave][0] + r * Rows::RS + 4 * g, *q1 = wst[wave][1] + r * Rows::RS + 4 * g;
#pragma unroll
        for (int u0 = 0; u0 < CH; u0 += 4) {
            const int u = u0 + g;
            if (u < CH) {
                const int j = (bq + c0 + u) & 7;       // sub-block within the super-block
                float a_g, b_g, a_u, b_u;
                k4_coef128(hd[0], j, a_g, b_g);
                k4_coef128(hd[1], j, a_u, b_u);
                coef[wave][u][r] = f32x4{a_g, b_g, a_u, b_u};
            }
        }
#pragma unroll
        for (int u = 0; u < CH; ++u) {
            const bf16x8 xb = as_bf16x8(xv[u]);
            const f32x4 pg = mfma16(xb, unpack_u4_128(*reinterpret_cast<const uint32_t *>(q0 + 16 * u)),
                                    f32x4{0.f, 0.f, 0.f, 0.f});
            const f32x4 pu = mfma16(xb, unpack_u4_128(*reinterpret_cast<const uint32_t *>(q1 + 16 * u)),
                                    f32x4{0.f, 0.f, 0.f, 0.f});
            const f32x4 sx = mfma16(xb, ones, f32x4{0.f, 0.f, 0.f, 0.f});    // the tokens' sums over the block
            const f32x4 cf = coef[wave][u][r];
            const float a_g = cf[0], b_g = cf[1], a_u = cf[2], b_u = cf[3];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                ag[i] = fmaf(a_g, pg[i], ag[i]);
                ag[i] = fmaf(-b_g, sx[i], ag[i]);
                au[i] = fmaf(a_u, pu[i], au[i]);
                au[i] = fmaf(-b_u, sx[i], au[i]);
            }
        }
    }
    // quarters of d added in wavefront order
    __syncthreads();                                   // (the table's last reads are done)
    if (wave > 0) {
        red[wave - 1][0][lane] = ag;
        red[wave - 1][1][lane] = au;
    }
    __syncthreads();
    if (wave != 0)
        return;
    uint16_t *act = reinterpret_cast<uint16_t *>(sh ? L.act_s : L.act) + int64_t(it.row0) * I + i0 + r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float gv = ((ag[i] + red[0][0][lane][i]) + red[1][0][lane][i]) + red[2][0][lane][i];
        const float uv = ((au[i] + red[0][1][lane][i]) + red[1][1][lane][i]) + red[2][1][lane][i];
        if (4 * g + i < n)
            act[int64_t(4 * g + i) * I] = f32_to_bf16(silu(gv) * uv);
    }
}

// Down, k6 stream path: a workgroup owns 64 output columns (16 per wavefront)
// over all of I, in groups of G super-blocks whose low nibbles and high parts
// (through WaveRows), act fragments and this lane's sub-block and
// super-block scales are issued together.  Act rows are the A operand, read
// straight from global memory (lanes past the item's rows repeat its last
// row), and weights the B operand (lane: token r / weight row c0 + r,
// elements 8g .. 8g + 7 of each block; outputs: tokens 4g .. 4g + 3 of column
// c0 + r).  Each 32-element block holds two 16-element sub-blocks: two MFMAs
// with the other half's weight lanes zeroed (lanes with g < 2 carry elements
// 0 .. 15), each partial scaled by its own d * sc.
template <int G>
__global__ void __launch_bounds__(256, 2) stream_down_kq_kernel(ExpertLaunch L)
{
    constexpr int NB = 8 * G;                          // 32-element blocks per group
    using QL = WaveRows<16 * NB>;                      // 16 bytes of low nibbles per block
    using QH = WaveRows<8 * NB>;                       // 8 bytes of high parts per block
    __shared__ __attribute__((aligned(16))) uint8_t lst[kqs::WAVES][16 * QL::RS];
    __shared__ __attribute__((aligned(16))) uint8_t hst[kqs::WAVES][16 * QH::RS];
    int t;
    WorkItem it;
    if (!kq_tile(L, L.d / (kqs::WAVES * kqs::ROWS), t, it) || it.nrows == 0 ||
        !slot_current(it, L.gen_dev, L.status))      // nrows 0: unpublished expert, no work
        return;
    const int n = it.nrows, d = L.d, I = L.I, nsb = I / 256;
    const bool sh = it.slot < 0;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int c0 = ((t - it.tile0) * kqs::WAVES + wave) * kqs::ROWS;
    const int r = lane & 15, g = lane >> 4;
    const uint8_t *base = sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const K6Planes P = k6_planes(base + 2 * k4_bytes(I, d), d, I);
    const int64_t row = c0 + r;                        // this lane's weight row (output column)
    const uint8_t *qlrows = P.ql + int64_t(c0) * (I / 2);
    const uint8_t *qhrows = P.qh + int64_t(c0) * (I / 4);
    const u32x4 *scp = reinterpret_cast<const u32x4 *>(P.sc + row * (I / 16));
    const uint16_t *ap = reinterpret_cast<const uint16_t *>(sh ? L.act_s : L.act) +
                         int64_t(it.row0 + min(r, n - 1)) * I + 8 * g;
    QL wl;
    QH wh;
    u32x4 av[NB], sc[G];
    float dd[G];
    auto issue = [&](int s0) {
        wl.load(qlrows + 128 * s0, I / 2, lane);
        wh.load(qhrows + 64 * s0, I / 4, lane);
#pragma unroll
        for (int u = 0; u < NB; ++u)
            av[u] = *reinterpret_cast<const u32x4 *>(ap + 32 * (8 * s0 + u));
#pragma unroll
        for (int s = 0; s < G; ++s) {
            sc[s] = scp[s0 + s];
            dd[s] = h2f(P.d[row * nsb + s0 + s]);
        }
    };
    const bool first_half = g < 2;
    const bf16x8 zero = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < nsb; s0 += G) {
        issue(s0);
        wl.store(lst[wave], lane);
        wh.store(hst[wave], lane);
        const uint8_t *lq = lst[wave] + r * QL::RS + 4 * g, *hq = hst[wave] + r * QH::RS + 2 * g;
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            const bf16x8 ab = as_bf16x8(av[u]);
            const bf16x8 w = unpack_k6(*reinterpret_cast<const uint32_t *>(lq + 16 * u),
                                       *reinterpret_cast<const uint16_t *>(hq + 8 * u));
            const f32x4 p0 = mfma16(ab, first_half ? w : zero, f32x4{0.f, 0.f, 0.f, 0.f});
            const f32x4 p1 = mfma16(ab, first_half ? zero : w, f32x4{0.f, 0.f, 0.f, 0.f});
            const int s = u >> 3, lb = u & 7;          // super-block of the group, block within it
            // scales 2 lb and 2 lb + 1 of the super-block: bytes 2 (lb & 1) and + 1 of word lb / 2
            const uint32_t word = sc[s][lb >> 1] >> (16 * (lb & 1));
            const float s0v = dd[s] * float(int(int8_t(word & 0xFFu)));
            const float s1v = dd[s] * float(int(int8_t((word >> 8) & 0xFFu)));
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                acc[i] = fmaf(s0v, p0[i], acc[i]);
                acc[i] = fmaf(s1v, p1[i], acc[i]);
            }
        }
    }
    uint16_t *y = static_cast<uint16_t *>(sh ? L.ys : L.y) + int64_t(it.row0) * d + c0 + r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int tok = 4 * g + i;
        if (tok < n) {
            const float w = sh ? 1.0f : L.row_weight[it.row0 + tok];
            y[int64_t(tok) * d] = f32_to_bf16(acc[i] * w);
        }
    }
}

hipError_t launch_gateup_kq_stream(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    if (L.d % 256 != 0)
        return hipErrorInvalidValue;
    // chunk: 8, 4 or 2 blocks, dividing a quarter of d's blocks (d / 128)
    const int nq = L.d / 128;
    if (nq % 8 == 0)
        launch_k(stream_gateup_kq_kernel<8>, L.n_tiles, 256, 0, s, L);
    else if (nq % 4 == 0)
        launch_k(stream_gateup_kq_kernel<4>, L.n_tiles, 256, 0, s, L);
    else
        launch_k(stream_gateup_kq_kernel<2>, L.n_tiles, 256, 0, s, L);
    return hipGetLastError();
}

hipError_t launch_down_kq_stream(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    if (L.I % 256 != 0 || L.d % 64 != 0)
        return hipErrorInvalidValue;
    if ((L.I / 256) % 2 == 0)
        launch_k(stream_down_kq_kernel<2>, L.n_tiles, 256, 0, s, L);
    else
        launch_k(stream_down_kq_kernel<1>, L.n_tiles, 256, 0, s, L);
    return hipGetLastError();
}

// ============================================================== tile path

namespace kqt {
constexpr int BM = 128, BN = 128, BK = 64, THREADS = 512;
constexpr int LDA = BK + 8;                 // bf16 elements per staged A row
constexpr int LDQ = BK / 2 + 4;             // bytes per staged low-nibble row (36: conflict-spread)
constexpr int LDH = BK / 4 + 4;             // bytes per staged high-part row (k6)
constexpr int A_BYTES = BM * LDA * 2;
constexpr int Q_BYTES = BN * LDQ;
constexpr int H_BYTES = BN * LDH;
constexpr int S_BYTES = BN * 16;            // four fp32 coefficients per weight row
constexpr int STAGE = A_BYTES + Q_BYTES + H_BYTES + S_BYTES;
constexpr size_t LDS_BYTES = size_t(2) * STAGE;
}  // namespace kqt

int tiles_gateup_kq_tile(int nrows, int d, int I)
{
    (void)d;
    return ((nrows + kqt::BM - 1) / kqt::BM) * (I / 64);
}

int tiles_down_kq_tile(int nrows, int d, int I)
{
    (void)I;
    return ((nrows + kqt::BM - 1) / kqt::BM) * (d / kqt::BN);
}

TileGeom geom_gateup_kq_tile(int d, int I)
{
    (void)d;
    return TileGeom{kqt::BM, I / 64};
}

TileGeom geom_down_kq_tile(int d, int I)
{
    (void)I;
    return TileGeom{kqt::BM, d / kqt::BN};
}

// 128 tokens x 128 weight rows per workgroup of eight wavefronts, K in
// stages of 64 (two 32-element blocks; a stage never crosses a 256-element
// super-block).  Wavefront (wm, wn), wm in 0..1, wn in 0..3, owns token rows
// wm*64 .. wm*64+63 and two 16-column blocks: for GATEUP the gate rows
// nt*64 + wn*16 .. (tile columns wn*16..) and the matching up rows (tile
// columns 64 + wn*16..), so SiLU * up forms in registers; for down the tile
// columns wn*32 .. wn*32+31.  Per stage each weight row's coefficients are
// decoded once into LDS as fp32: gate/up {a0, a1, b0', b1'} (scale d sc_j and
// folded min dmin m_j + 128 d sc_j of the stage's two blocks), down
// {s0 .. s3} (d sc_j of its four 16-element sub-blocks).  The k4 min
// multiplies the tokens' sums over the block, from one MFMA against ones per
// token block; the k6 sub-blocks are two MFMAs with the other half's weight
// lanes zeroed.
template <bool GATEUP>
__global__ void __launch_bounds__(kqt::THREADS, 1) tile_kq_kernel(ExpertLaunch L)
{
    using namespace kqt;
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
    const int wm = wave >> 2, wn = wave & 3;

    const uint16_t *abase = reinterpret_cast<const uint16_t *>(GATEUP ? L.x : (sh ? L.act_s : L.act));
    const int32_t *perm = (GATEUP && !sh) ? L.perm : nullptr;
    const uint8_t *obj = sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const uint32_t mbytes = k4_bytes(I, d);

    // A: 128 rows x 64 bf16 per stage = 8 chunks of 16 B per row; 2 per thread
    uint32_t aoff[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int r = (tid >> 3) + 64 * i;
        int64_t src = 0;
        if (m0 + r < it.nrows)
            src = perm ? int64_t(perm[it.row0 + m0 + r]) : int64_t(it.row0 + m0 + r);
        aoff[i] = uint32_t(src * K) + (tid & 7) * 8;
    }
    auto weight_row = [&](int c) -> int {          // tile column -> row of its matrix
        if (GATEUP)
            return nt * 64 + (c & 63);
        return nt * BN + c;
    };
    auto matrix_of = [&](int c) -> const uint8_t * {
        if (GATEUP)
            return obj + (c < 64 ? 0u : mbytes);
        return obj + 2 * mbytes;
    };
    // threads 0..255: low nibbles, 128 rows x 32 B per stage, 2 chunks of 16 B per row;
    // threads 256..383: tile column tid - 256's header (gate/up) or high parts (down);
    // threads 384..511: tile column tid - 384's sub-block scales (down)
    const int role = tid >> 7;                      // 0, 1: nibbles; 2: header / high parts; 3: scales
    const int brow_l = (tid & 255) >> 1, bchunk = tid & 1;
    const uint8_t *qrow = matrix_of(brow_l) + int64_t(weight_row(brow_l)) * (K / 2) + bchunk * 16;
    const int cc = tid & 127;
    const uint8_t *cmat = matrix_of(cc);
    const int64_t crow = weight_row(cc);
    const int rows_m = GATEUP ? I : d;
    const u32x4 *hdr = reinterpret_cast<const u32x4 *>(cmat + uint32_t(rows_m) * uint32_t(K / 2)) + crow * (K / 256);
    const K6Planes P = k6_planes(cmat, rows_m, K);

    // the 16-byte word of roles 0..2 (nibbles, header or high parts) goes through one register
    // quadruple, loaded from a per-role address
    u32x4 ra[2], rw;
    uint32_t rsc = 0;
    uint16_t rd = 0;
    auto load = [&](int k0) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
            ra[i] = *reinterpret_cast<const u32x4 *>(abase + (aoff[i] + uint32_t(k0)));
        if (role < 3) {
            const u32x4 *src = role < 2 ? reinterpret_cast<const u32x4 *>(qrow + k0 / 2)
                               : GATEUP ? hdr + k0 / 256
                                        : reinterpret_cast<const u32x4 *>(P.qh + crow * (K / 4) + k0 / 4);
            rw = *src;
        } else if (!GATEUP) {
            rsc = *reinterpret_cast<const uint32_t *>(P.sc + crow * (K / 16) + k0 / 16);
            rd = P.d[crow * (K / 256) + k0 / 256];
        }
    };
    auto store = [&](int buf, int k0) {
        uint8_t *st = lds8 + buf * STAGE;
        uint16_t *a = reinterpret_cast<uint16_t *>(st);
#pragma unroll
        for (int i = 0; i < 2; ++i)
            *reinterpret_cast<u32x4 *>(a + ((tid >> 3) + 64 * i) * LDA + (tid & 7) * 8) = ra[i];
        float *cfp = reinterpret_cast<float *>(st + A_BYTES + Q_BYTES + H_BYTES + cc * 16);
        if (role < 2) {
            uint32_t *q = reinterpret_cast<uint32_t *>(st + A_BYTES + brow_l * LDQ + bchunk * 16);
#pragma unroll
            for (int w = 0; w < 4; ++w)
                q[w] = rw[w];
        } else if (role == 2) {
            if (GATEUP) {
                const int j0 = (k0 & 255) >> 5;
                float a0, b0, a1, b1;
                k4_coef128(rw, j0, a0, b0);
                k4_coef128(rw, j0 + 1, a1, b1);
                *reinterpret_cast<f32x4 *>(cfp) = f32x4{a0, a1, b0, b1};
            } else {
                uint32_t *h = reinterpret_cast<uint32_t *>(st + A_BYTES + Q_BYTES + cc * LDH);
#pragma unroll
                for (int w = 0; w < 4; ++w)
                    h[w] = rw[w];
            }
        } else if (!GATEUP) {
            const float dv = h2f(rd);
            f32x4 cf;
#pragma unroll
            for (int k = 0; k < 4; ++k)
                cf[k] = dv * float(int(int8_t((rsc >> (8 * k)) & 0xFFu)));
            *reinterpret_cast<f32x4 *>(cfp) = cf;
        }
    };

    f32x4 acc[4][2];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
            acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int r16 = lane & 15, g = lane >> 4;
    auto col_of = [&](int nb) -> int {              // tile column block of this wavefront
        if (GATEUP)
            return nb * 64 + wn * 16;
        return wn * 32 + nb * 16;
    };
    const bf16x8 ones = __builtin_bit_cast(bf16x8, u32x4{BF16_ONE2, BF16_ONE2, BF16_ONE2, BF16_ONE2});
    const bf16x8 zero = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    const bool first_half = g < 2;                  // B lanes of elements 0 .. 15 of a block
    auto compute = [&](int buf) {
        const uint8_t *st = lds8 + buf * STAGE;
        const uint16_t *a = reinterpret_cast<const uint16_t *>(st);
        const uint8_t *q = st + A_BYTES;
        const uint8_t *h = st + A_BYTES + Q_BYTES;
        const float *cf = reinterpret_cast<const float *>(st + A_BYTES + Q_BYTES + H_BYTES);
#pragma unroll
        for (int kb = 0; kb < BK / 32; ++kb) {
            bf16x8 af[4];
#pragma unroll
            for (int mb = 0; mb < 4; ++mb)
                af[mb] = as_bf16x8(*reinterpret_cast<const u32x4 *>(a + (wm * 64 + mb * 16 + r16) * LDA + kb * 32 + g * 8));
            if (GATEUP) {
                f32x4 sx[4];                        // tokens' sums over the block
#pragma unroll
                for (int mb = 0; mb < 4; ++mb)
                    sx[mb] = mfma16(af[mb], ones, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
                for (int nb = 0; nb < 2; ++nb) {
                    const int c = col_of(nb) + r16;                // B fragment: weight row c
                    const bf16x8 bq = unpack_u4_128(*reinterpret_cast<const uint32_t *>(q + c * LDQ + kb * 16 + g * 4));
                    const float sa = cf[c * 4 + kb], sb = cf[c * 4 + 2 + kb];   // output column = c
#pragma unroll
                    for (int mb = 0; mb < 4; ++mb) {
                        const f32x4 part = mfma16(af[mb], bq, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
                        for (int rr = 0; rr < 4; ++rr) {
                            acc[mb][nb][rr] = fmaf(sa, part[rr], acc[mb][nb][rr]);
                            acc[mb][nb][rr] = fmaf(-sb, sx[mb][rr], acc[mb][nb][rr]);
                        }
                    }
                }
            } else {
#pragma unroll
                for (int nb = 0; nb < 2; ++nb) {
                    const int c = col_of(nb) + r16;
                    const bf16x8 w = unpack_k6(*reinterpret_cast<const uint32_t *>(q + c * LDQ + kb * 16 + g * 4),
                                               *reinterpret_cast<const uint16_t *>(h + c * LDH + kb * 8 + g * 2));
                    const bf16x8 w0 = first_half ? w : zero, w1 = first_half ? zero : w;
                    const float s0 = cf[c * 4 + 2 * kb], s1 = cf[c * 4 + 2 * kb + 1];
#pragma unroll
                    for (int mb = 0; mb < 4; ++mb) {
                        const f32x4 p0 = mfma16(af[mb], w0, f32x4{0.f, 0.f, 0.f, 0.f});
                        const f32x4 p1 = mfma16(af[mb], w1, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
                        for (int rr = 0; rr < 4; ++rr) {
                            acc[mb][nb][rr] = fmaf(s0, p0[rr], acc[mb][nb][rr]);
                            acc[mb][nb][rr] = fmaf(s1, p1[rr], acc[mb][nb][rr]);
                        }
                    }
                }
            }
        }
    };

    const int nk = K / BK;
    load(0);
    store(0, 0);
    if (nk > 1)
        load(BK);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        compute(kt & 1);
        if (kt + 1 < nk)
            store((kt + 1) & 1, (kt + 1) * BK);
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
                act[nt * 64 + wn * 16 + r16] = f32_to_bf16(silu(acc[mb][0][rr]) * acc[mb][1][rr]);
            } else {
                uint16_t *y = static_cast<uint16_t *>(sh ? L.ys : L.y) + orow * d;
                const float w = sh ? 1.0f : L.row_weight[orow];
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
                    y[nt * BN + wn * 32 + nb * 16 + r16] = f32_to_bf16(acc[mb][nb][rr] * w);
            }
        }
}

hipError_t launch_gateup_kq_tile(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    if (L.d % 256 != 0 || L.I % 64 != 0)
        return hipErrorInvalidValue;
    launch_k(tile_kq_kernel<true>, L.n_tiles, kqt::THREADS, kqt::LDS_BYTES, s, L);
    return hipGetLastError();
}

hipError_t launch_down_kq_tile(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    if (L.I % 256 != 0 || L.d % kqt::BN != 0)
        return hipErrorInvalidValue;
    launch_k(tile_kq_kernel<false>, L.n_tiles, kqt::THREADS, kqt::LDS_BYTES, s, L);
    return hipGetLastError();
}

hipError_t init_kq_attributes()
{
    const void *ks[] = {reinterpret_cast<const void *>(&tile_kq_kernel<true>),
                        reinterpret_cast<const void *>(&tile_kq_kernel<false>)};
    for (const void *k : ks) {
        const hipError_t e = allow_large_lds(k);
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

}  // namespace msi
