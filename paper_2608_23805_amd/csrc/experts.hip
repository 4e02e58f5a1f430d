// experts.hip -- per-expert gate/up (SiLU-gated) and down projections for
// gfx950, three variants chosen per expert from its routed-token count only:
//
//  * tile path (bf16, > STREAM tokens): tiles.hip.
//  * stream path (bf16, <= 16 tokens): weight streaming.  The weights are the
//    MFMA A operand read straight from HBM in the 16x16x32 fragment layout
//    (each wavefront owns 16 weight rows; each weight byte is read once), the
//    expert's tokens (at most 16, zero-padded) are the B operand held in LDS.
//  * f32 path (fp32 layers): FMA dot products in fixed sequential order.
//
// Every workgroup checks the slot generation first and writes nothing on a
// mismatch (fail closed).  Outputs: act[row, I] = silu(x Wg^T) * (x Wu^T) and
// y[row, d] = row_weight * (act Wd^T), rows in permuted order, both rounded
// to bf16 once (fp32 throughout for fp32 layers).
#include "common.h"
#include "kernels.h"

namespace msi {

// ============================================================== stream path

namespace stream {
constexpr int MAXN = 16;        // tokens per expert handled by this path
constexpr int WAVES = 4;
constexpr int ROWS = 16;        // weight rows per wavefront
}  // namespace stream

int tiles_gateup_stream(int nrows, int d, int I)
{
    (void)nrows;
    (void)d;
    return I / stream::ROWS;
}

int tiles_down_stream(int nrows, int d, int I)
{
    (void)nrows;
    (void)I;
    return d / (stream::WAVES * stream::ROWS);
}

// Stream-path prologue, ordered so that the dependent memory round trips
// before the first MFMA are few: the item is found by division (every stream
// item of a launch has the same tile count), the slot generation word is read
// alongside and checked only before the store (a stale slot is read but
// nothing is written), and the first weight batch is issued before the
// kernel waits for anything else.
struct StreamTile {
    WorkItem it;
    int local;          // tile index within the item
    bool valid;
};

__device__ __forceinline__ StreamTile stream_tile(const ExpertLaunch &L, int per_item)
{
    StreamTile st{};
    if (L.direct.demand) {
        int i;
        direct_tile(int(blockIdx.x), per_item, i, st.local);
        if (!direct_item(L.direct, i, per_item, L.status, st.it))
            return st;
        st.valid = st.it.nrows > 0;       // nrows 0: unpublished expert, no work
        return st;
    }
    int n_items, n_tiles;
    const int t = launch_tile(L, n_items, n_tiles);
    const int i = t / per_item;
    if (t < 0 || i >= n_items)
        return st;
    st.it = L.items[i];
    st.local = t - i * per_item;
    st.valid = st.it.nrows > 0;
    return st;
}

// Weight slabs.  A wavefront's 16 weight rows reach registers in whole
// 128-byte lines: one 16-byte load per lane covers 8 rows x 128 bytes (lane l:
// row l / 8, chunk l % 8), two loads cover a slab of 16 rows x 64 columns.
// (Loading in the MFMA fragment layout instead, 16 rows x 64 bytes per load,
// reads every line in two halves and streams about 15% slower.)  The slab is
// then rearranged into fragments through the wavefront's own 2 KiB of LDS,
// chunks XOR-swizzled by row so that both the writes and the fragment reads
// are free of bank conflicts.
namespace slab {
constexpr int BYTES = 16 * 128;

// element offset, from the slab's first row and column, of lane's load h (rows 8h .. 8h + 7)
__device__ __forceinline__ int src(int lane, int h, int ld) { return (8 * h + (lane >> 3)) * ld + (lane & 7) * 8; }

// LDS byte offset of the 16 bytes that load h brought to lane
__device__ __forceinline__ int dst(int lane, int h)
{
    const int r = 8 * h + (lane >> 3);
    return r * 128 + (((lane & 7) ^ ((r >> 1) & 7)) << 4);
}

// LDS byte offset of lane's MFMA fragment (row lane % 16, elements 8 (lane / 16) ..) of K step ks (0, 1)
__device__ __forceinline__ int frag(int lane, int ks)
{
    const int r = lane & 15;
    return r * 128 + (((4 * ks + (lane >> 4)) ^ ((r >> 1) & 7)) << 4);
}
}  // namespace slab

__device__ __forceinline__ void lds_wait()
{
    __builtin_amdgcn_s_waitcnt(0xC07F);          // lgkmcnt(0): this wavefront's LDS accesses done
    __builtin_amdgcn_wave_barrier();
    asm volatile("" ::: "memory");
}

// Gate/up, stream path: a workgroup owns 16 rows of Wg and of Wu; its four
// wavefronts take the four quarters of d (U K steps of 32, U / 2 slabs per
// matrix, per weight batch) and their fp32 partial sums are added in
// wavefront order before SiLU(g) * u.  The weights (A operand) are streamed
// once, in whole lines (weight slabs above); the lanes of token j (B operand)
// read row j of the item straight from x, which stays in the caches (every
// item reads rows of the same few tokens).  Sixteen-row workgroups keep the
// grid many times larger than the number of resident workgroups, so the last
// partial round of the launch is short.
template <int U, int NB>
__global__ void __launch_bounds__(256, 3) stream_gateup_kernel(ExpertLaunch L)
{
    constexpr int SL = U / 2;                     // slabs per matrix per batch
    __shared__ f32x4 red[3][2][64];
    __shared__ __attribute__((aligned(16))) uint8_t tr[stream::WAVES][2 * SL * slab::BYTES];
    const int d = L.d, I = L.I;
    const StreamTile st = stream_tile(L, I / stream::ROWS);
    if (!st.valid)
        return;
    const WorkItem &it = st.it;
    const int n = it.nrows;
    const bool sh = it.slot < 0;
    const uint32_t gnow = slot_gen_now(it, L.gen_dev);

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int i0 = st.local * stream::ROWS;
    const int kq = d / stream::WAVES;             // this wavefront's quarter of d
    const int j = lane & 15, kg = (lane >> 4) * 8;
    const uint8_t *base = sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const uint16_t *w0 = reinterpret_cast<const uint16_t *>(base) + int64_t(i0) * d + wave * kq;
    const uint16_t *gp0 = w0 + slab::src(lane, 0, d), *gp1 = w0 + slab::src(lane, 1, d);
    const int64_t um = int64_t(I) * d;            // Wu follows Wg
    const bool live = j < n;
    uint8_t *t = tr[wave];

    // This lane's token (the shared expert's rows are the tokens in order),
    // read before the weights are issued: memory reads complete in order, so
    // waiting for it later leaves the weight batch in flight.  Lanes past
    // the item's rows read its last row: an MFMA output column depends only
    // on its own B column, and those columns are never stored.  Every read is
    // unconditional, so the compiler's waits stay exact.
    const int jr = it.row0 + min(j, n - 1);
    const int64_t xrow = sh ? int64_t(jr) : int64_t(L.perm[jr]);
    // The quarter goes in chunks of NB batches, each fully unrolled: weight
    // and token batches are double-buffered in registers (batch b + 1 is in
    // flight while batch b is rearranged and multiplied), and with no
    // register live across chunks the compiler's memory waits stay exact.
    // (The empty asm statements keep the issue order: token index, weights,
    // token rows.)
    const uint16_t *xp = reinterpret_cast<const uint16_t *>(L.x) + xrow * d + wave * kq + kg;
    auto load_w = [&](u32x4(&dst)[2][SL][2], int k0) {
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int s = 0; s < SL; ++s) {
                dst[m][s][0] = load_stream16(gp0 + m * um + k0 + 64 * s);
                dst[m][s][1] = load_stream16(gp1 + m * um + k0 + 64 * s);
            }
    };
    auto load_x = [&](u32x4(&dst)[U], int k0) {
#pragma unroll
        for (int u = 0; u < U; ++u)
            dst[u] = *reinterpret_cast<const u32x4 *>(xp + k0 + 32 * u);
    };
    f32x4 ag = {0.f, 0.f, 0.f, 0.f}, au = {0.f, 0.f, 0.f, 0.f};
    const int nchunk = kq / (32 * U * NB);
    for (int c = 0; c < nchunk; ++c) {
        const int kc = c * 32 * U * NB;
        u32x4 w[2][2][SL][2], xb[2][U];               // [buffer][matrix][slab][load]
        asm volatile("" ::: "memory");
        load_w(w[0], kc);
        asm volatile("" ::: "memory");
        load_x(xb[0], kc);
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            if (b + 1 < NB) {
                load_w(w[(b + 1) & 1], kc + (b + 1) * 32 * U);
                load_x(xb[(b + 1) & 1], kc + (b + 1) * 32 * U);
            }
            // rearrange batch b into fragments
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int s = 0; s < SL; ++s)
#pragma unroll
                    for (int q = 0; q < 2; ++q)
                        *reinterpret_cast<u32x4 *>(t + (m * SL + s) * slab::BYTES + slab::dst(lane, q)) =
                            w[b & 1][m][s][q];
            lds_wait();
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const bf16x8 bx = as_bf16x8(xb[b & 1][u]);
                const u32x4 fg =
                    *reinterpret_cast<const u32x4 *>(t + (u >> 1) * slab::BYTES + slab::frag(lane, u & 1));
                const u32x4 fu =
                    *reinterpret_cast<const u32x4 *>(t + (SL + (u >> 1)) * slab::BYTES + slab::frag(lane, u & 1));
                ag = mfma16(as_bf16x8(fg), bx, ag);
                au = mfma16(as_bf16x8(fu), bx, au);
            }
            lds_wait();                               // the next batch overwrites this wavefront's slabs
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
    for (int r = 0; r < 4; ++r) {
        ag[r] = ((ag[r] + red[0][0][lane][r]) + red[1][0][lane][r]) + red[2][0][lane][r];
        au[r] = ((au[r] + red[0][1][lane][r]) + red[1][1][lane][r]) + red[2][1][lane][r];
    }
    if (!slot_gen_ok(it, gnow, L.status))
        return;
    // lane holds rows i0 + 4*(lane/16) + r of token j
    if (live) {
        uint2 v;
        v.x = pack_bf16x2(silu(ag[0]) * au[0], silu(ag[1]) * au[1]);
        v.y = pack_bf16x2(silu(ag[2]) * au[2], silu(ag[3]) * au[3]);
        uint16_t *act = reinterpret_cast<uint16_t *>(sh ? L.act_s : L.act) + int64_t(it.row0 + j) * I + i0 +
                        4 * (lane >> 4);
        *reinterpret_cast<uint2 *>(act) = v;
    }
}

// Down, stream path: a workgroup owns 64 output columns (16 per wavefront)
// over all of I, in chunks of NB batches of 4 K steps (2 slabs of Wd rows,
// loaded in whole lines and rearranged through the wavefront's LDS as in the
// gate/up kernel), each chunk fully unrolled.  The lanes of token j (B
// operand) read row j of the item's act rows straight from memory with each
// weight batch (the rows are contiguous and few; lanes past the item's rows
// read its last row, whose outputs are never stored), so no workgroup
// barrier or LDS staging comes before the first MFMA.
template <int NB>
__global__ void __launch_bounds__(256, 4) stream_down_kernel(ExpertLaunch L)
{
    constexpr int U = 4, SL = U / 2;
    __shared__ __attribute__((aligned(16))) uint8_t tr[stream::WAVES][SL * slab::BYTES];
    const int d = L.d, I = L.I;
    const StreamTile st = stream_tile(L, d / (stream::WAVES * stream::ROWS));
    if (!st.valid)
        return;
    const WorkItem &it = st.it;
    const int n = it.nrows;
    const bool sh = it.slot < 0;
    const uint32_t gnow = slot_gen_now(it, L.gen_dev);

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int c0 = (st.local * stream::WAVES + wave) * stream::ROWS;
    const int j = lane & 15, kg = (lane >> 4) * 8;
    const uint8_t *base = sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const uint16_t *w0 = reinterpret_cast<const uint16_t *>(base) + int64_t(2) * I * d + int64_t(c0) * I;
    const uint16_t *gp0 = w0 + slab::src(lane, 0, I), *gp1 = w0 + slab::src(lane, 1, I);
    const uint16_t *ap = reinterpret_cast<const uint16_t *>(sh ? L.act_s : L.act) +
                         int64_t(it.row0 + min(j, n - 1)) * I + kg;
    const bool live = j < n;
    uint8_t *t = tr[wave];
    auto load_w = [&](u32x4(&dst)[SL][2], u32x4(&adst)[U], int k0) {
#pragma unroll
        for (int s = 0; s < SL; ++s) {
            dst[s][0] = load_stream16(gp0 + k0 + 64 * s);
            dst[s][1] = load_stream16(gp1 + k0 + 64 * s);
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            adst[u] = *reinterpret_cast<const u32x4 *>(ap + k0 + 32 * u);
    };
    u32x4 w[2][SL][2], av[2][U];
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    const int nchunk = I / (32 * U * NB);
    for (int c = 0; c < nchunk; ++c) {
        const int kc = c * 32 * U * NB;
        asm volatile("" ::: "memory");
        load_w(w[0], av[0], kc);
        if (NB > 1)
            load_w(w[1], av[1], kc + 32 * U);
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            if (b >= 1 && b + 1 < NB)                 // batches 0 and 1 went out with the chunk
                load_w(w[(b + 1) & 1], av[(b + 1) & 1], kc + (b + 1) * 32 * U);
#pragma unroll
            for (int s = 0; s < SL; ++s)
#pragma unroll
                for (int q = 0; q < 2; ++q)
                    *reinterpret_cast<u32x4 *>(t + s * slab::BYTES + slab::dst(lane, q)) = w[b & 1][s][q];
            lds_wait();
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const u32x4 fw = *reinterpret_cast<const u32x4 *>(t + (u >> 1) * slab::BYTES + slab::frag(lane, u & 1));
                acc = mfma16(as_bf16x8(fw), as_bf16x8(av[b & 1][u]), acc);
            }
            lds_wait();                               // the next batch overwrites this wavefront's slabs
        }
    }
    if (!slot_gen_ok(it, gnow, L.status))
        return;
    if (live) {
        const int64_t row = it.row0 + j;
        const float wt = sh ? 1.0f : L.row_weight[row];
        *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(sh ? L.ys : L.y) + row * d + c0 + 4 * (lane >> 4)) =
            make_uint2(pack_bf16x2(acc[0] * wt, acc[1] * wt), pack_bf16x2(acc[2] * wt, acc[3] * wt));
    }
}

hipError_t launch_gateup_stream(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    // chunks of NB batches of U K steps of 32 must divide the quarter d / 4 (d % 256 == 0)
    const int kq = L.d / 4;
    if (kq % 512 == 0)
        launch_k(stream_gateup_kernel<4, 4>, L.n_tiles, 256, 0, s, L);
    else if (kq % 256 == 0)
        launch_k(stream_gateup_kernel<4, 2>, L.n_tiles, 256, 0, s, L);
    else if (kq % 128 == 0)
        launch_k(stream_gateup_kernel<4, 1>, L.n_tiles, 256, 0, s, L);
    else
        launch_k(stream_gateup_kernel<2, 1>, L.n_tiles, 256, 0, s, L);
    return hipGetLastError();
}

hipError_t launch_down_stream(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    // chunks of NB batches of 128 columns must divide I (I % 128 == 0)
    if (L.I % 512 == 0)
        launch_k(stream_down_kernel<4>, L.n_tiles, 256, 0, s, L);
    else if (L.I % 256 == 0)
        launch_k(stream_down_kernel<2>, L.n_tiles, 256, 0, s, L);
    else
        launch_k(stream_down_kernel<1>, L.n_tiles, 256, 0, s, L);
    return hipGetLastError();
}

// ============================================================== f32 path

namespace f32p {
constexpr int TR = 16, TC = 16;   // 16 rows x 16 columns per 256-thread block
}

int tiles_gateup_f32(int nrows, int d, int I)
{
    (void)d;
    return ((nrows + f32p::TR - 1) / f32p::TR) * (I / f32p::TC);
}

int tiles_down_f32(int nrows, int d, int I)
{
    (void)I;
    return ((nrows + f32p::TR - 1) / f32p::TR) * (d / f32p::TC);
}

__global__ void __launch_bounds__(256) gateup_f32_kernel(ExpertLaunch L)
{
    const int t = int(blockIdx.x);
    const WorkItem it = L.items[find_item(L.items, L.n_items, t)];
    if (!slot_current(it, L.gen_dev, L.status))
        return;
    const int local = t - it.tile0;
    const int nct = L.I / f32p::TC;
    const int r = (local / nct) * f32p::TR + int(threadIdx.x) / f32p::TC;
    const int c = (local % nct) * f32p::TC + int(threadIdx.x) % f32p::TC;
    if (r >= it.nrows)
        return;
    const int d = L.d;
    const bool sh = it.slot < 0;
    const int64_t src = sh ? int64_t(it.row0 + r) : int64_t(L.perm[it.row0 + r]);
    const float *x = reinterpret_cast<const float *>(L.x) + src * d;
    const uint8_t *base = sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const float *wg = reinterpret_cast<const float *>(base) + int64_t(c) * d;
    const float *wu = wg + int64_t(L.I) * d;
    float g = 0.f, u = 0.f;
    for (int k = 0; k < d; ++k) {
        g = fmaf(x[k], wg[k], g);
        u = fmaf(x[k], wu[k], u);
    }
    reinterpret_cast<float *>(sh ? L.act_s : L.act)[int64_t(it.row0 + r) * L.I + c] = silu(g) * u;
}

__global__ void __launch_bounds__(256) down_f32_kernel(ExpertLaunch L)
{
    const int t = int(blockIdx.x);
    const WorkItem it = L.items[find_item(L.items, L.n_items, t)];
    if (!slot_current(it, L.gen_dev, L.status))
        return;
    const int local = t - it.tile0;
    const int nct = L.d / f32p::TC;
    const int r = (local / nct) * f32p::TR + int(threadIdx.x) / f32p::TC;
    const int c = (local % nct) * f32p::TC + int(threadIdx.x) % f32p::TC;
    if (r >= it.nrows)
        return;
    const int I = L.I;
    const int64_t row = it.row0 + r;
    const bool sh = it.slot < 0;
    const float *a = reinterpret_cast<const float *>(sh ? L.act_s : L.act) + row * I;
    const uint8_t *base = sh ? L.shared_w : L.wbase + uint64_t(it.slot) * L.wstride;
    const float *wd = reinterpret_cast<const float *>(base) + int64_t(2) * I * L.d + int64_t(c) * I;
    float acc = 0.f;
    for (int k = 0; k < I; ++k)
        acc = fmaf(a[k], wd[k], acc);
    const float w = sh ? 1.0f : L.row_weight[row];
    static_cast<float *>(sh ? L.ys : L.y)[row * L.d + c] = acc * w;
}

hipError_t launch_gateup_f32(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    launch_k(gateup_f32_kernel, L.n_tiles, 256, 0, s, L);
    return hipGetLastError();
}

hipError_t launch_down_f32(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    launch_k(down_f32_kernel, L.n_tiles, 256, 0, s, L);
    return hipGetLastError();
}

}  // namespace msi

namespace msi {

hipError_t init_kernel_attributes()
{
    hipError_t e = hipSuccess;
    auto set = [&](const void *f) {
        if (e == hipSuccess)
            e = allow_large_lds(f);
    };
    set(reinterpret_cast<const void *>(&stream_down_kernel<4>));
    set(reinterpret_cast<const void *>(&stream_down_kernel<2>));
    set(reinterpret_cast<const void *>(&stream_down_kernel<1>));
    if (e == hipSuccess)
        e = init_tile_attributes();
    if (e == hipSuccess)
        e = init_route_attributes();
    if (e == hipSuccess)
        e = init_q4_attributes();
    if (e == hipSuccess)
        e = init_kq_attributes();
    return e;
}

}  // namespace msi
