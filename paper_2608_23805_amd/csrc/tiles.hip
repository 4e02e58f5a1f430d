// tiles.hip -- launches of the tile kernels: the routed-expert gate/up and
// down projections of experts with more than 16 routed rows (gemm_ring.h)
// and the router logits of long batches (gemm_tile.h).
#include "common.h"
#include "gemm_ring.h"
#include "gemm_tile.h"
#include "kernels.h"

namespace msi {

int tiles_gateup_tile(int nrows, int d, int I)
{
    (void)d;
    return ring_tiles_gateup(nrows, I);
}

int tiles_down_tile(int nrows, int d, int I)
{
    (void)I;
    return ring_tiles_down(nrows, d);
}

hipError_t launch_gateup_tile(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    launch_k(ring_gemm_kernel<RingMode::GateUp>, L.n_tiles, ring::THREADS, 0, s, L);
    return hipGetLastError();
}

// workgroups of a persistent launch: one per compute unit
static int g_persistent_wgs = 256;

hipError_t launch_down_tile(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    if (L.I / ring::SK >= 8 && L.n_tiles > g_persistent_wgs) {
        // K loop long enough for the cross-tile pipeline: one workgroup per CU walks its tiles
        launch_k(ring_gemm_persistent<RingMode::Down>, g_persistent_wgs, ring::THREADS, 0, s, L);
    } else {
        launch_k(ring_gemm_kernel<RingMode::Down>, L.n_tiles, ring::THREADS, 0, s, L);
    }
    return hipGetLastError();
}

hipError_t launch_router_logits_bf16(const uint16_t *x, const uint16_t *wr, const float *bias, float *L, int T,
                                     int d, int E, hipStream_t s)
{
    if (T == 0)
        return hipSuccess;
    TileArgs p{};
    p.a = x;
    p.lda = d;
    p.perm = nullptr;
    p.wbase = reinterpret_cast<const uint8_t *>(wr);
    p.wstride = 0;
    p.K = d;
    p.n_valid = E;
    p.n_tiles_n = (E + tile::BN - 1) / tile::BN;
    p.d = d;
    p.items = nullptr;
    p.n_items = 1;
    p.single = WorkItem{-1, -1, 0u, 0, T, 0};
    p.gen_dev = nullptr;
    p.status = nullptr;
    p.out = L;
    p.ldo = E;
    p.bias = bias;
    const int tiles = ((T + tile::BM - 1) / tile::BM) * p.n_tiles_n;
    launch_k(tile_gemm_kernel<TileMode::Router>, tiles, tile::THREADS, tile::LDS_BYTES, s, p);
    return hipGetLastError();
}

hipError_t init_tile_attributes()
{
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess)
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess)
        return e;
    // a multiple of the 8 XCDs keeps each XCD's workgroups on its own tile range
    g_persistent_wgs = cus >= 8 ? cus / 8 * 8 : 8;
    return allow_large_lds(reinterpret_cast<const void *>(&tile_gemm_kernel<TileMode::Router>));
}

}  // namespace msi
