// tiles.hip -- launches of the ring tile kernels (gemm_ring.h): the
// routed-expert gate/up and down projections of experts with more than 16
// routed rows, and the router logits of batches of more than 16 tokens.
#include "common.h"
#include "gemm_ring.h"
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

TileGeom geom_gateup_tile(int d, int I)
{
    (void)d;
    return TileGeom{ring::TM, I / 128};
}

TileGeom geom_down_tile(int d, int I)
{
    (void)I;
    return TileGeom{ring::TM, d / ring::TN};
}

// workgroups of a persistent launch: one per compute unit
static int g_persistent_wgs = 256;

hipError_t launch_gateup_tile(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    // (the persistent form is slower for gate/up: its extra state spills registers, and the spill reloads
    // wait for every copy in flight)
    launch_k(ring_gemm_kernel<RingMode::GateUp>, L.n_tiles, ring::THREADS, 0, s, L);
    return hipGetLastError();
}

hipError_t launch_down_tile(const ExpertLaunch &L, hipStream_t s)
{
    if (L.n_tiles == 0)
        return hipSuccess;
    if ((L.I / ring::SK) % 4 == 0 && L.I / ring::SK >= 8 && L.n_tiles > g_persistent_wgs) {
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
    ExpertLaunch R{};
    R.x = x;
    R.wbase = reinterpret_cast<const uint8_t *>(wr);
    R.d = d;
    R.bias = bias;
    R.logits = L;
    R.T = T;
    R.E = E;
    const int tiles = ((T + ring::TM - 1) / ring::TM) * ((E + ring::TN - 1) / ring::TN);
    launch_k(ring_gemm_kernel<RingMode::Router>, tiles, ring::THREADS, 0, s, R);
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
    return hipSuccess;
}

}  // namespace msi
