// kernels.h -- host launchers of the gfx950 kernels (all asynchronous on the
// given stream; they return the launch error, if any).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

#include "common.h"

namespace msi {

// Per-launch telemetry: while `stop` is set, kernels launched through
// launch_k carry HIP events that the runtime records at the first kernel's
// start and at each kernel's end (the last one's end is the one that stays),
// so the measured span is the kernels' own execution, not the host's
// enqueue gaps.
struct LaunchTiming {
    hipEvent_t start = nullptr, stop = nullptr;
};
inline LaunchTiming &launch_timing()
{
    static thread_local LaunchTiming t;
    return t;
}

template <typename... KArgs, typename... Args>
inline void launch_k(void (*k)(KArgs...), dim3 grid, dim3 block, size_t lds, hipStream_t s, Args &&...args)
{
    LaunchTiming &t = launch_timing();
    if (t.stop) {
        hipExtLaunchKernelGGL<KArgs...>(k, grid, block, uint32_t(lds), s, t.start, t.stop, 0u,
                                        static_cast<KArgs>(std::forward<Args>(args))...);
        t.start = nullptr;
    } else {
        k<<<grid, block, lds, s>>>(std::forward<Args>(args)...);
    }
}

// ---- router and permutation (route.hip)
hipError_t launch_router_logits_f32(const float *x, const float *wr, const float *bias, float *L, int T, int d,
                                    int E, hipStream_t s);
hipError_t launch_router_logits_bf16(const uint16_t *x, const uint16_t *wr, const float *bias, float *L, int T,
                                     int d, int E, hipStream_t s);
// raise the dynamic LDS limit of the kernels that use more than 64 KiB
hipError_t init_kernel_attributes();

// Let kernel f use all of the CU's 160 KiB of LDS (dynamic part = 160 KiB
// minus its static LDS).
inline hipError_t allow_large_lds(const void *f)
{
    hipFuncAttributes a{};
    hipError_t e = hipFuncGetAttributes(&a, f);
    if (e != hipSuccess)
        return e;
    return hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize,
                               int(160 * 1024 - a.sharedSizeBytes));
}
// Outputs of one routing (device arrays, see msi_routing).
struct RouteOut {
    int32_t *idx;
    float *w;
    int32_t *counts;
    int32_t *offsets;
    int32_t *demand;
    int32_t *perm;
    int32_t *inv;
    float *row_weight;
};
// top-K + restricted softmax + permutation of logits L (bias included): one
// fused workgroup when T <= 256, else top-K, histogram, scan and scatter
hipError_t launch_route_select(const float *L, const RouteOut &o, int32_t *blockhist, int T, int K, int E,
                               hipStream_t s);
hipError_t init_route_attributes();
hipError_t init_tile_attributes();
// decode routing for 1 <= T <= 16 tokens (bf16) in one launch: logits plus
// bias to L, then, in the last workgroup to finish, top-K, softmax and
// permutation.  `arrive` is a zero device word that the launch leaves zero;
// launches that share it must not overlap.
hipError_t launch_route_decode(const uint16_t *x, const uint16_t *wr, const float *bias, float *L,
                               uint32_t *arrive, const RouteOut &o, int T, int d, int K, int E, hipStream_t s);

// ---- expert projections (experts.hip).  `items` lists the experts of one
// launch (device memory), `n_tiles` the launch's total tile count.
struct ExpertLaunch {
    const WorkItem *items;
    int n_items;
    int n_tiles;
    const void *x;               // [T, d] hidden states (bf16 or f32)
    const int32_t *perm;         // gather map of routed rows
    const uint8_t *wbase;        // slot pool
    uint64_t wstride;
    // items with slot < 0 are the shared expert: weights at shared_w, rows
    // are tokens (no gather), act / y go to act_s / ys, weight 1
    const uint8_t *shared_w;
    void *act_s;
    void *ys;                    // [T, d] shared-expert output (bf16; f32 for f32 layers)
    const uint32_t *gen_dev;
    uint32_t *status;
    void *act;                   // [rows, I] bf16 (f32 for f32 layers)
    void *y;                     // [rows, d] weighted expert outputs (bf16; f32 for f32 layers)
    const float *row_weight;     // per permuted row, or null (1.0)
    int d, I;
    // device-built work list (stream kernels only): items resolved by each
    // workgroup from the routing's demanded experts and the residency table;
    // the grid (n_tiles) is then an upper bound and workgroups past the last
    // item exit.  direct.demand null: `items` is the list.
    DirectList direct;
    // device-built work list: when set, the list's length (items, tiles) is
    // read from here and the grid (n_tiles on the host) is an upper bound
    const DevCount *dev_n;
    // router logits launches (ring tiles in router mode) only: x [T, d] tokens,
    // wbase the router weight [E, d], logits[t, e] = x[t] . Wr[e] + bias[e]
    const float *bias;
    float *logits;
    int T, E;
};

// Tile of this workgroup and the launch's work counts: from the device-built
// list (L.dev_n; the grid is an upper bound, tiles spread over the XCDs by
// the real count) or the host list (the grid is the tile count); -1 if this
// workgroup has no tile.  (Scalar loads: the counts are uniform.)
__device__ __forceinline__ int launch_tile(const ExpertLaunch &L, int &n_items, int &n_tiles)
{
    if (L.dev_n) {
        n_items = __builtin_amdgcn_readfirstlane(L.dev_n->n_items);
        n_tiles = __builtin_amdgcn_readfirstlane(L.dev_n->n_tiles);
        return xcd_tile(int(blockIdx.x), n_tiles);
    }
    n_items = L.n_items;
    n_tiles = L.n_tiles;
    return xcd_swizzle(int(blockIdx.x), int(gridDim.x));
}

// Row and weight-slice geometry of a tile-path launch kind: an item of n
// rows has ceil(n / rows) * slices tiles.
struct TileGeom {
    int rows, slices;
};
TileGeom geom_gateup_tile(int d, int I);
TileGeom geom_down_tile(int d, int I);
TileGeom geom_gateup_q4_tile(int d, int I);
TileGeom geom_down_q4_tile(int d, int I);

// Device-built work list of a forward whose demanded experts are all
// published (build_worklist_kernel): the four launch lists (tile and stream
// path, gate/up and down), each ascending by expert, the shared expert first
// in the tile lists, with their counts.
struct WorklistArgs {
    const int32_t *counts, *offsets;     // routing
    const int32_t *slot_of;              // [E] published global slot, -1 if none
    const uint32_t *gen_of;              // [E] published generation
    uint32_t *status;                    // STATUS_MISS if a demanded expert is unpublished
    WorkItem *items[4];                  // gate/up tile, down tile, gate/up stream, down stream; E + 1 each
    DevCount *counts_out;                // [4]
    int E, T, thr, has_shared;
    int clear_status;                    // zero the status word first (the last forward left it set)
    TileGeom gu, dn;                     // tile-path geometry
    int per_gu_stream, per_dn_stream;    // tiles per stream item
};
hipError_t launch_build_worklist(const WorklistArgs &A, hipStream_t s);

// tiles per item of each launch kind
int tiles_gateup_tile(int nrows, int d, int I);
int tiles_down_tile(int nrows, int d, int I);
int tiles_gateup_stream(int nrows, int d, int I);
int tiles_down_stream(int nrows, int d, int I);
int tiles_gateup_f32(int nrows, int d, int I);
int tiles_down_f32(int nrows, int d, int I);

hipError_t launch_gateup_tile(const ExpertLaunch &L, hipStream_t s);
hipError_t launch_down_tile(const ExpertLaunch &L, hipStream_t s);
hipError_t launch_gateup_stream(const ExpertLaunch &L, hipStream_t s);
hipError_t launch_down_stream(const ExpertLaunch &L, hipStream_t s);
hipError_t launch_gateup_f32(const ExpertLaunch &L, hipStream_t s);
hipError_t launch_down_f32(const ExpertLaunch &L, hipStream_t s);

// 4-bit block-quantized experts (experts_q4.hip)
int tiles_gateup_q4_stream(int nrows, int d, int I);
int tiles_down_q4_stream(int nrows, int d, int I);
int tiles_gateup_q4_tile(int nrows, int d, int I);
int tiles_down_q4_tile(int nrows, int d, int I);
hipError_t launch_gateup_q4_stream(const ExpertLaunch &L, hipStream_t s);
hipError_t launch_down_q4_stream(const ExpertLaunch &L, hipStream_t s);
hipError_t launch_gateup_q4_tile(const ExpertLaunch &L, hipStream_t s);
hipError_t launch_down_q4_tile(const ExpertLaunch &L, hipStream_t s);
hipError_t init_q4_attributes();

// quantized-expert mix, Wg / Wu in k4 and Wd in k6 (experts_kq.hip)
int tiles_gateup_kq_stream(int nrows, int d, int I);
int tiles_down_kq_stream(int nrows, int d, int I);
int tiles_gateup_kq_tile(int nrows, int d, int I);
int tiles_down_kq_tile(int nrows, int d, int I);
TileGeom geom_gateup_kq_tile(int d, int I);
TileGeom geom_down_kq_tile(int d, int I);
hipError_t launch_gateup_kq_stream(const ExpertLaunch &L, hipStream_t s);
hipError_t launch_down_kq_stream(const ExpertLaunch &L, hipStream_t s);
hipError_t launch_gateup_kq_tile(const ExpertLaunch &L, hipStream_t s);
hipError_t launch_down_kq_tile(const ExpertLaunch &L, hipStream_t s);
hipError_t init_kq_attributes();

// The expert kernels of one storage format: the tile path (rows above the
// stream threshold, and every row of an f32 layer) and the stream path, for
// gate/up and down, with their tiles per item and tile geometry.  f32 layers
// have no stream path and no device-built lists (null entries).
struct KernelSet {
    using Tiles = int (*)(int nrows, int d, int I);
    using Geom = TileGeom (*)(int d, int I);
    using Launch = hipError_t (*)(const ExpertLaunch &L, hipStream_t s);
    Tiles tiles_gu_tile, tiles_gu_stream, tiles_dn_tile, tiles_dn_stream;
    Geom geom_gu, geom_dn;
    Launch gu_tile, gu_stream, dn_tile, dn_stream;
};

// ---- combine / publication and slot generation words (combine.hip)
// Status word of a forward and where the combine publishes it.
struct CombinePublish {
    uint32_t *status;            // device status word
    uint32_t *arrive;            // zero device word, left zero: the last workgroup to read the status
                                 // clears it; or null (large grids): the word is left as it is
    uint32_t *host;              // pinned host words (device-visible address), or null:
                                 // [0] status | STATUS_DONE, then, with demand, [1] count, [2..] ids
    const int32_t *demand;       // routing's demanded experts, or null
};
// out[t] = ys[t] + sum_k y[inv[t, k]] in that order (y, ys bf16, or fp32 when
// f32), unless the status word is nonzero
hipError_t launch_combine(const void *y, const void *ys, bool f32, const int32_t *inv, float *out,
                          const CombinePublish &P, int T, int K, int d, hipStream_t s);
constexpr int GEN_BATCH = 64;
struct GenBatch {
    uint32_t n;
    uint32_t slot[GEN_BATCH];
    uint32_t value[GEN_BATCH];
};
hipError_t launch_set_gens(uint32_t *gen_dev, const GenBatch &b, hipStream_t s);
// x0 != null: h = float(x0); else h += out.  Then x = bf16(rmsnorm(h)) per row.
hipError_t launch_residual(const uint16_t *x0, const float *out, float *h, uint16_t *x, int rows, int cols,
                           hipStream_t s);
hipError_t launch_clear_word(uint32_t *word, hipStream_t s);

}  // namespace msi
