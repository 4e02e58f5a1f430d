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
// streaming router for 1 <= T <= 16 tokens (bf16): partial logits
// P[ROUTER_SPLIT][T][E] without the bias
constexpr int ROUTER_SPLIT = 4;
hipError_t launch_router_stream(const uint16_t *x, const uint16_t *wr, float *P, int T, int d, int E,
                                hipStream_t s);
// top-K + restricted softmax + permutation (one fused workgroup when T <= 256).
// With P (T <= 16 only) the logits are formed from the partials plus the bias
// and stored to L; otherwise they are read from L.
hipError_t launch_route_select(float *L, const float *P, const float *bias, int32_t *idx, float *w,
                               int32_t *counts, int32_t *offsets, int32_t *perm, int32_t *inv, float *row_weight,
                               int32_t *blockhist, int T, int K, int E, hipStream_t s);
hipError_t init_route_attributes();

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
    // device-built work list: {n_items, n_tiles} read by the kernel (the
    // grid is an upper bound; workgroups past n_tiles exit), or null
    const int32_t *dev_counts;
};

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

// Device-built stream-path work list of one forward whose demanded experts
// are all published (one workgroup): shared expert first, then demanded
// experts in ascending id; a demanded expert without a published slot sets
// STATUS_MISS in *status and gets an item that writes nothing.  info =
// {n_gu, tiles_gu, n_dn, tiles_dn}; host_counts[E] (pinned host words,
// device-visible address) receives the per-expert token counts.
hipError_t launch_fast_worklist(const int32_t *counts, const int32_t *offsets, const int32_t *slot_of,
                                const uint32_t *gen_of, int E, int T, int has_shared, int tpg, int tpd,
                                WorkItem *gu, WorkItem *dn, int32_t *info, uint32_t *status, uint32_t *host_counts,
                                hipStream_t s);

// ---- combine / publication and slot generation words (combine.hip)
// out[t] = ys[t] + sum_k y[inv[t, k]] in that order (y, ys bf16, or fp32 when f32),
// unless *status is nonzero; *status is also copied to host_status (a pinned
// host word, device-visible address), if given
hipError_t launch_combine(const void *y, const void *ys, bool f32, const int32_t *inv, float *out,
                          const uint32_t *status, uint32_t *host_status, int T, int K, int d, hipStream_t s);
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
