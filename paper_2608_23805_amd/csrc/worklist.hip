// worklist.hip -- the work list of a forward built on the device, when every
// demanded expert of the layer is published: the host then needs neither
// the per-expert counts nor a schedule before launching the expert kernels
// (no device-to-host round trip between the routing and the expert work).
#include "common.h"
#include "kernels.h"

namespace msi {

// Exclusive scan of one value per thread over a 1024-thread workgroup, and
// the total (integers: the grouping does not change the result).
__device__ __forceinline__ int scan_excl_1024(int v, int32_t *wsum, int &total)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int x = wave_scan_incl(v);
    __syncthreads();                            // wsum is reused by consecutive scans
    if (lane == 63)
        wsum[wave] = x;
    __syncthreads();
    int base = 0;
    total = 0;
    for (int w = 0; w < 16; ++w) {
        base += w < wave ? wsum[w] : 0;
        total += wsum[w];
    }
    return base + x - v;
}

// One 1024-thread workgroup, thread e for expert e (E <= 1024): an expert
// with more than thr rows goes to the tile lists (ceil(rows / geom.rows) *
// geom.slices tiles), one with 1..thr rows to the stream lists; ascending by
// expert, the shared expert's item first in the tile lists, so the lists and
// their tile numbering are those the host schedule builds for an all-resident
// round.  A demanded expert without a published slot raises STATUS_MISS.
// With clear_status the kernel first zeroes the status word (in place of a
// launch of its own): the store completes before the workgroup's barrier,
// ahead of any bit this forward raises.
__global__ void __launch_bounds__(1024) build_worklist_kernel(WorklistArgs A)
{
    __shared__ int32_t wsum[16];
    if (A.clear_status) {
        if (threadIdx.x == 0)
            __hip_atomic_store(A.status, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __syncthreads();
    }
    const int e = threadIdx.x;
    const bool in = e < A.E;
    const int c = in ? A.counts[e] : 0;
    const int slot = in ? A.slot_of[e] : -1;
    const uint32_t gen = in ? A.gen_of[e] : 0u;
    const int row0 = in ? A.offsets[e] : 0;
    if (c > 0 && slot < 0)
        atomicOr(A.status, STATUS_MISS);
    const bool tile = c > A.thr, stream = c > 0 && c <= A.thr;
    const int tg = tile ? (c + A.gu.rows - 1) / A.gu.rows * A.gu.slices : 0;
    const int td = tile ? (c + A.dn.rows - 1) / A.dn.rows * A.dn.slices : 0;
    int n_tile, n_stream, n_tg, n_td;
    const int p_tile = scan_excl_1024(tile ? 1 : 0, wsum, n_tile);
    const int p_stream = scan_excl_1024(stream ? 1 : 0, wsum, n_stream);
    const int p_tg = scan_excl_1024(tg, wsum, n_tg);
    const int p_td = scan_excl_1024(td, wsum, n_td);
    const int sh = A.has_shared ? 1 : 0;
    const int sh_tg = sh ? (A.T + A.gu.rows - 1) / A.gu.rows * A.gu.slices : 0;
    const int sh_td = sh ? (A.T + A.dn.rows - 1) / A.dn.rows * A.dn.slices : 0;
    if (tile) {
        A.items[0][sh + p_tile] = WorkItem{e, slot, gen, row0, c, sh_tg + p_tg};
        A.items[1][sh + p_tile] = WorkItem{e, slot, gen, row0, c, sh_td + p_td};
    }
    if (stream) {
        A.items[2][p_stream] = WorkItem{e, slot, gen, row0, c, p_stream * A.per_gu_stream};
        A.items[3][p_stream] = WorkItem{e, slot, gen, row0, c, p_stream * A.per_dn_stream};
    }
    if (e == 0) {
        if (sh) {
            A.items[0][0] = WorkItem{-1, -1, 0u, 0, A.T, 0};
            A.items[1][0] = WorkItem{-1, -1, 0u, 0, A.T, 0};
        }
        A.counts_out[0] = DevCount{sh + n_tile, sh_tg + n_tg};
        A.counts_out[1] = DevCount{sh + n_tile, sh_td + n_td};
        A.counts_out[2] = DevCount{n_stream, n_stream * A.per_gu_stream};
        A.counts_out[3] = DevCount{n_stream, n_stream * A.per_dn_stream};
    }
}

hipError_t launch_build_worklist(const WorklistArgs &A, hipStream_t s)
{
    if (A.E <= 0 || A.E > 1024)
        return hipErrorInvalidValue;
    launch_k(build_worklist_kernel, 1, 1024, 0, s, A);
    return hipGetLastError();
}

}  // namespace msi
