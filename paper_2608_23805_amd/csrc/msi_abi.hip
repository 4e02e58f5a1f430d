// msi_abi.hip -- C ABI of the slot-backed MoE layer (declared in include/msi.h).
//
// Host side of the paper's scheduling loop (Implementation, "Scheduling and
// copies"): layer entry requests
// the bundle of demanded experts, misses are copied from their host windows
// into reserved slots on a side stream, a device event publishes readiness,
// the expert kernels consume the slots at stable addresses, and layer exit
// releases the consumers.  Residency decisions live in PlanCore (pure C++);
// this file owns HIP memory, streams, events and kernel launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cstring>
#include <deque>
#include <mutex>
#include <new>
#include <string>
#include <unordered_map>
#include <vector>

#include "../../include/msi.h"
#include "kernels.h"
#include "plan_core.hpp"
#include "source.hpp"

using namespace msi;

namespace {

thread_local std::string g_err;
uint32_t g_stream_threshold = 16;   // tokens per expert at or below which the stream path runs

msi_status fail(msi_status st, const std::string &m)
{
    g_err = m;
    return st;
}

#define HIP_OK(expr)                                                                        \
    do {                                                                                    \
        hipError_t e_ = (expr);                                                             \
        if (e_ != hipSuccess)                                                               \
            return fail(MSI_E_DEVICE, std::string(#expr) + ": " + hipGetErrorString(e_)); \
    } while (0)

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// bytes of a [rows, cols] matrix; for MSI_W_KQ, `down` selects Wd's k6
// format (Wg and Wu are k4)
uint64_t matrix_bytes(uint32_t wdtype, uint64_t rows, uint64_t cols, bool down)
{
    switch (wdtype) {
    case MSI_W_F32: return rows * cols * 4;
    case MSI_W_BF16: return rows * cols * 2;
    case MSI_W_KQ:
        if (down)
            return rows * cols / 2 + rows * cols / 4 + rows * cols / 16 + rows * (cols / 256) * 2;
        return rows * cols / 2 + rows * (cols / 256) * 16;
    default: return rows * cols / 2 + rows * (cols / 32) * 2;
    }
}

// expert kernels of each storage format
const KernelSet &kernel_set(uint32_t wdtype)
{
    static const KernelSet f32{tiles_gateup_f32, nullptr, tiles_down_f32, nullptr, nullptr, nullptr,
                               launch_gateup_f32, nullptr, launch_down_f32, nullptr};
    static const KernelSet bf16{tiles_gateup_tile, tiles_gateup_stream, tiles_down_tile, tiles_down_stream,
                                geom_gateup_tile, geom_down_tile,
                                launch_gateup_tile, launch_gateup_stream, launch_down_tile, launch_down_stream};
    static const KernelSet q4{tiles_gateup_q4_tile, tiles_gateup_q4_stream, tiles_down_q4_tile,
                              tiles_down_q4_stream, geom_gateup_q4_tile, geom_down_q4_tile,
                              launch_gateup_q4_tile, launch_gateup_q4_stream, launch_down_q4_tile,
                              launch_down_q4_stream};
    static const KernelSet kq{tiles_gateup_kq_tile, tiles_gateup_kq_stream, tiles_down_kq_tile,
                              tiles_down_kq_stream, geom_gateup_kq_tile, geom_down_kq_tile,
                              launch_gateup_kq_tile, launch_gateup_kq_stream, launch_down_kq_tile,
                              launch_down_kq_stream};
    switch (wdtype) {
    case MSI_W_F32: return f32;
    case MSI_W_Q4B32: return q4;
    case MSI_W_KQ: return kq;
    default: return bf16;
    }
}

uint64_t object_bytes_of(const msi_plan_desc &d)
{
    return 2 * matrix_bytes(d.wdtype, d.d_ff, d.d_model, false) + matrix_bytes(d.wdtype, d.d_model, d.d_ff, true);
}

// Workspace layout for T tokens (offsets in bytes, each region 256-aligned).
struct Workspace {
    size_t logits, blockhist, act, act_s, y, ys, total;
};

Workspace workspace_layout(const msi_plan_desc &d, uint64_t T)
{
    const uint64_t E = d.n_experts, K = d.top_k, I = d.d_ff, D = d.d_model;
    const uint64_t nblk = (T + PERM_BLOCK - 1) / PERM_BLOCK;
    const uint64_t ab = d.wdtype == MSI_W_F32 ? 4 : 2;   // act element bytes
    Workspace w{};
    size_t off = 0;
    w.logits = off;
    off += align256(T * E * 4);
    w.blockhist = off;
    off += align256(std::max<uint64_t>(nblk, 1) * E * 4);
    w.act = off;
    off += align256(T * K * I * ab);
    w.act_s = off;
    off += align256(T * I * ab);
    w.y = off;
    off += align256(T * K * D * ab);    // y and ys: bf16 (fp32 for fp32 layers)
    w.ys = off;
    off += align256(T * D * ab);
    w.total = off;
    return w;
}

// act / y scratch of one forward (device pointers)
struct FwdBufs {
    uint8_t *act, *act_s, *y, *ys;
};

}  // namespace

// Scratch of msi_moe_forward_noalloc: the act and y parts of a forward's
// workspace live here, so that entry point needs no allocation.  Each device
// the library runs on holds its own copy for the life of the process; host
// code uses only the per-device address from scratch_address(), never the
// array's name (which in host code is a stand-in, not a device address).
static __device__ __align__(256) uint8_t scratch[MSI_NOALLOC_SCRATCH_BYTES];

namespace {

// Device address of `scratch` on `device`, looked up once per device with
// that device current (at plan creation).
hipError_t scratch_address(int device, void **out)
{
    static std::mutex mu;
    static std::unordered_map<int, void *> addr;
    std::lock_guard<std::mutex> lock(mu);
    auto it = addr.find(device);
    if (it != addr.end()) {
        *out = it->second;
        return hipSuccess;
    }
    void *ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess)
        return e;
    addr.emplace(device, ptr);
    *out = ptr;
    return hipSuccess;
}

}  // namespace

struct msi_plan {
    msi_plan_desc desc{};
    std::vector<const void *> windows;
    uint64_t object_bytes = 0;
    PlanCore *core = nullptr;
    SourceService *src = nullptr;       // bounded source service (plans whose objects live in files)
    // A fill whose bytes come from the source: queued, reading into a staging
    // window, copying window -> slot, then done; or failed (never published).
    struct SrcFill {
        FillRecord rec;
        hipStream_t side = nullptr;
        int round = -1;                 // forward round it serves; -1: an explicit fill (copied when ready)
        int window = -1;
        int state = 0;                  // SF_* below
        bool cancel = false;            // its forward failed: never copy it
        hipEvent_t ev = nullptr;        // copy complete (owned)
    };
    std::deque<SrcFill> sfills;         // submission order
    int src_round = -1;                 // rounds <= this may be copied (the forward's current round)
    struct FaultReq {
        uint32_t layer, expert, component, mode;
    };
    std::vector<FaultReq> src_faults;   // test hooks, applied at the object's next request
    double src_wait_s = 0.0;            // forwards blocked on the source
    int device = 0;
    void *scratch = nullptr;            // this device's copy of the static scratch (msi_moe_forward_noalloc)
    uint32_t *gen_dev = nullptr;        // [n_layers * pool_slots]
    uint32_t *status_dev = nullptr;     // [status, counts copy [E]] (device work-list path)
    WorkItem *table_dev = nullptr;
    WorkItem *table_host = nullptr;     // pinned staging
    size_t table_cap = 0;
    int32_t *counts_host = nullptr;     // pinned [E]
    uint32_t *status_host = nullptr;    // pinned
    std::vector<hipEvent_t> free_events;
    std::vector<hipEvent_t> all_events;
    std::vector<hipEvent_t> fill_ev;    // per global slot: pending fill (owned)
    std::vector<int64_t> fill_ev_id;    // fill id the pending event completes
    std::vector<hipEvent_t> release_ev; // per global slot: last round reading it (current forward)
    std::vector<uint8_t> fill_ev_shared;// event shared by a round batch (not owned per slot)
    // device work-list path (all demanded experts published)
    int32_t *res_slot_dev = nullptr;    // [n_layers][E] published global slot or -1
    uint32_t *res_gen_dev = nullptr;    // [n_layers][E]
    int32_t *res_host = nullptr;        // pinned staging [2 * E]
    uint32_t *arrive_dev = nullptr;     // arrival counters (zero between launches): [ARRIVE_ROUTE], [ARRIVE_COMBINE]
    WorkItem *dlist_dev = nullptr;      // device-built work lists: 4 x (E + 1) items
    DevCount *dcount_dev = nullptr;     // their counts [4]
    bool status_clean = true;           // status_dev is zero (the last forward's combine cleared it)
    uint32_t *tail_host = nullptr;      // pinned [2 + E]: status | DONE, demanded count, ids (written by the combine)
    uint32_t *tail_hdev = nullptr;      // device-visible address of tail_host
    uint32_t *status_hdev = nullptr;    // device-visible address of status_host
    std::vector<uint64_t> res_version;  // per layer: layer version uploaded
    std::vector<uint8_t> direct_ok;     // per layer: last forward needed no fill
    // timing telemetry
    struct Timed {
        int kind;
        hipEvent_t a, b;
    };
    bool timing = false;
    uint32_t timing_mask = 0;           // kernel kinds bracketed by events
    uint32_t timing_period = 1;         // time every period-th launch of a kind
    uint64_t timing_seen[MSI_NKERN] = {};
    std::vector<Timed> timed;
    std::vector<hipEvent_t> tfree;
    uint64_t t_launches[MSI_NKERN] = {};
    double t_ms[MSI_NKERN] = {};

    hipEvent_t get_tevent()
    {
        if (tfree.empty()) {
            hipEvent_t e;
            if (hipEventCreate(&e) != hipSuccess)
                return nullptr;
            all_events.push_back(e);
            return e;
        }
        hipEvent_t e = tfree.back();
        tfree.pop_back();
        return e;
    }

    // Run `launch` with telemetry when it is on for this kind: the kernels it
    // launches carry start / stop events recorded by the runtime at their own
    // start and end.  A launch that started no kernel leaves no sample.
    template <typename F>
    hipError_t timed_launch(int kind, hipStream_t s, F &&launch)
    {
        (void)s;
        if (!timing || !(timing_mask & (1u << kind)) || (timing_seen[kind]++ % timing_period) != 0)
            return launch();
        if (timed.size() >= 8192)
            resolve_timings();
        hipEvent_t a = get_tevent(), b = get_tevent();
        if (!a || !b)
            return hipErrorOutOfMemory;
        launch_timing() = LaunchTiming{a, b};
        const hipError_t e = launch();
        const bool used = launch_timing().start == nullptr;
        launch_timing() = LaunchTiming{};
        if (used)
            timed.push_back(Timed{kind, a, b});
        else {
            tfree.push_back(a);
            tfree.push_back(b);
        }
        return e;
    }

    // Copies are bracketed by events on their stream instead.
    template <typename F>
    hipError_t timed_copy(int kind, hipStream_t s, F &&copy)
    {
        if (!timing || !(timing_mask & (1u << kind)) || (timing_seen[kind]++ % timing_period) != 0)
            return copy();
        if (timed.size() >= 8192)
            resolve_timings();
        hipEvent_t a = get_tevent(), b = get_tevent();
        if (!a || !b)
            return hipErrorOutOfMemory;
        hipError_t e = hipEventRecord(a, s);
        if (e == hipSuccess)
            e = copy();
        if (e == hipSuccess)
            e = hipEventRecord(b, s);
        timed.push_back(Timed{kind, a, b});
        return e;
    }

    void resolve_timings()
    {
        for (const Timed &t : timed) {
            float ms = 0.f;
            if (hipEventSynchronize(t.b) == hipSuccess && hipEventElapsedTime(&ms, t.a, t.b) == hipSuccess) {
                t_launches[t.kind]++;
                t_ms[t.kind] += ms;
            }
            tfree.push_back(t.a);
            tfree.push_back(t.b);
        }
        timed.clear();
    }

    hipEvent_t get_event()
    {
        if (free_events.empty()) {
            hipEvent_t e;
            if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess)
                return nullptr;
            all_events.push_back(e);
            return e;
        }
        hipEvent_t e = free_events.back();
        free_events.pop_back();
        return e;
    }
};

namespace {

// Observe a completed fill event of global slot gs.
void observe_fill(msi_plan *p, uint32_t gs)
{
    if (!p->fill_ev[gs])
        return;
    p->core->complete_fill(p->fill_ev_id[gs]);
    if (!p->fill_ev_shared[gs])
        p->free_events.push_back(p->fill_ev[gs]);
    p->fill_ev[gs] = nullptr;
    p->fill_ev_id[gs] = -1;
    p->fill_ev_shared[gs] = 0;
}

void poll_fills(msi_plan *p)
{
    for (uint32_t gs = 0; gs < p->fill_ev.size(); ++gs)
        if (p->fill_ev[gs] && hipEventQuery(p->fill_ev[gs]) == hipSuccess)
            observe_fill(p, gs);
}

// ---- source-backed fills --------------------------------------------------
// States of a SrcFill.
constexpr int SF_QUEUED = 0, SF_READING = 1, SF_READY = 2, SF_COPYING = 3, SF_DONE = 4, SF_FAILED = 5;

msi_status source_error_status(SourceError e)
{
    switch (e) {
    case SourceError::Short: return MSI_E_SHORT;
    case SourceError::Io: return MSI_E_IO;
    case SourceError::Stale: return MSI_E_STALE;
    default: return MSI_E_SHORT;
    }
}

// Copy a HostReady window into its slot on the fill's side stream: after the
// slot's earlier fill and its last readers, invalidate the generation word,
// copy each extent from its place in the window to its offset in the slot,
// publish the generation, record the fill's event.
msi_status copy_window(msi_plan *p, msi_plan::SrcFill &f)
{
    const PlanCore &c = *p->core;
    const uint32_t gs = c.global_slot(f.rec.layer, f.rec.slot);
    const SourceObject *so = c.source_object(f.rec.layer, f.rec.expert);
    uint64_t place[SourceService::MAX_EXTENTS];
    if (!so || !p->src->layout(so->ext, so->n, place, nullptr))
        return fail(MSI_E_INVALID_ARG, "internal: source object layout");
    if (p->fill_ev[gs] && p->fill_ev[gs] != f.ev)
        HIP_OK(hipStreamWaitEvent(f.side, p->fill_ev[gs], 0));
    if (p->release_ev[gs])
        HIP_OK(hipStreamWaitEvent(f.side, p->release_ev[gs], 0));
    GenBatch inval{}, pub{};
    inval.n = pub.n = 1;
    inval.slot[0] = pub.slot[0] = gs;
    inval.value[0] = 0u;
    pub.value[0] = f.rec.gen;
    HIP_OK(launch_set_gens(p->gen_dev, inval, f.side));
    uint8_t *dst = static_cast<uint8_t *>(p->desc.slot_pool) + uint64_t(gs) * p->desc.slot_stride;
    for (int i = 0; i < so->n; ++i) {
        HIP_OK(hipMemcpyAsync(dst, p->src->window(uint32_t(f.window)) + place[i], so->ext[i].nbytes,
                              hipMemcpyHostToDevice, f.side));
        dst += so->ext[i].nbytes;
    }
    HIP_OK(launch_set_gens(p->gen_dev, pub, f.side));
    if (!f.ev && !(f.ev = p->get_event()))
        return fail(MSI_E_DEVICE, "event creation failed");
    HIP_OK(hipEventRecord(f.ev, f.side));
    p->src->set_copying(uint32_t(f.window));
    // the slot's pending fill is now this copy (the plan observes it through the event)
    if (p->fill_ev[gs] && !p->fill_ev_shared[gs])
        p->free_events.push_back(p->fill_ev[gs]);
    p->fill_ev[gs] = f.ev;
    p->fill_ev_id[gs] = f.rec.id;
    p->fill_ev_shared[gs] = 1;
    f.state = SF_COPYING;
    return MSI_OK;
}

// Whether a source fill may still be published: a forward's fill while the
// epoch holds (a later round of the same forward may reuse its slot, which
// supersedes the plan's record but not this round's copy); an explicit fill
// while it is its slot's current version.
bool sf_current(const msi_plan *p, const msi_plan::SrcFill &f)
{
    return f.round >= 0 ? f.rec.epoch == p->core->epoch() : p->core->fill_current(f.rec.id, f.rec.epoch, f.rec.gen);
}

// One step of the source engine: finished copies free their windows,
// completed reads are judged (a stale ticket, short read or negative status
// fails the fill closed: its window is freed, nothing is copied), ready
// windows whose round has come are copied, and queued fills are submitted
// into free windows (at most the service's in-flight limit reads at once).
// With wait_ms > 0 and no progress, waits for a read or the oldest copy.
// Returns the first failure of a fill that serves a forward round.
msi_status source_progress(msi_plan *p, int wait_ms)
{
    SourceService &S = *p->src;
    PlanCore &c = *p->core;
    msi_status first_err = MSI_OK;
    bool moved = false;
    for (msi_plan::SrcFill &f : p->sfills)
        if (f.state == SF_COPYING && hipEventQuery(f.ev) == hipSuccess) {
            S.set_free(uint32_t(f.window));
            const uint32_t gs = c.global_slot(f.rec.layer, f.rec.slot);
            if (p->fill_ev[gs] == f.ev) {
                p->core->complete_fill(f.rec.id);
                p->fill_ev[gs] = nullptr;
                p->fill_ev_id[gs] = -1;
                p->fill_ev_shared[gs] = 0;
            }
            f.state = SF_DONE;
            moved = true;
        }
    auto judge = [&](const std::vector<SourceService::Done> &done) {
        for (const SourceService::Done &d : done) {
            moved = true;
            for (msi_plan::SrcFill &f : p->sfills) {
                if (f.state != SF_READING || f.rec.id != int64_t(d.tag))
                    continue;
                if (d.error == SourceError::None && !f.cancel) {
                    f.state = SF_READY;
                } else {
                    if (d.error == SourceError::None)
                        S.set_free(d.window);               // cancelled: ready but never copied
                    c.fail_fill(f.rec.id);
                    f.state = SF_FAILED;
                    if (f.round >= 0 && !f.cancel && first_err == MSI_OK)
                        first_err = fail(source_error_status(d.error),
                                         std::string("source read of expert ") + std::to_string(f.rec.expert) +
                                             " failed (" +
                                             (d.error == SourceError::Short ? "short read"
                                              : d.error == SourceError::Io ? std::string("errno ") + std::to_string(d.sys_errno)
                                                                            : "stale ticket") +
                                             "); nothing published");
                }
                break;
            }
        }
    };
    auto current = [&](uint64_t tag, uint32_t, uint32_t) {
        for (const msi_plan::SrcFill &f : p->sfills)
            if (f.rec.id == int64_t(tag))
                return sf_current(p, f);
        return false;
    };
    judge(S.collect(0, current));
    for (msi_plan::SrcFill &f : p->sfills)
        if (f.state == SF_READY && (f.round < 0 || f.round <= p->src_round)) {
            if (!sf_current(p, f)) {                // superseded or reset meanwhile
                S.set_free(uint32_t(f.window));
                c.fail_fill(f.rec.id);
                f.state = SF_FAILED;
            } else {
                const msi_status st = copy_window(p, f);
                if (st != MSI_OK)
                    return st;
            }
            moved = true;
        }
    for (msi_plan::SrcFill &f : p->sfills) {
        if (f.state != SF_QUEUED)
            continue;
        if (f.cancel || !sf_current(p, f)) {
            c.fail_fill(f.rec.id);
            f.state = SF_FAILED;
            moved = true;
            continue;
        }
        const int w = S.free_window();
        if (w < 0)
            break;
        const SourceObject *so = c.source_object(f.rec.layer, f.rec.expert);
        for (auto it = p->src_faults.begin(); it != p->src_faults.end();)
            if (it->layer == f.rec.layer && it->expert == f.rec.expert) {
                S.inject(uint64_t(f.rec.id), int(it->component), SourceFault(it->mode));
                it = p->src_faults.erase(it);
            } else {
                ++it;
            }
        if (!so || !S.submit(uint32_t(w), so->ext, so->n, uint64_t(f.rec.id), f.rec.epoch, f.rec.gen))
            return fail(MSI_E_INVALID_ARG, "internal: source submission refused");
        f.window = w;
        f.state = SF_READING;
        moved = true;
    }
    while (!p->sfills.empty() && (p->sfills.front().state == SF_DONE || p->sfills.front().state == SF_FAILED)) {
        if (p->sfills.front().ev)
            p->free_events.push_back(p->sfills.front().ev);
        p->sfills.pop_front();
    }
    if (!moved && wait_ms > 0) {
        const auto t0 = std::chrono::steady_clock::now();
        if (S.outstanding()) {
            judge(S.collect(wait_ms, current));
        } else {
            for (msi_plan::SrcFill &f : p->sfills)
                if (f.state == SF_COPYING) {
                    (void)hipEventSynchronize(f.ev);
                    break;
                }
        }
        p->src_wait_s += std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
    }
    return first_err;
}

// Drive the engine until `done()` holds; stops at the first failure.
template <typename Pred>
msi_status source_until(msi_plan *p, Pred done)
{
    const auto t0 = std::chrono::steady_clock::now();
    while (!done()) {
        const msi_status st = source_progress(p, 5);
        if (st != MSI_OK)
            return st;
        if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(120))
            return fail(MSI_E_DEVICE, "source service made no progress for 120 s");
    }
    return MSI_OK;
}

// Cancel every forward fill not yet copied and drain the reads in flight:
// their windows return to Free and nothing of theirs is published.
void source_cancel_forward(msi_plan *p)
{
    for (msi_plan::SrcFill &f : p->sfills)
        if (f.round >= 0 && (f.state == SF_QUEUED || f.state == SF_READING || f.state == SF_READY))
            f.cancel = true;
    for (msi_plan::SrcFill &f : p->sfills)
        if (f.cancel && f.state == SF_READY) {
            p->src->set_free(uint32_t(f.window));
            p->core->fail_fill(f.rec.id);
            f.state = SF_FAILED;
        }
    (void)source_until(p, [&] {
        for (const msi_plan::SrcFill &f : p->sfills)
            if (f.state == SF_QUEUED || f.state == SF_READING || f.state == SF_COPYING)
                return false;
        return true;
    });
}

// Enqueue on `side` the invalidate -> copy -> publish sequence of a batch of
// fills (all ids already recorded by the core).  The side stream first waits
// for every earlier fill and every reading round of each target slot.
msi_status enqueue_fills(msi_plan *p, uint32_t layer, const std::vector<FillRecord> &fills, hipStream_t side)
{
    const PlanCore &c = *p->core;
    for (const FillRecord &fr : fills) {
        const FillRecord *f = &fr;
        const uint32_t gs = c.global_slot(layer, f->slot);
        if (p->fill_ev[gs])
            HIP_OK(hipStreamWaitEvent(side, p->fill_ev[gs], 0));
        if (p->release_ev[gs])
            HIP_OK(hipStreamWaitEvent(side, p->release_ev[gs], 0));
    }
    for (size_t b = 0; b < fills.size(); b += GEN_BATCH) {
        GenBatch inval{}, pub{};
        const size_t e = std::min(fills.size(), b + GEN_BATCH);
        for (size_t i = b; i < e; ++i) {
            const FillRecord *f = &fills[i];
            const uint32_t gs = c.global_slot(layer, f->slot);
            inval.slot[inval.n] = gs;
            inval.value[inval.n++] = 0u;
            pub.slot[pub.n] = gs;
            pub.value[pub.n++] = f->gen;
        }
        HIP_OK(launch_set_gens(p->gen_dev, inval, side));
        // consecutive fills whose sources follow each other in one window and
        // whose slots follow each other in the pool (objects exactly one
        // stride long) go out as one copy: each copy costs the copy engine a
        // fixed setup time, about a sixth of a 6 MiB object's transfer
        for (size_t i = b; i < e;) {
            const FillRecord *f = &fills[i];
            const uint32_t gs = c.global_slot(layer, f->slot);
            uint8_t *dst = static_cast<uint8_t *>(p->desc.slot_pool) + uint64_t(gs) * p->desc.slot_stride;
            const uint8_t *src = static_cast<const uint8_t *>(p->windows[f->window]) + f->offset;
            uint64_t bytes = f->nbytes;
            size_t j = i + 1;
            while (j < e && f->nbytes == p->desc.slot_stride && fills[j].nbytes == f->nbytes &&
                   fills[j].window == f->window && fills[j].offset == f->offset + (j - i) * f->nbytes &&
                   c.global_slot(layer, fills[j].slot) == gs + (j - i)) {
                bytes += f->nbytes;
                ++j;
            }
            HIP_OK(hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, side));
            i = j;
        }
        HIP_OK(launch_set_gens(p->gen_dev, pub, side));
    }
    return MSI_OK;
}

// The per-expert arrays are always written; the per-row ones may be null
// for an empty batch (zero-length arrays).
bool routing_ok(const msi_routing &r, uint64_t T)
{
    return r.counts && r.offsets && r.demand &&
           (T == 0 || (r.idx && r.weights && r.perm && r.inv && r.row_weight));
}

RouteOut route_out(const msi_routing &r)
{
    return RouteOut{r.idx, r.weights, r.counts, r.offsets, r.demand, r.perm, r.inv, r.row_weight};
}

constexpr int ARRIVE_ROUTE = 0, ARRIVE_COMBINE = 32;   // words of arrive_dev, 128 bytes apart

// Wait for the combine of a direct forward to publish STATUS_DONE in the
// pinned word w.  The host spins on the word (no interrupt wake-up); every
// 256 polls it asks the stream, so a stream that failed, or finished without
// publishing, ends the wait with an error.
hipError_t wait_published(const uint32_t *w, hipStream_t s)
{
    for (uint32_t i = 1;; ++i) {
        if (__atomic_load_n(w, __ATOMIC_ACQUIRE) & STATUS_DONE)
            return hipSuccess;
        if ((i & 255u) == 0) {
            const hipError_t e = hipStreamQuery(s);
            if (e == hipSuccess)
                return (__atomic_load_n(w, __ATOMIC_ACQUIRE) & STATUS_DONE) ? hipSuccess : hipErrorUnknown;
            if (e != hipErrorNotReady)
                return e;
        }
        __builtin_ia32_pause();
    }
}

}  // namespace

extern "C" {

const char *msi_last_error(void) { return g_err.c_str(); }

uint32_t msi_abi_version(void) { return MSI_ABI_VERSION; }

uint32_t msi_stream_threshold(uint32_t v)
{
    if (v)
        g_stream_threshold = std::min<uint32_t>(v, 16u);
    return g_stream_threshold;
}

msi_status msi_plan_create(const msi_plan_desc *desc, msi_plan **out)
{
    if (!desc || !out)
        return fail(MSI_E_INVALID_ARG, "null argument");
    *out = nullptr;
    const uint64_t ob = object_bytes_of(*desc);
    // the source service first: its files' sizes bound the manifest's extents
    SourceService *src = nullptr;
    std::vector<uint64_t> fsizes;
    if (desc->source) {
        const msi_source_desc &sd = *desc->source;
        if (!sd.files || sd.n_files == 0 || !desc->windows || desc->n_windows == 0)
            return fail(MSI_E_INVALID_ARG, "a source needs files and staging windows");
        std::vector<std::string> files;
        for (uint32_t f = 0; f < sd.n_files; ++f) {
            if (!sd.files[f])
                return fail(MSI_E_INVALID_ARG, "null source file name");
            files.emplace_back(sd.files[f]);
        }
        std::vector<void *> wins;
        for (uint32_t w = 0; w < desc->n_windows; ++w)
            wins.push_back(const_cast<void *>(desc->windows[w]));
        src = new (std::nothrow) SourceService(files, wins, desc->window_bytes, sd.inflight, sd.align ? sd.align : 4096,
                                               (sd.flags & MSI_SOURCE_BUFFERED_OK) != 0);
        if (!src)
            return fail(MSI_E_NOMEM, "host allocation failed");
        if (!src->ok()) {
            const std::string m = src->error();
            delete src;
            return fail(MSI_E_INVALID_ARG, m);
        }
        for (uint32_t f = 0; f < sd.n_files; ++f)
            fsizes.push_back(src->file_size(f));
    }
    PlanCore *core = new (std::nothrow) PlanCore(*desc, ob, fsizes);
    if (!core) {
        delete src;
        return fail(MSI_E_NOMEM, "host allocation failed");
    }
    if (core->status() != MSI_OK) {
        const msi_status st = core->status();
        const std::string m = core->error();
        delete core;
        delete src;
        return fail(st, m);
    }
    if (src)
        for (uint32_t l = 0; l < desc->n_layers; ++l)
            for (uint32_t e = 0; e < desc->n_experts; ++e) {
                const SourceObject *so = core->source_object(l, e);
                uint64_t place[SourceService::MAX_EXTENTS];
                if (so && !src->layout(so->ext, so->n, place, nullptr)) {
                    delete core;
                    delete src;
                    return fail(MSI_E_INVALID_ARG, "window_bytes is smaller than the covering reads of (layer " +
                                                       std::to_string(l) + ", expert " + std::to_string(e) + ")");
                }
            }
    msi_plan *p = new (std::nothrow) msi_plan();
    if (!p) {
        delete core;
        delete src;
        return fail(MSI_E_NOMEM, "host allocation failed");
    }
    p->desc = *desc;
    p->windows.assign(desc->windows, desc->windows + desc->n_windows);
    p->desc.windows = nullptr;
    p->desc.objects = nullptr;
    p->desc.source = nullptr;
    p->object_bytes = ob;
    p->core = core;
    p->src = src;
    const size_t nslots = size_t(core->n_layers()) * core->pool_slots();
    p->fill_ev.assign(nslots, nullptr);
    p->fill_ev_id.assign(nslots, -1);
    p->release_ev.assign(nslots, nullptr);
    p->fill_ev_shared.assign(nslots, 0);
    p->table_cap = 2 * size_t(desc->n_experts) + 8;
    auto cleanup = [&](msi_status st, const std::string &m) {
        msi_plan_destroy(p);
        return fail(st, m);
    };
    if (hipGetDevice(&p->device) != hipSuccess)
        return cleanup(MSI_E_DEVICE, "no HIP device");
    if (init_kernel_attributes() != hipSuccess)
        return cleanup(MSI_E_DEVICE, "hipFuncSetAttribute failed");
    if (scratch_address(p->device, &p->scratch) != hipSuccess)
        return cleanup(MSI_E_DEVICE, "hipGetSymbolAddress of the static scratch failed");
    const size_t E = desc->n_experts, NL = desc->n_layers;
    p->res_version.assign(NL, 0);
    p->direct_ok.assign(NL, 0);
    if (hipMalloc(&p->gen_dev, nslots * sizeof(uint32_t)) != hipSuccess ||
        hipMalloc(&p->status_dev, sizeof(uint32_t) * (E + 64)) != hipSuccess ||
        hipMalloc(&p->res_slot_dev, sizeof(int32_t) * E * NL) != hipSuccess ||
        hipMalloc(&p->res_gen_dev, sizeof(uint32_t) * E * NL) != hipSuccess ||
        hipMalloc(&p->arrive_dev, 256) != hipSuccess ||
        hipMalloc(&p->dlist_dev, 4 * (E + 1) * sizeof(WorkItem)) != hipSuccess ||
        hipMalloc(&p->dcount_dev, 4 * sizeof(DevCount)) != hipSuccess ||
        hipMalloc(&p->table_dev, p->table_cap * sizeof(WorkItem)) != hipSuccess)
        return cleanup(MSI_E_DEVICE, "device allocation failed");
    if (hipHostMalloc(&p->table_host, p->table_cap * sizeof(WorkItem), hipHostMallocDefault) != hipSuccess ||
        hipHostMalloc(&p->counts_host, sizeof(int32_t) * desc->n_experts, hipHostMallocDefault) != hipSuccess ||
        hipHostMalloc(&p->status_host, 256, hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess ||
        hipHostMalloc(&p->res_host, sizeof(int32_t) * 2 * E, hipHostMallocDefault) != hipSuccess ||
        hipHostMalloc(&p->tail_host, sizeof(uint32_t) * (E + 2), hipHostMallocMapped | hipHostMallocCoherent) !=
            hipSuccess ||
        hipHostGetDevicePointer(reinterpret_cast<void **>(&p->tail_hdev), p->tail_host, 0) != hipSuccess ||
        hipHostGetDevicePointer(reinterpret_cast<void **>(&p->status_hdev), p->status_host, 0) != hipSuccess)
        return cleanup(MSI_E_DEVICE, "pinned host allocation failed");
    if (hipMemset(p->gen_dev, 0, nslots * sizeof(uint32_t)) != hipSuccess ||
        hipMemset(p->status_dev, 0, sizeof(uint32_t) * (E + 64)) != hipSuccess ||
        hipMemset(p->arrive_dev, 0, 256) != hipSuccess ||
        hipDeviceSynchronize() != hipSuccess)
        return cleanup(MSI_E_DEVICE, "device initialisation failed");
    *out = p;
    return MSI_OK;
}

msi_status msi_plan_destroy(msi_plan *p)
{
    if (!p)
        return MSI_OK;
    p->resolve_timings();
    if (p->src && p->core) {
        // shutdown drains the source: held reads are let go, every submitted
        // request completes and its window returns to Free
        p->src->release_holds();
        (void)source_until(p, [&] { return p->sfills.empty(); });
    }
    if (p->core) {
        for (uint32_t gs = 0; gs < p->fill_ev.size(); ++gs)
            if (p->fill_ev[gs]) {
                (void)hipEventSynchronize(p->fill_ev[gs]);
                observe_fill(p, gs);
            }
        if (p->core->any_holds()) {
            p->core->stats().rejections++;
            return fail(MSI_E_BUSY, "shutdown with a live held consumer");
        }
    }
    for (hipEvent_t e : p->all_events)
        (void)hipEventDestroy(e);
    if (p->gen_dev)
        (void)hipFree(p->gen_dev);
    if (p->status_dev)
        (void)hipFree(p->status_dev);
    if (p->table_dev)
        (void)hipFree(p->table_dev);
    if (p->res_slot_dev)
        (void)hipFree(p->res_slot_dev);
    if (p->res_gen_dev)
        (void)hipFree(p->res_gen_dev);
    if (p->arrive_dev)
        (void)hipFree(p->arrive_dev);
    if (p->dlist_dev)
        (void)hipFree(p->dlist_dev);
    if (p->dcount_dev)
        (void)hipFree(p->dcount_dev);
    if (p->res_host)
        (void)hipHostFree(p->res_host);
    if (p->tail_host)
        (void)hipHostFree(p->tail_host);
    if (p->table_host)
        (void)hipHostFree(p->table_host);
    if (p->counts_host)
        (void)hipHostFree(p->counts_host);
    if (p->status_host)
        (void)hipHostFree(p->status_host);
    delete p->src;
    delete p->core;
    delete p;
    return MSI_OK;
}

msi_status msi_plan_reset(msi_plan *p)
{
    if (!p)
        return fail(MSI_E_INVALID_ARG, "null plan");
    // fills not yet observed are outstanding work: their completions will be
    // judged against the new epoch and not published
    const msi_status st = p->core->reset();
    return st == MSI_OK ? st : fail(st, p->core->error());
}

msi_status msi_workspace_size(const msi_plan *p, uint32_t T, uint64_t *bytes)
{
    if (!p || !bytes)
        return fail(MSI_E_INVALID_ARG, "null argument");
    *bytes = workspace_layout(p->desc, T).total;
    return MSI_OK;
}

msi_status msi_plan_poll(msi_plan *p)
{
    if (!p)
        return fail(MSI_E_INVALID_ARG, "null plan");
    if (p->src) {
        HIP_OK(hipSetDevice(p->device));
        const msi_status st = source_progress(p, 0);
        if (st != MSI_OK && st != MSI_E_SHORT && st != MSI_E_IO && st != MSI_E_STALE)
            return st;
    }
    poll_fills(p);
    return MSI_OK;
}

msi_status msi_slot_fill(msi_plan *p, uint32_t layer, uint32_t expert, int32_t slot, void *side_stream,
                         msi_ticket *ticket)
{
    if (!p || !ticket)
        return fail(MSI_E_INVALID_ARG, "null argument");
    HIP_OK(hipSetDevice(p->device));
    poll_fills(p);
    int64_t id = -1;
    const msi_status st = p->core->request_fill(layer, expert, slot, ticket, &id);
    if (st != MSI_OK)
        return fail(st, p->core->error());
    if (ticket->hit)
        return MSI_OK;
    hipStream_t side = static_cast<hipStream_t>(side_stream);
    if (p->src) {
        // asynchronous: the read runs on the source's workers; the copy into
        // the slot is enqueued on `side` once the read completes (driven by
        // later calls on this plan)
        msi_plan::SrcFill f;
        f.rec = *p->core->fill(id);
        f.side = side;
        f.round = -1;
        p->sfills.push_back(f);
        const msi_status pst = source_progress(p, 0);
        return pst == MSI_OK || pst == MSI_E_SHORT || pst == MSI_E_IO || pst == MSI_E_STALE ? MSI_OK : pst;
    }
    const uint32_t gs = p->core->global_slot(layer, uint32_t(ticket->slot));
    const std::vector<FillRecord> fills{*p->core->fill(id)};
    msi_status est = enqueue_fills(p, layer, fills, side);
    if (est != MSI_OK)
        return est;
    // the superseded fill (if any) was accounted by the core; its event is
    // still waited on above, so release it now
    if (p->fill_ev[gs]) {
        if (!p->fill_ev_shared[gs])
            p->free_events.push_back(p->fill_ev[gs]);
        p->fill_ev[gs] = nullptr;
    }
    hipEvent_t ev = p->get_event();
    if (!ev)
        return fail(MSI_E_DEVICE, "event creation failed");
    HIP_OK(hipEventRecord(ev, side));
    p->fill_ev[gs] = ev;
    p->fill_ev_id[gs] = id;
    p->fill_ev_shared[gs] = 0;
    return MSI_OK;
}

msi_status msi_prefetch(msi_plan *p, uint32_t layer, const int32_t *experts, uint32_t n, void *side_stream,
                        uint32_t *issued)
{
    if (issued)
        *issued = 0;
    if (!p || (n && !experts))
        return fail(MSI_E_INVALID_ARG, "null argument");
    HIP_OK(hipSetDevice(p->device));
    poll_fills(p);
    std::vector<int64_t> ids;
    const msi_status st = p->core->request_prefetch(layer, std::vector<int32_t>(experts, experts + n), &ids);
    if (st != MSI_OK)
        return fail(st, p->core->error());
    hipStream_t side = static_cast<hipStream_t>(side_stream);
    if (p->src) {
        for (int64_t id : ids) {
            msi_plan::SrcFill f;
            f.rec = *p->core->fill(id);
            f.side = side;
            f.round = -1;
            p->sfills.push_back(f);
        }
        const msi_status pst = source_progress(p, 0);
        if (pst != MSI_OK && pst != MSI_E_SHORT && pst != MSI_E_IO && pst != MSI_E_STALE)
            return pst;
    } else if (!ids.empty()) {
        std::vector<FillRecord> fills;
        for (int64_t id : ids)
            fills.push_back(*p->core->fill(id));
        const msi_status est = enqueue_fills(p, layer, fills, side);
        if (est != MSI_OK)
            return est;
        // one owned event per filled slot, recorded after the whole batch
        for (const FillRecord &fr : fills) {
            const uint32_t gs = p->core->global_slot(layer, fr.slot);
            hipEvent_t ev = p->get_event();
            if (!ev)
                return fail(MSI_E_DEVICE, "event creation failed");
            HIP_OK(hipEventRecord(ev, side));
            if (p->fill_ev[gs] && !p->fill_ev_shared[gs])
                p->free_events.push_back(p->fill_ev[gs]);
            p->fill_ev[gs] = ev;
            p->fill_ev_id[gs] = fr.id;
            p->fill_ev_shared[gs] = 0;
        }
    }
    if (issued)
        *issued = uint32_t(ids.size());
    return MSI_OK;
}

msi_status msi_route(msi_plan *p, const msi_route_args *a, void *stream)
{
    if (!p || !a)
        return fail(MSI_E_INVALID_ARG, "null argument");
    const msi_plan_desc &d = p->desc;
    const int T = int(a->n_tokens), E = int(d.n_experts), K = int(d.top_k), D = int(d.d_model);
    const std::string lim = batch_limit_error(d, a->n_tokens);
    if (!lim.empty())
        return fail(MSI_E_INVALID_ARG, lim);
    if (!routing_ok(a->r, a->n_tokens) || (T > 0 && (!a->x || !a->w_router)))
        return fail(MSI_E_INVALID_ARG, "null routing or input pointer");
    const Workspace ws = workspace_layout(d, a->n_tokens);
    if (!a->workspace || a->workspace_bytes < ws.total)
        return fail(MSI_E_NOMEM, "workspace smaller than msi_workspace_size");
    HIP_OK(hipSetDevice(p->device));
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint8_t *wsb = static_cast<uint8_t *>(a->workspace);
    float *L = reinterpret_cast<float *>(wsb + ws.logits);
    const RouteOut o = route_out(a->r);
    if (T > 0) {
        if (d.wdtype == MSI_W_F32)
            HIP_OK(p->timed_launch(MSI_K_ROUTER_LOGITS, s, [&] {
                return launch_router_logits_f32(static_cast<const float *>(a->x),
                                                static_cast<const float *>(a->w_router), a->bias, L, T, D, E, s);
            }));
        else if (T <= 16) {
            // logits, selection and permutation in one launch
            HIP_OK(p->timed_launch(MSI_K_ROUTER_LOGITS, s, [&] {
                return launch_route_decode(static_cast<const uint16_t *>(a->x),
                                           static_cast<const uint16_t *>(a->w_router), a->bias, L,
                                           p->arrive_dev + ARRIVE_ROUTE, o, T, D, K, E, s);
            }));
            return MSI_OK;
        } else
            HIP_OK(p->timed_launch(MSI_K_ROUTER_LOGITS, s, [&] {
                return launch_router_logits_bf16(static_cast<const uint16_t *>(a->x),
                                                 static_cast<const uint16_t *>(a->w_router), a->bias, L, T, D, E, s);
            }));
    }
    HIP_OK(p->timed_launch(MSI_K_TOPK, s, [&] {
        return launch_route_select(L, o, reinterpret_cast<int32_t *>(wsb + ws.blockhist), T, K, E, s);
    }));
    return MSI_OK;
}

// Argument checks shared by both forward entry points (before any device work).
static msi_status forward_check(const msi_plan *p, const msi_forward_args *a)
{
    if (!p || !a)
        return fail(MSI_E_INVALID_ARG, "null argument");
    const msi_plan_desc &d = p->desc;
    if (a->layer >= d.n_layers)
        return fail(MSI_E_INVALID_ARG, "layer out of range");
    const std::string lim = batch_limit_error(d, a->n_tokens);
    if (!lim.empty())
        return fail(MSI_E_INVALID_ARG, lim);
    if (!routing_ok(a->r, a->n_tokens) || (a->n_tokens > 0 && (!a->x || !a->out)))
        return fail(MSI_E_INVALID_ARG, "null routing, input or output pointer");
    return MSI_OK;
}

// The forward itself; B holds the act / y scratch of T tokens (from the
// caller's workspace or the library's static scratch).
static msi_status forward_impl(msi_plan *p, const msi_forward_args *a, const FwdBufs &B, void *compute_stream,
                               void *side_stream)
{
    const msi_plan_desc &d = p->desc;
    PlanCore &core = *p->core;
    const int T = int(a->n_tokens), E = int(d.n_experts), K = int(d.top_k), D = int(d.d_model), I = int(d.d_ff);
    HIP_OK(hipSetDevice(p->device));
    hipStream_t cs = static_cast<hipStream_t>(compute_stream);
    hipStream_t side = static_cast<hipStream_t>(side_stream);
    poll_fills(p);

    // ---- layer entry, device work list: when the layer's last forward needed
    // no fill and every expert takes the stream path (T <= threshold), the
    // work list is built on the device from the counts and the published
    // residency table, with no host round trip before the expert launches.
    // A demanded expert without a published slot makes the attempt publish
    // nothing (STATUS_MISS) and the forward continues on the scheduled path.
    const bool f32w = d.wdtype == MSI_W_F32;
    if (!core.zero_cache() && !f32w && T > 0 && uint32_t(T) <= g_stream_threshold && p->direct_ok[a->layer]) {
        const uint32_t L0 = a->layer;
        if (p->res_version[L0] != core.layer_version(L0)) {
            core.published_map(L0, p->res_host, reinterpret_cast<uint32_t *>(p->res_host + E));
            HIP_OK(hipMemcpyAsync(p->res_slot_dev + size_t(L0) * E, p->res_host, sizeof(int32_t) * E,
                                  hipMemcpyHostToDevice, cs));
            HIP_OK(hipMemcpyAsync(p->res_gen_dev + size_t(L0) * E, p->res_host + E, sizeof(uint32_t) * E,
                                  hipMemcpyHostToDevice, cs));
            p->res_version[L0] = core.layer_version(L0);
        }
        const KernelSet &ks = kernel_set(d.wdtype);
        const int tpg = ks.tiles_gu_stream(1, D, I);
        const int tpd = ks.tiles_dn_stream(1, D, I);
        const int has_sh = a->shared_object ? 1 : 0;
        const int max_items = (std::min(E, T * K) + has_sh + 7) / 8 * 8;   // whole rounds of 8 items (XCDs)
        if (!p->status_clean)
            HIP_OK(launch_clear_word(p->status_dev, cs));
        p->status_clean = false;
        __atomic_store_n(&p->tail_host[0], 0u, __ATOMIC_RELAXED);   // the combine of this forward sets STATUS_DONE
        ExpertLaunch X{};
        X.x = a->x;
        X.perm = a->r.perm;
        X.wbase = static_cast<const uint8_t *>(d.slot_pool);
        X.wstride = d.slot_stride;
        X.gen_dev = p->gen_dev;
        X.status = p->status_dev;
        X.act = B.act;
        X.y = B.y;
        X.row_weight = a->r.row_weight;
        X.shared_w = static_cast<const uint8_t *>(a->shared_object);
        X.act_s = B.act_s;
        X.ys = B.ys;
        X.d = D;
        X.I = I;
        X.direct = DirectList{a->r.demand, p->res_slot_dev + size_t(L0) * E, p->res_gen_dev + size_t(L0) * E,
                              a->r.counts, a->r.offsets, has_sh, T, E};
        ExpertLaunch G = X, Dn = X;
        G.n_tiles = max_items * tpg;
        Dn.n_tiles = max_items * tpd;
        HIP_OK(p->timed_launch(MSI_K_GATEUP_STREAM, cs, [&] { return ks.gu_stream(G, cs); }));
        HIP_OK(p->timed_launch(MSI_K_DOWN_STREAM, cs, [&] { return ks.dn_stream(Dn, cs); }));
        const CombinePublish pub{p->status_dev, p->arrive_dev + ARRIVE_COMBINE, p->tail_hdev, a->r.demand};
        HIP_OK(p->timed_launch(MSI_K_COMBINE, cs, [&] {
            return launch_combine(B.y, has_sh ? B.ys : nullptr, false, a->r.inv, a->out, pub, T, K,
                                  D, cs);
        }));
        p->status_clean = true;
        // the combine publishes the status and the demanded experts straight
        // into tail_host once the expert kernels are done; the output rows it
        // is still writing are ordered before later work on the stream
        HIP_OK(wait_published(&p->tail_host[0], cs));
        const uint32_t st = __atomic_load_n(&p->tail_host[0], __ATOMIC_ACQUIRE);
        if (!(st & STATUS_MISS)) {
            const uint32_t n = std::min<uint32_t>(p->tail_host[1], uint32_t(E));
            std::vector<int32_t> dem(p->tail_host + 2, p->tail_host + 2 + n);
            if (st & STATUS_STALE) {
                core.stats().stale_detected++;
                core.stats().forwards++;
                core.invalidate_experts(L0, dem);
                p->direct_ok[L0] = 0;
                return fail(MSI_E_STALE, "a kernel saw a slot generation it did not expect; output not published");
            }
            core.note_direct_hits(L0, dem);
            return MSI_OK;
        }
        p->direct_ok[L0] = 0;       // a demanded expert was not resident: schedule it
    }

    // ---- layer entry, device-built work lists (T above the stream threshold):
    // when the layer's last forward needed no fill, a one-workgroup kernel
    // builds the four launch lists from the counts and the published
    // residency table and the expert kernels read their lengths on the
    // device (grids sized for the largest possible lists), so nothing waits
    // for the host between the routing and the combine.  A demanded expert
    // without a published slot makes the attempt publish nothing
    // (STATUS_MISS) and the forward continues on the scheduled path.
    if (!core.zero_cache() && !f32w && uint32_t(T) > g_stream_threshold && p->direct_ok[a->layer]) {
        const uint32_t L0 = a->layer;
        if (p->res_version[L0] != core.layer_version(L0)) {
            core.published_map(L0, p->res_host, reinterpret_cast<uint32_t *>(p->res_host + E));
            HIP_OK(hipMemcpyAsync(p->res_slot_dev + size_t(L0) * E, p->res_host, sizeof(int32_t) * E,
                                  hipMemcpyHostToDevice, cs));
            HIP_OK(hipMemcpyAsync(p->res_gen_dev + size_t(L0) * E, p->res_host + E, sizeof(uint32_t) * E,
                                  hipMemcpyHostToDevice, cs));
            p->res_version[L0] = core.layer_version(L0);
        }
        const KernelSet &ks = kernel_set(d.wdtype);
        const int thr = int(g_stream_threshold);
        const int has_sh = a->shared_object ? 1 : 0;
        WorklistArgs W{};
        W.counts = a->r.counts;
        W.offsets = a->r.offsets;
        W.slot_of = p->res_slot_dev + size_t(L0) * E;
        W.gen_of = p->res_gen_dev + size_t(L0) * E;
        W.status = p->status_dev;
        for (int k = 0; k < 4; ++k)
            W.items[k] = p->dlist_dev + size_t(k) * (E + 1);
        W.counts_out = p->dcount_dev;
        W.E = E;
        W.T = T;
        W.thr = thr;
        W.has_shared = has_sh;
        W.gu = ks.geom_gu(D, I);
        W.dn = ks.geom_dn(D, I);
        W.per_gu_stream = ks.tiles_gu_stream(1, D, I);
        W.per_dn_stream = ks.tiles_dn_stream(1, D, I);
        W.clear_status = p->status_clean ? 0 : 1;
        p->status_clean = false;
        __atomic_store_n(&p->tail_host[0], 0u, __ATOMIC_RELAXED);
        HIP_OK(p->timed_launch(MSI_K_PERMUTE, cs, [&] { return launch_build_worklist(W, cs); }));
        // grids for the largest lists this routing could give
        const int64_t rows = int64_t(T) * K;
        const int64_t n_tile_max = std::min<int64_t>(E, rows / (thr + 1));
        // (whole multiples of 8: each XCD's share of the real tiles must fit its workgroups)
        auto round8 = [](int64_t v) { return int((v + 7) / 8 * 8); };
        auto tile_ub = [&](TileGeom g) {
            return round8(((rows + g.rows - 1) / g.rows + n_tile_max + (has_sh ? (T + g.rows - 1) / g.rows : 0)) *
                          g.slices);
        };
        const int n_stream_max = int(std::min<int64_t>(E, rows));
        ExpertLaunch X{};
        X.x = a->x;
        X.perm = a->r.perm;
        X.wbase = static_cast<const uint8_t *>(d.slot_pool);
        X.wstride = d.slot_stride;
        X.gen_dev = p->gen_dev;
        X.status = p->status_dev;
        X.act = B.act;
        X.y = B.y;
        X.row_weight = a->r.row_weight;
        X.shared_w = static_cast<const uint8_t *>(a->shared_object);
        X.act_s = B.act_s;
        X.ys = B.ys;
        X.d = D;
        X.I = I;
        ExpertLaunch GT = X, DT = X, GS = X, DS = X;
        GT.items = W.items[0];
        GT.dev_n = p->dcount_dev + 0;
        GT.n_tiles = tile_ub(W.gu);
        DT.items = W.items[1];
        DT.dev_n = p->dcount_dev + 1;
        DT.n_tiles = tile_ub(W.dn);
        GS.items = W.items[2];
        GS.dev_n = p->dcount_dev + 2;
        GS.n_tiles = round8(int64_t(n_stream_max) * W.per_gu_stream);
        DS.items = W.items[3];
        DS.dev_n = p->dcount_dev + 3;
        DS.n_tiles = round8(int64_t(n_stream_max) * W.per_dn_stream);
        HIP_OK(p->timed_launch(MSI_K_GATEUP_TILE, cs, [&] { return ks.gu_tile(GT, cs); }));
        HIP_OK(p->timed_launch(MSI_K_GATEUP_STREAM, cs, [&] { return ks.gu_stream(GS, cs); }));
        HIP_OK(p->timed_launch(MSI_K_DOWN_TILE, cs, [&] { return ks.dn_tile(DT, cs); }));
        HIP_OK(p->timed_launch(MSI_K_DOWN_STREAM, cs, [&] { return ks.dn_stream(DS, cs); }));
        // large grid: no arrival counter (the next forward clears the status word)
        const CombinePublish pub{p->status_dev, nullptr, p->tail_hdev, a->r.demand};
        HIP_OK(p->timed_launch(MSI_K_COMBINE, cs, [&] {
            return launch_combine(B.y, has_sh ? B.ys : nullptr, false, a->r.inv, a->out, pub, T, K, D, cs);
        }));
        HIP_OK(wait_published(&p->tail_host[0], cs));
        const uint32_t st = __atomic_load_n(&p->tail_host[0], __ATOMIC_ACQUIRE);
        if (!(st & STATUS_MISS)) {
            const uint32_t n = std::min<uint32_t>(p->tail_host[1], uint32_t(E));
            std::vector<int32_t> dem(p->tail_host + 2, p->tail_host + 2 + n);
            if (st & STATUS_STALE) {
                core.stats().stale_detected++;
                core.stats().forwards++;
                core.invalidate_experts(L0, dem);
                p->direct_ok[L0] = 0;
                return fail(MSI_E_STALE, "a kernel saw a slot generation it did not expect; output not published");
            }
            core.note_direct_hits(L0, dem);
            return MSI_OK;
        }
        p->direct_ok[L0] = 0;       // a demanded expert was not resident: schedule it
        HIP_OK(hipStreamSynchronize(cs));
    }

    // ---- layer entry: the demanded set (one device-to-host read of the counts)
    HIP_OK(hipMemcpyAsync(p->counts_host, a->r.counts, sizeof(int32_t) * E, hipMemcpyDeviceToHost, cs));
    HIP_OK(hipStreamSynchronize(cs));
    std::vector<int32_t> demanded;
    std::vector<int32_t> counts(p->counts_host, p->counts_host + E);
    std::vector<int32_t> offsets(E + 1, 0);
    for (int e = 0; e < E; ++e) {
        if (counts[e] < 0 || counts[e] > T)
            return fail(MSI_E_INVALID_ARG, "routing counts out of range");
        offsets[e + 1] = offsets[e] + counts[e];
        if (counts[e] > 0)
            demanded.push_back(e);
    }
    if (offsets[E] != T * K)
        return fail(MSI_E_INVALID_ARG, "routing counts do not sum to T * K");

    Schedule sched;
    const msi_status sst = core.schedule_forward(a->layer, demanded, &sched);
    if (sst != MSI_OK)
        return fail(sst, core.error());

    // ---- work tables: per round, gate/up and down launches of each path
    enum Kind { GU_TILE, GU_STREAM, DN_TILE, DN_STREAM, NKIND };
    struct Launch {
        int kind;
        size_t off;
        int n_items;
        int n_tiles;
    };
    std::vector<std::vector<Launch>> launches(sched.rounds.size());
    std::vector<WorkItem> table;
    const bool f32 = d.wdtype == MSI_W_F32;
    const KernelSet &ks = kernel_set(d.wdtype);
    auto add_launch = [&](size_t r, int kind, const std::vector<WorkItem> &items) {
        if (items.empty())
            return;
        Launch l{kind, table.size(), int(items.size()), 0};
        int tiles = 0;
        for (WorkItem w : items) {
            int n;
            switch (kind) {
            case GU_TILE: n = ks.tiles_gu_tile(w.nrows, D, I); break;
            case GU_STREAM: n = ks.tiles_gu_stream(w.nrows, D, I); break;
            case DN_TILE: n = ks.tiles_dn_tile(w.nrows, D, I); break;
            default: n = ks.tiles_dn_stream(w.nrows, D, I); break;
            }
            w.tile0 = tiles;
            tiles += n;
            table.push_back(w);
        }
        l.n_tiles = tiles;
        launches[r].push_back(l);
    };
    const uint32_t thr = g_stream_threshold;
    const bool has_shared = a->shared_object && T > 0;
    if (has_shared && sched.rounds.empty())
        launches.emplace_back();
    for (size_t r = 0; r < launches.size(); ++r) {
        std::vector<WorkItem> tile_items, stream_items;
        if (r == 0 && has_shared)   // the shared expert rides in the first round's launches
            (f32 || uint32_t(T) > thr ? tile_items : stream_items).push_back(WorkItem{-1, -1, 0u, 0, T, 0});
        const std::vector<SchedItem> none;
        for (const SchedItem &si : r < sched.rounds.size() ? sched.rounds[r].items : none) {
            WorkItem w{si.expert, int32_t(core.global_slot(a->layer, uint32_t(si.slot))), si.gen, offsets[si.expert],
                       counts[si.expert], 0};
            (f32 || uint32_t(w.nrows) > thr ? tile_items : stream_items).push_back(w);
        }
        add_launch(r, GU_TILE, tile_items);
        add_launch(r, GU_STREAM, stream_items);      // (empty for f32 layers)
        add_launch(r, DN_TILE, tile_items);
        add_launch(r, DN_STREAM, stream_items);
    }
    if (table.size() > p->table_cap)
        return fail(MSI_E_INVALID_ARG, "internal: schedule table overflow");
    if (!table.empty()) {
        std::memcpy(p->table_host, table.data(), table.size() * sizeof(WorkItem));
        HIP_OK(hipMemcpyAsync(p->table_dev, p->table_host, table.size() * sizeof(WorkItem), hipMemcpyHostToDevice,
                              cs));
    }
    if (!p->status_clean)
        HIP_OK(launch_clear_word(p->status_dev, cs));
    p->status_clean = false;            // set again below once the word is read back as zero

    // ---- rounds: fills on the side stream, kernels on the compute stream
    std::vector<hipEvent_t> round_events;
    auto new_event = [&]() -> hipEvent_t {
        hipEvent_t e = p->get_event();
        if (e)
            round_events.push_back(e);
        return e;
    };
    msi_status rst = MSI_OK;
    if (p->src) {
        // source-backed: earlier explicit fills first (rounds may count them
        // as hits), then every round's misses go to the source at once, in
        // round order (reads run as staging windows allow); a round's copies
        // into its slots are enqueued when the loop below reaches it
        rst = source_until(p, [&] {
            for (const msi_plan::SrcFill &f : p->sfills)
                if (f.round < 0 && f.state <= SF_READY)
                    return false;
            return true;
        });
        for (size_t r = 0; r < sched.rounds.size(); ++r)
            for (const FillRecord &fr : sched.rounds[r].fills) {
                msi_plan::SrcFill f;
                f.rec = fr;
                f.side = side;
                f.round = int(r);
                p->sfills.push_back(f);
            }
    }
    auto round_copied = [&](const SchedRound &round) {
        for (const FillRecord &fr : round.fills)
            for (const msi_plan::SrcFill &f : p->sfills)
                if (f.rec.id == fr.id && f.round >= 0 && f.state < SF_COPYING)
                    return false;
        return true;
    };
    for (size_t r = 0; r < launches.size() && rst == MSI_OK; ++r) {
        if (r < sched.rounds.size() && p->src) {
            const SchedRound &round = sched.rounds[r];
            p->src_round = int(r);
            rst = source_until(p, [&] { return round_copied(round); });
            if (rst != MSI_OK)
                break;
            // the copies set each filled slot's pending event; the kernels wait on them below
            for (const SchedItem &si : round.items) {
                const uint32_t gs = core.global_slot(a->layer, uint32_t(si.slot));
                if (p->fill_ev[gs])
                    HIP_OK(hipStreamWaitEvent(cs, p->fill_ev[gs], 0));
            }
        } else if (r < sched.rounds.size()) {
            const SchedRound &round = sched.rounds[r];
            if (!round.fills.empty()) {
                msi_status fst = MSI_OK;
                const hipError_t fe_ = p->timed_copy(MSI_K_FILL, side, [&] {
                    fst = enqueue_fills(p, a->layer, round.fills, side);
                    return fst == MSI_OK ? hipSuccess : hipErrorUnknown;
                });
                rst = fst != MSI_OK ? fst : (fe_ != hipSuccess ? fail(MSI_E_DEVICE, "fill timing event") : MSI_OK);
                if (rst != MSI_OK)
                    break;
                hipEvent_t fe = new_event();
                if (!fe) {
                    rst = fail(MSI_E_DEVICE, "event creation failed");
                    break;
                }
                HIP_OK(hipEventRecord(fe, side));
                for (const FillRecord &f : round.fills) {
                    const uint32_t gs = core.global_slot(a->layer, f.slot);
                    if (p->fill_ev[gs] && !p->fill_ev_shared[gs])
                        p->free_events.push_back(p->fill_ev[gs]);
                    p->fill_ev[gs] = fe;
                    p->fill_ev_id[gs] = f.id;
                    p->fill_ev_shared[gs] = 1;
                }
            }
            // hits whose fill (an earlier explicit request) is still pending
            for (const SchedItem &si : round.items) {
                const uint32_t gs = core.global_slot(a->layer, uint32_t(si.slot));
                if (p->fill_ev[gs])
                    HIP_OK(hipStreamWaitEvent(cs, p->fill_ev[gs], 0));
            }
        }
        for (const Launch &l : launches[r]) {
            ExpertLaunch L{};
            L.items = p->table_dev + l.off;
            L.n_items = l.n_items;
            L.n_tiles = l.n_tiles;
            L.x = a->x;
            L.gen_dev = p->gen_dev;
            L.status = p->status_dev;
            L.d = D;
            L.I = I;
            L.perm = a->r.perm;
            L.wbase = static_cast<const uint8_t *>(d.slot_pool);
            L.wstride = d.slot_stride;
            L.act = B.act;
            L.y = B.y;
            L.row_weight = a->r.row_weight;
            L.shared_w = static_cast<const uint8_t *>(a->shared_object);
            L.act_s = B.act_s;
            L.ys = B.ys;
            static const int tkind[NKIND] = {MSI_K_GATEUP_TILE, MSI_K_GATEUP_STREAM, MSI_K_DOWN_TILE,
                                             MSI_K_DOWN_STREAM};
            const hipError_t e = p->timed_launch(f32 ? MSI_K_EXPERT_F32 : tkind[l.kind], cs, [&] {
                switch (l.kind) {
                case GU_TILE: return ks.gu_tile(L, cs);
                case GU_STREAM: return ks.gu_stream(L, cs);
                case DN_TILE: return ks.dn_tile(L, cs);
                default: return ks.dn_stream(L, cs);
                }
            });
            if (e != hipSuccess) {
                rst = fail(MSI_E_DEVICE, std::string("expert kernel launch: ") + hipGetErrorString(e));
                break;
            }
        }
        if (rst != MSI_OK)
            break;
        if (r < sched.rounds.size()) {
            hipEvent_t re = new_event();
            if (!re) {
                rst = fail(MSI_E_DEVICE, "event creation failed");
                break;
            }
            HIP_OK(hipEventRecord(re, cs));
            for (const SchedItem &si : sched.rounds[r].items)
                p->release_ev[core.global_slot(a->layer, uint32_t(si.slot))] = re;
        }
    }

    // ---- publication: out written only if every tile saw its generation; the
    // combine publishes the status word to status_host (also when T == 0)
    *p->status_host = 0u;
    if (rst == MSI_OK) {
        // no arrival counter: one counter update per workgroup of a large grid costs more than the clear
        const CombinePublish pub{p->status_dev, nullptr, p->status_hdev, nullptr};
        if (p->timed_launch(MSI_K_COMBINE, cs, [&] {
                return launch_combine(B.y, has_shared ? B.ys : nullptr, f32w, a->r.inv,
                                      a->out, pub, T, K, D, cs);
            }) != hipSuccess)
            rst = fail(MSI_E_DEVICE, "combine launch failed");
    }
    const hipError_t se = hipStreamSynchronize(cs);
    (void)hipStreamSynchronize(side);
    if (se != hipSuccess && rst == MSI_OK)
        rst = fail(MSI_E_DEVICE, std::string("compute stream: ") + hipGetErrorString(se));
    // the device word still holds what the combine read: clean if that was zero
    const uint32_t hst = __atomic_load_n(p->status_host, __ATOMIC_ACQUIRE);
    p->status_clean = rst == MSI_OK && hst == STATUS_DONE;

    if (p->src) {
        p->src_round = -1;
        if (rst != MSI_OK)
            source_cancel_forward(p);     // nothing more of this forward is copied; reads drain
        (void)source_progress(p, 0);      // finished copies free their windows
    }
    // ---- layer exit: observe this forward's fills, release consumers
    for (const SchedRound &round : sched.rounds)
        for (const FillRecord &f : round.fills) {
            if (!core.fill(f.id))
                continue;      // superseded by a later round of this forward
            const uint32_t gs = core.global_slot(a->layer, f.slot);
            if (p->fill_ev_id[gs] == f.id)
                observe_fill(p, gs);
            else
                core.complete_fill(f.id);
        }
    for (const SchedRound &round : sched.rounds)
        for (const SchedItem &si : round.items)
            p->release_ev[core.global_slot(a->layer, uint32_t(si.slot))] = nullptr;
    for (hipEvent_t e : round_events)
        p->free_events.push_back(e);
    core.end_forward(a->layer, sched);
    {
        bool filled = false;
        for (const SchedRound &round : sched.rounds)
            filled |= !round.fills.empty();
        p->direct_ok[a->layer] = filled ? 0 : 1;
    }
    if (rst != MSI_OK)
        return rst;
    if (hst & STATUS_STALE) {
        core.stats().stale_detected++;
        core.invalidate_read_slots(a->layer, sched);
        p->direct_ok[a->layer] = 0;
        return fail(MSI_E_STALE, "a kernel saw a slot generation it did not expect; output not published");
    }
    return MSI_OK;
}

msi_status msi_moe_forward(msi_plan *p, const msi_forward_args *a, void *compute_stream, void *side_stream)
{
    const msi_status st = forward_check(p, a);
    if (st != MSI_OK)
        return st;
    const Workspace ws = workspace_layout(p->desc, a->n_tokens);
    if (!a->workspace || a->workspace_bytes < ws.total)
        return fail(MSI_E_NOMEM, "workspace smaller than msi_workspace_size");
    uint8_t *w = static_cast<uint8_t *>(a->workspace);
    return forward_impl(p, a, FwdBufs{w + ws.act, w + ws.act_s, w + ws.y, w + ws.ys}, compute_stream, side_stream);
}

msi_status msi_moe_forward_noalloc(msi_plan *p, const msi_forward_args *a, void *compute_stream, void *side_stream)
{
    const msi_status st = forward_check(p, a);
    if (st != MSI_OK)
        return st;
    if (a->workspace || a->workspace_bytes)
        return fail(MSI_E_INVALID_ARG, "msi_moe_forward_noalloc takes no workspace (workspace must be NULL and "
                                       "workspace_bytes 0)");
    const Workspace ws = workspace_layout(p->desc, a->n_tokens);
    const uint64_t need = ws.total - ws.act;     // act, shared act, y, shared y
    if (need > MSI_NOALLOC_SCRATCH_BYTES)
        return fail(MSI_E_INVALID_ARG, "forward of " + std::to_string(a->n_tokens) + " tokens needs " +
                                           std::to_string(need) + " bytes of scratch, above the " +
                                           std::to_string(uint64_t(MSI_NOALLOC_SCRATCH_BYTES)) +
                                           " bytes of msi_moe_forward_noalloc");
    uint8_t *base = static_cast<uint8_t *>(p->scratch);
    if (!base)
        return fail(MSI_E_DEVICE, "static scratch address unknown for this device");
    return forward_impl(p, a,
                        FwdBufs{base, base + (ws.act_s - ws.act), base + (ws.y - ws.act), base + (ws.ys - ws.act)},
                        compute_stream, side_stream);
}

msi_status msi_slot_hold(msi_plan *p, uint32_t layer, uint32_t slot)
{
    if (!p)
        return fail(MSI_E_INVALID_ARG, "null plan");
    const msi_status st = p->core->hold(layer, slot);
    return st == MSI_OK ? st : fail(st, p->core->error());
}

msi_status msi_slot_unhold(msi_plan *p, uint32_t layer, uint32_t slot)
{
    if (!p)
        return fail(MSI_E_INVALID_ARG, "null plan");
    const msi_status st = p->core->unhold(layer, slot);
    return st == MSI_OK ? st : fail(st, p->core->error());
}

msi_status msi_slot_query(const msi_plan *p, uint32_t layer, uint32_t slot, msi_slot_info *info)
{
    if (!p || !info)
        return fail(MSI_E_INVALID_ARG, "null argument");
    if (layer >= p->core->n_layers() || slot >= p->core->pool_slots())
        return fail(MSI_E_INVALID_ARG, "layer or slot out of range");
    const Slot &s = p->core->slot(layer, slot);
    *info = msi_slot_info{uint32_t(s.state), s.expert, s.gen, s.epoch, s.consumers + s.holds, s.holds, s.last_use};
    return MSI_OK;
}

msi_status msi_plan_stats(const msi_plan *p, msi_stats *st)
{
    if (!p || !st)
        return fail(MSI_E_INVALID_ARG, "null argument");
    *st = p->core->stats();
    st->fills_in_flight = p->core->fills_in_flight();
    st->windows_busy = p->src ? p->src->busy_windows() : p->core->windows_busy();
    st->consumers_live = p->core->consumers_live();
    st->epoch = p->core->epoch();
    return MSI_OK;
}

msi_status msi_plan_set_timing(msi_plan *p, int enable)
{
    if (!p)
        return fail(MSI_E_INVALID_ARG, "null plan");
    p->timing = enable != 0;
    p->timing_mask = enable == 1 ? ~0u : uint32_t(enable);
    return MSI_OK;
}

msi_status msi_plan_set_timing_period(msi_plan *p, uint32_t period)
{
    if (!p || period == 0)
        return fail(MSI_E_INVALID_ARG, "null plan or zero period");
    p->timing_period = period;
    for (uint64_t &c : p->timing_seen)
        c = 0;
    return MSI_OK;
}

msi_status msi_plan_timings(msi_plan *p, msi_timings *out, int reset)
{
    if (!p || !out)
        return fail(MSI_E_INVALID_ARG, "null argument");
    HIP_OK(hipSetDevice(p->device));
    p->resolve_timings();
    for (int k = 0; k < MSI_NKERN; ++k) {
        out->launches[k] = p->t_launches[k];
        out->ms[k] = p->t_ms[k];
        if (reset) {
            p->t_launches[k] = 0;
            p->t_ms[k] = 0.0;
        }
    }
    return MSI_OK;
}

msi_status msi_residual_init(const uint16_t *x0, float *h, uint16_t *x, uint32_t rows, uint32_t cols,
                             void *stream)
{
    if (uint64_t(rows) * cols && (!x0 || !h || !x))
        return fail(MSI_E_INVALID_ARG, "null pointer");
    HIP_OK(launch_residual(x0, nullptr, h, x, int(rows), int(cols), static_cast<hipStream_t>(stream)));
    return MSI_OK;
}

msi_status msi_residual_add(const float *out, float *h, uint16_t *x, uint32_t rows, uint32_t cols, void *stream)
{
    if (uint64_t(rows) * cols && (!out || !h || !x))
        return fail(MSI_E_INVALID_ARG, "null pointer");
    HIP_OK(launch_residual(nullptr, out, h, x, int(rows), int(cols), static_cast<hipStream_t>(stream)));
    return MSI_OK;
}

msi_status msi_source_stats_get(const msi_plan *p, msi_source_stats *st)
{
    if (!p || !st)
        return fail(MSI_E_INVALID_ARG, "null argument");
    *st = msi_source_stats{};
    if (!p->src)
        return MSI_OK;
    const SourceStats s = p->src->stats();
    *st = msi_source_stats{s.reads_issued, s.reads_completed, s.reads_failed, s.requests, s.requests_ready,
                           s.requests_failed, s.requests_stale, s.logical_bytes, s.physical_bytes, s.padding_bytes,
                           s.peak_depth, p->src->busy_windows(), s.read_seconds, p->src_wait_s, s.direct, s.buffered,
                           s.bounced};
    return MSI_OK;
}

msi_status msi_debug_source_fault(msi_plan *p, uint32_t layer, uint32_t expert, uint32_t component, uint32_t mode)
{
    if (!p || !p->src)
        return fail(MSI_E_INVALID_ARG, "null plan or plan without a source");
    const SourceObject *so = p->core->source_object(layer, expert);
    if (!so || component >= uint32_t(so->n) || mode < MSI_FAULT_SHORT || mode > MSI_FAULT_HOLD)
        return fail(MSI_E_INVALID_ARG, "no such source object / component, or unknown fault mode");
    p->src_faults.push_back(msi_plan::FaultReq{layer, expert, component, mode});
    return MSI_OK;
}

msi_status msi_debug_source_release(msi_plan *p)
{
    if (!p || !p->src)
        return fail(MSI_E_INVALID_ARG, "null plan or plan without a source");
    p->src->release_holds();
    return MSI_OK;
}

msi_status msi_debug_set_device_gen(msi_plan *p, uint32_t layer, uint32_t slot, uint32_t gen)
{
    if (!p)
        return fail(MSI_E_INVALID_ARG, "null plan");
    if (layer >= p->core->n_layers() || slot >= p->core->pool_slots())
        return fail(MSI_E_INVALID_ARG, "layer or slot out of range");
    HIP_OK(hipSetDevice(p->device));
    HIP_OK(hipDeviceSynchronize());
    HIP_OK(hipMemcpy(p->gen_dev + p->core->global_slot(layer, slot), &gen, sizeof(uint32_t), hipMemcpyHostToDevice));
    return MSI_OK;
}

}  // extern "C"
