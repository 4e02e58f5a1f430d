// plan_core.hpp -- host-side residency planner of the slot-backed MoE layer.
//
// Pure C++17, no HIP: the HIP layer (msi_abi.cpp) owns events, streams and
// device memory and drives this class with explicit calls.  It holds the
// immutable manifest and the mutable per-slot / per-window state of the
// paper's Plan ("A Shared Cross-Adapter Plan Core": object, generation, request epoch, readiness,
// live-consumer count; replacement policy kept apart from the lifecycle) and
// the GPU-slot state sequence Vacant -> Loading -> DeviceReady -> InUse ->
// Recyclable -> Vacant of "Separate Window and GPU-Slot Lifecycles", with tickets carrying object,
// generation, epoch and slot.  Host windows are caller-owned pinned buffers
// that always hold their extents, so of the window sequence only
// HostReady <-> Copying is tracked (a window is busy while a copy reads it).
#pragma once

#include <cstdint>
#include <string>
#include <unordered_map>
#include <vector>

#include "../../include/msi.h"
#include "source.hpp"

namespace msi {

enum class SlotState : uint32_t {
    Vacant = MSI_SLOT_VACANT,
    Loading = MSI_SLOT_LOADING,
    DeviceReady = MSI_SLOT_DEVICE_READY,
    InUse = MSI_SLOT_IN_USE,
    Recyclable = MSI_SLOT_RECYCLABLE,
};

struct Slot {
    SlotState state = SlotState::Vacant;
    int32_t expert = -1;       // object currently denoted (or being loaded)
    uint32_t gen = 0;          // generation of that version; bumps on every fill
    uint32_t epoch = 0;        // epoch of the fill that produced it
    uint32_t consumers = 0;    // live consumers from forward rounds
    uint32_t holds = 0;        // consumers held through the API
    uint64_t last_use = 0;     // LRU tick
    int64_t fill_id = -1;      // unobserved fill targeting this slot, -1 if none
    bool prot = false;         // protected segment (protected LRU)
    bool prefetched = false;   // filled by a prefetch and not used yet
};

struct FillRecord {
    int64_t id = -1;
    uint32_t layer = 0, slot = 0, expert = 0, gen = 0, epoch = 0, window = 0;
    uint64_t offset = 0, nbytes = 0;
    bool consumed = false;     // a forward round reads this version (stream-ordered)
};

struct SchedItem {
    int32_t expert;
    int32_t slot;      // index within the layer's pool
    uint32_t gen;      // generation the kernels must see
};

struct SchedRound {
    std::vector<SchedItem> items;     // ascending by position in the demand order
    std::vector<FillRecord> fills;    // copies of the fills submitted for this round
                                      // (a later round may supersede the core's record)
};

struct Schedule {
    std::vector<SchedRound> rounds;
};

// Batch-size limit of a plan's kernels: "" if T tokens are addressable, else
// why not.  The tile kernels gather token rows of x through 32-bit byte
// offsets from the start of x, so T * d_model * (element bytes) must stay
// below 2^31 for bf16 and 4-bit layers; every layer keeps T <= 2^24.
std::string batch_limit_error(const msi_plan_desc &d, uint64_t n_tokens);

// window of an object that the source service reads from canonical files
constexpr uint32_t SOURCE_WINDOW = 0xFFFFFFFFu;

struct ObjectInfo {
    uint32_t window;           // SOURCE_WINDOW: read from its extents
    uint64_t offset, nbytes;
};

// Extents of a source-backed object, in component order.
struct SourceObject {
    int n = 0;
    SourceExtent ext[SourceService::MAX_EXTENTS];
};

class PlanCore {
public:
    // Validates the manifest; on failure status() != MSI_OK and error() says
    // why.  file_sizes: sizes of the source's files (plans with a source).
    PlanCore(const msi_plan_desc &d, uint64_t object_bytes, const std::vector<uint64_t> &file_sizes = {});

    msi_status status() const { return status_; }
    const std::string &error() const { return err_; }

    uint32_t n_layers() const { return n_layers_; }
    uint32_t n_experts() const { return n_experts_; }
    uint32_t pool_slots() const { return pool_slots_; }
    bool zero_cache() const { return zero_cache_; }
    uint32_t epoch() const { return epoch_; }
    const msi_stats &stats() const { return stats_; }
    msi_stats &stats() { return stats_; }

    const Slot &slot(uint32_t layer, uint32_t s) const { return slots_[layer * pool_slots_ + s]; }
    Slot &slot(uint32_t layer, uint32_t s) { return slots_[layer * pool_slots_ + s]; }
    uint32_t global_slot(uint32_t layer, uint32_t s) const { return layer * pool_slots_ + s; }
    const ObjectInfo *object(uint32_t layer, uint32_t expert) const;
    const SourceObject *source_object(uint32_t layer, uint32_t expert) const;
    bool source_backed() const { return source_backed_; }
    const FillRecord *fill(int64_t id) const;
    // True while fill `id` is the slot's current, same-epoch version (a source
    // completion carrying this ticket may still be published).
    bool fill_current(int64_t id, uint32_t epoch, uint32_t gen) const;

    // Slot holding a published (or same-epoch loading) version of the object,
    // usable as a hit; -1 if none.  Zero-cache plans never report hits.
    int32_t resident_slot(uint32_t layer, uint32_t expert) const;

    // Victim among the demand bank's slots of `layer` (all slots without a
    // prefetch bank) that have no holds and are not in `exclude` (one flag
    // per pool slot), by the plan's policy; -1 if none.  prefetch: choose in
    // the prefetch bank instead (least recently used).
    int32_t choose_victim(uint32_t layer, const std::vector<uint8_t> &exclude, bool prefetch = false) const;
    uint32_t demand_slots() const { return pool_slots_ - prefetch_slots_; }
    bool in_prefetch_bank(uint32_t s) const { return s >= pool_slots_ - prefetch_slots_; }

    // Prefetch (msi_prefetch): fills for the listed experts not resident or
    // loading, into the prefetch bank, at most its size.  Fill ids in *ids.
    msi_status request_prefetch(uint32_t layer, const std::vector<int32_t> &experts, std::vector<int64_t> *ids);

    // Explicit fill (msi_slot_fill).  On MSI_OK *t is the ticket and, unless
    // t->hit, *fill_id the new fill to submit.
    msi_status request_fill(uint32_t layer, uint32_t expert, int32_t forced_slot, msi_ticket *t,
                            int64_t *fill_id);

    // Completion of a submitted fill observed by the device layer.
    void complete_fill(int64_t fill_id);
    // A fill whose source request failed (short read, EIO, stale ticket):
    // never published; its slot goes Vacant.
    void fail_fill(int64_t fill_id);

    // Resolve the demanded experts (ascending ids) of one forward into
    // rounds: hits first, then misses in ascending id; rounds hold at most
    // the pool size (half of it when there are several, so the next round's
    // fills go to slots the current round does not read).  Submits the fills
    // and takes one consumer per round item.  MSI_E_BUSY if no victim exists.
    msi_status schedule_forward(uint32_t layer, const std::vector<int32_t> &demanded, Schedule *out);

    // Drop the consumers a schedule took (after its kernels completed).
    // Zero-cache plans then forget every object they loaded.
    void end_forward(uint32_t layer, const Schedule &s);

    // After a forward that saw a stale generation: every slot it read is
    // suspect, so none of them stays published (the next use refills).
    void invalidate_read_slots(uint32_t layer, const Schedule &s);

    msi_status hold(uint32_t layer, uint32_t s);
    msi_status unhold(uint32_t layer, uint32_t s);
    msi_status reset();                        // epoch++ (MSI_E_BUSY with holds)
    bool any_holds() const;
    uint64_t fills_in_flight() const;
    uint64_t windows_busy() const;
    uint64_t consumers_live() const;

    void set_error(msi_status st, const std::string &msg) { status_ = st; err_ = msg; }

    // Bumped whenever a slot of the layer changes what it publishes.
    uint64_t layer_version(uint32_t layer) const { return layer_version_[layer]; }
    // Published (expert -> global slot, generation) of a layer: slot -1 when
    // the expert has no published version (Loading versions are excluded).
    void published_map(uint32_t layer, int32_t *slot_of, uint32_t *gen_of) const;
    // A forward served entirely by published slots: count the hits and
    // refresh the LRU ticks of the demanded experts' slots.
    void note_direct_hits(uint32_t layer, const std::vector<int32_t> &demanded);
    // After a stale generation seen on published slots: forget the listed
    // experts' versions (the next use refills).
    void invalidate_experts(uint32_t layer, const std::vector<int32_t> &experts);

private:
    int64_t new_fill(uint32_t layer, uint32_t s, uint32_t expert);
    void publish_state(Slot &sl);
    void touch(uint32_t layer, uint32_t s);    // a use: LRU tick, protection, prefetch accounting

    msi_status status_ = MSI_OK;
    std::string err_;
    uint32_t n_layers_ = 0, n_experts_ = 0, pool_slots_ = 0, prefetch_slots_ = 0;
    uint32_t policy_ = MSI_POLICY_LRU;
    bool zero_cache_ = false;
    uint32_t epoch_ = 0;
    uint64_t tick_ = 0;
    std::vector<Slot> slots_;
    std::vector<ObjectInfo> objects_;          // [layer * E + expert]
    std::vector<uint8_t> has_object_;
    std::vector<SourceObject> src_;            // [layer * E + expert], source-backed plans
    bool source_backed_ = false;
    std::vector<uint32_t> window_busy_;
    std::unordered_map<int64_t, FillRecord> fills_;   // unobserved fills
    std::vector<uint64_t> layer_version_;
    // resident_slot lookup table per layer ([layer * E + expert] -> first
    // qualifying slot), rebuilt when the layer's version or the epoch moved
    mutable std::vector<int32_t> res_index_;
    mutable std::vector<uint64_t> res_index_version_;   // 0: never built
    mutable std::vector<uint32_t> res_index_epoch_;
    void rebuild_res_index(uint32_t layer) const;
    int64_t next_fill_ = 0;
    msi_stats stats_{};
};

}  // namespace msi
