// plan_core.cpp -- residency planner: manifest checks, slot lifecycle,
// generations and epochs, LRU / zero-cache policies, forward round schedule.
// The paper's Design section: "A Shared Cross-Adapter Plan Core" (manifest
// and mutable state), "Bounded Source Service" (extent rejection
// conditions), "Stable Slots and Bundle Publication", "Separate Window and
// GPU-Slot Lifecycles" (state sequences, tickets, reset); Implementation,
// "Scheduling and copies".
#include "plan_core.hpp"

#include <algorithm>
#include <limits>

namespace msi {

std::string batch_limit_error(const msi_plan_desc &d, uint64_t n_tokens)
{
    if (n_tokens > (uint64_t(1) << 24))
        return "n_tokens above 2^24";
    if (d.wdtype != MSI_W_F32 && n_tokens * d.d_model * 2 > uint64_t(0x7fffffff))
        return "n_tokens * d_model * 2 bytes of hidden states must stay below 2^31 (token rows are addressed "
               "with 32-bit offsets)";
    return "";
}

PlanCore::PlanCore(const msi_plan_desc &d, uint64_t object_bytes, const std::vector<uint64_t> &file_sizes)
{
    auto fail = [&](msi_status st, std::string m) { set_error(st, std::move(m)); };
    if (d.abi_version != MSI_ABI_VERSION)
        { fail(MSI_E_INVALID_ARG, "abi_version mismatch"); return; }
    if (d.n_layers == 0 || d.n_experts == 0 || d.n_experts > 1024)
        { fail(MSI_E_INVALID_ARG, "n_layers must be >= 1 and n_experts in [1, 1024]"); return; }
    if (d.d_model == 0 || d.d_model % 256 != 0)
        { fail(MSI_E_INVALID_ARG, "d_model must be a positive multiple of 256"); return; }
    if (d.d_ff == 0 || d.d_ff % 128 != 0)
        { fail(MSI_E_INVALID_ARG, "d_ff must be a positive multiple of 128"); return; }
    if (d.top_k == 0 || d.top_k > d.n_experts || d.top_k > 16)
        { fail(MSI_E_INVALID_ARG, "top_k must be in [1, min(n_experts, 16)]"); return; }
    if (d.wdtype > MSI_W_KQ)
        { fail(MSI_E_INVALID_ARG, "unknown wdtype"); return; }
    if (d.wdtype == MSI_W_KQ && d.d_ff % 256 != 0)
        { fail(MSI_E_INVALID_ARG, "the KQ format needs d_ff to be a multiple of 256"); return; }
    zero_cache_ = d.slots_per_layer == 0;
    pool_slots_ = zero_cache_ ? (d.transient_slots ? d.transient_slots : 8u) : d.slots_per_layer;
    if (zero_cache_ && pool_slots_ < 2)
        { fail(MSI_E_INVALID_ARG, "transient_slots must be >= 2"); return; }
    if (d.policy > MSI_POLICY_PROTECTED_LRU)
        { fail(MSI_E_INVALID_ARG, "unknown replacement policy"); return; }
    policy_ = d.policy;
    if (d.prefetch_slots && (zero_cache_ || d.prefetch_slots >= pool_slots_))
        { fail(MSI_E_INVALID_ARG, "prefetch_slots must be below slots_per_layer (and 0 for zero-cache)"); return; }
    prefetch_slots_ = d.prefetch_slots;
    if (d.slot_stride < object_bytes || d.slot_stride % 256 != 0)
        { fail(MSI_E_INVALID_ARG, "slot_stride must be >= the object size and a multiple of 256"); return; }
    if (!d.slot_pool || reinterpret_cast<uintptr_t>(d.slot_pool) % 256 != 0)
        { fail(MSI_E_INVALID_ARG, "slot_pool must be non-null and 256-byte aligned"); return; }
    const double need = double(d.n_layers) * pool_slots_ * double(d.slot_stride);
    if (double(d.slot_pool_bytes) < need)
        { fail(MSI_E_INVALID_ARG, "slot_pool_bytes smaller than n_layers * pool_slots * slot_stride"); return; }
    if (d.n_windows == 0 || !d.windows || d.window_bytes == 0)
        { fail(MSI_E_INVALID_ARG, "windows missing"); return; }
    for (uint32_t w = 0; w < d.n_windows; ++w)
        if (!d.windows[w])
            { fail(MSI_E_INVALID_ARG, "null window " + std::to_string(w)); return; }
    if (d.n_objects && !d.objects)
        { fail(MSI_E_INVALID_ARG, "objects missing"); return; }
    if (d.source && d.n_objects)
        { fail(MSI_E_INVALID_ARG, "a plan with a source takes its objects from the source's extents"); return; }

    n_layers_ = d.n_layers;
    n_experts_ = d.n_experts;
    objects_.assign(size_t(n_layers_) * n_experts_, ObjectInfo{0, 0, 0});
    has_object_.assign(size_t(n_layers_) * n_experts_, 0);
    if (d.source) {
        const msi_source_desc &sd = *d.source;
        if (sd.n_extents && !sd.extents)
            { fail(MSI_E_INVALID_ARG, "source extents missing"); return; }
        if (file_sizes.size() != sd.n_files)
            { fail(MSI_E_INVALID_ARG, "source file sizes unknown"); return; }
        source_backed_ = true;
        src_.assign(size_t(n_layers_) * n_experts_, SourceObject{});
        std::vector<uint32_t> seen(size_t(n_layers_) * n_experts_, 0);   // component bit mask
        for (uint32_t i = 0; i < sd.n_extents; ++i) {
            const msi_extent_desc &x = sd.extents[i];
            const std::string who = "extent " + std::to_string(i);
            if (x.layer >= n_layers_ || x.expert >= n_experts_ || x.file >= sd.n_files)
                { fail(MSI_E_INVALID_ARG, who + ": layer/expert/file out of range"); return; }
            if (x.component >= uint32_t(SourceService::MAX_EXTENTS) || x.nbytes == 0)
                { fail(MSI_E_INVALID_ARG, who + ": component must be < 4 and the extent non-empty"); return; }
            if (x.offset > file_sizes[x.file] || x.nbytes > file_sizes[x.file] - x.offset)
                { fail(MSI_E_SHORT, who + ": extent runs past the end of its file"); return; }
            const size_t k = size_t(x.layer) * n_experts_ + x.expert;
            if (seen[k] & (1u << x.component))
                { fail(MSI_E_INVALID_ARG, who + ": duplicate component of (layer " + std::to_string(x.layer) +
                                             ", expert " + std::to_string(x.expert) + ")"); return; }
            seen[k] |= 1u << x.component;
            src_[k].ext[x.component] = SourceExtent{x.file, x.offset, x.nbytes};
        }
        for (size_t k = 0; k < seen.size(); ++k) {
            if (!seen[k])
                continue;
            const uint32_t m = seen[k];
            if (m & (m + 1))
                { fail(MSI_E_INVALID_ARG, "object " + std::to_string(k) + ": component indices have a gap"); return; }
            int n = 0;
            uint64_t total = 0;
            while (n < SourceService::MAX_EXTENTS && (m >> n) & 1u)
                total += src_[k].ext[n++].nbytes;
            src_[k].n = n;
            if (total != object_bytes)
                { fail(MSI_E_SHORT, "object " + std::to_string(k) + ": extents add up to " + std::to_string(total) +
                                        " bytes, not the object size " + std::to_string(object_bytes)); return; }
            has_object_[k] = 1;
            objects_[k] = ObjectInfo{SOURCE_WINDOW, 0, object_bytes};
        }
    }
    for (uint32_t i = 0; i < d.n_objects; ++i) {
        const msi_object_desc &o = d.objects[i];
        if (o.layer >= n_layers_ || o.expert >= n_experts_ || o.window >= d.n_windows)
            { fail(MSI_E_INVALID_ARG, "object " + std::to_string(i) + ": layer/expert/window out of range"); return; }
        if (o.nbytes != object_bytes)
            { fail(MSI_E_SHORT, "object " + std::to_string(i) + ": extent length " +
                                         std::to_string(o.nbytes) + " != object size " +
                                         std::to_string(object_bytes)); return; }
        if (o.offset > d.window_bytes || o.nbytes > d.window_bytes - o.offset)
            { fail(MSI_E_SHORT, "object " + std::to_string(i) + ": extent runs past its window"); return; }
        const size_t k = size_t(o.layer) * n_experts_ + o.expert;
        if (has_object_[k])
            { fail(MSI_E_INVALID_ARG, "duplicate object (layer " + std::to_string(o.layer) +
                                               ", expert " + std::to_string(o.expert) + ")"); return; }
        has_object_[k] = 1;
        objects_[k] = ObjectInfo{o.window, o.offset, o.nbytes};
    }
    slots_.assign(size_t(n_layers_) * pool_slots_, Slot{});
    window_busy_.assign(d.n_windows, 0);
    layer_version_.assign(n_layers_, 1);
    res_index_.assign(size_t(n_layers_) * n_experts_, -1);
    res_index_version_.assign(n_layers_, 0);
    res_index_epoch_.assign(n_layers_, 0);
}

void PlanCore::published_map(uint32_t layer, int32_t *slot_of, uint32_t *gen_of) const
{
    for (uint32_t e = 0; e < n_experts_; ++e) {
        slot_of[e] = -1;
        gen_of[e] = 0;
    }
    if (zero_cache_)
        return;
    for (uint32_t s = 0; s < pool_slots_; ++s) {
        const Slot &sl = slot(layer, s);
        if (sl.expert < 0 || sl.fill_id >= 0)
            continue;
        if (sl.state == SlotState::DeviceReady || sl.state == SlotState::InUse ||
            sl.state == SlotState::Recyclable) {
            slot_of[sl.expert] = int32_t(global_slot(layer, s));
            gen_of[sl.expert] = sl.gen;
        }
    }
}

void PlanCore::invalidate_experts(uint32_t layer, const std::vector<int32_t> &experts)
{
    for (int32_t e : experts) {
        const int32_t s = resident_slot(layer, uint32_t(e));
        if (s < 0)
            continue;
        Slot &sl = slot(layer, uint32_t(s));
        if (sl.fill_id < 0 && sl.holds == 0 && sl.consumers == 0) {
            sl.state = SlotState::Vacant;
            sl.expert = -1;
        }
    }
    layer_version_[layer]++;
}

void PlanCore::note_direct_hits(uint32_t layer, const std::vector<int32_t> &demanded)
{
    for (int32_t e : demanded) {
        const int32_t s = resident_slot(layer, uint32_t(e));
        if (s >= 0)
            touch(layer, uint32_t(s));
        stats_.hits++;
    }
    stats_.rounds++;
    stats_.forwards++;
}

const ObjectInfo *PlanCore::object(uint32_t layer, uint32_t expert) const
{
    if (layer >= n_layers_ || expert >= n_experts_)
        return nullptr;
    const size_t k = size_t(layer) * n_experts_ + expert;
    return has_object_[k] ? &objects_[k] : nullptr;
}

const FillRecord *PlanCore::fill(int64_t id) const
{
    auto it = fills_.find(id);
    return it == fills_.end() ? nullptr : &it->second;
}

const SourceObject *PlanCore::source_object(uint32_t layer, uint32_t expert) const
{
    if (!source_backed_ || layer >= n_layers_ || expert >= n_experts_)
        return nullptr;
    const size_t k = size_t(layer) * n_experts_ + expert;
    return has_object_[k] ? &src_[k] : nullptr;
}

bool PlanCore::fill_current(int64_t id, uint32_t epoch, uint32_t gen) const
{
    auto it = fills_.find(id);
    if (it == fills_.end() || epoch != epoch_)
        return false;
    const Slot &sl = slot(it->second.layer, it->second.slot);
    return sl.fill_id == id && sl.gen == gen && sl.state == SlotState::Loading;
}

void PlanCore::fail_fill(int64_t id)
{
    auto it = fills_.find(id);
    if (it == fills_.end())
        return;
    const FillRecord rec = it->second;
    fills_.erase(it);
    if (rec.window != SOURCE_WINDOW)
        window_busy_[rec.window]--;
    stats_.fills_discarded++;
    Slot &sl = slot(rec.layer, rec.slot);
    if (sl.fill_id != id)
        return;
    sl.fill_id = -1;
    sl.state = SlotState::Vacant;
    sl.expert = -1;
    layer_version_[rec.layer]++;
}

void PlanCore::rebuild_res_index(uint32_t layer) const
{
    int32_t *ix = res_index_.data() + size_t(layer) * n_experts_;
    std::fill(ix, ix + n_experts_, -1);
    for (uint32_t s = 0; s < pool_slots_; ++s) {
        const Slot &sl = slot(layer, s);
        if (sl.expert < 0 || ix[sl.expert] >= 0)
            continue;
        switch (sl.state) {
        case SlotState::DeviceReady:
        case SlotState::InUse:
        case SlotState::Recyclable:
            ix[sl.expert] = int32_t(s);
            break;
        case SlotState::Loading:
            if (sl.epoch == epoch_)
                ix[sl.expert] = int32_t(s);   // usable once its ready event has completed
            break;
        default:
            break;
        }
    }
    res_index_version_[layer] = layer_version_[layer];
    res_index_epoch_[layer] = epoch_;
}

// Every change of a slot's object, of Vacant / Loading / published, or of the
// epoch moves the layer version or the epoch, so the table is current when
// both match.
int32_t PlanCore::resident_slot(uint32_t layer, uint32_t expert) const
{
    if (zero_cache_)
        return -1;
    if (res_index_version_[layer] != layer_version_[layer] || res_index_epoch_[layer] != epoch_)
        rebuild_res_index(layer);
    return res_index_[size_t(layer) * n_experts_ + expert];
}

int32_t PlanCore::choose_victim(uint32_t layer, const std::vector<uint8_t> &exclude, bool prefetch) const
{
    int32_t best = -1;
    uint64_t best_key = std::numeric_limits<uint64_t>::max();
    const uint32_t s0 = prefetch ? demand_slots() : 0, s1 = prefetch ? pool_slots_ : demand_slots();
    for (uint32_t s = s0; s < s1; ++s) {
        const Slot &sl = slot(layer, s);
        if (sl.holds > 0 || (!exclude.empty() && exclude[s]))
            continue;
        uint64_t key = sl.state == SlotState::Vacant ? 0 : sl.last_use + 1;
        if (!prefetch && policy_ == MSI_POLICY_PROTECTED_LRU && sl.prot && sl.state != SlotState::Vacant)
            key += uint64_t(1) << 62;          // protected: only when no unprotected slot is left
        if (key < best_key) {
            best_key = key;
            best = int32_t(s);
        }
    }
    return best;
}

void PlanCore::touch(uint32_t layer, uint32_t s)
{
    Slot &sl = slot(layer, s);
    sl.last_use = ++tick_;
    if (sl.prefetched) {
        sl.prefetched = false;
        stats_.prefetch_used++;
    }
    if (policy_ != MSI_POLICY_PROTECTED_LRU || in_prefetch_bank(s) || sl.prot)
        return;
    sl.prot = true;
    // the protected segment holds at most half of the demand bank: its least
    // recently used member returns to the unprotected one
    uint32_t n = 0;
    int32_t lru = -1;
    for (uint32_t q = 0; q < demand_slots(); ++q) {
        const Slot &o = slot(layer, q);
        if (!o.prot)
            continue;
        ++n;
        if (lru < 0 || o.last_use < slot(layer, uint32_t(lru)).last_use)
            lru = int32_t(q);
    }
    if (n > std::max(1u, demand_slots() / 2))
        slot(layer, uint32_t(lru)).prot = false;
}

msi_status PlanCore::request_prefetch(uint32_t layer, const std::vector<int32_t> &experts, std::vector<int64_t> *ids)
{
    ids->clear();
    if (layer >= n_layers_ || prefetch_slots_ == 0) {
        set_error(MSI_E_INVALID_ARG, "layer out of range or the plan has no prefetch bank");
        return MSI_E_INVALID_ARG;
    }
    for (int32_t e : experts)
        if (e < 0 || !object(layer, uint32_t(e))) {
            stats_.rejections++;
            set_error(MSI_E_WRONG_OBJECT, "prefetch of an expert outside the layer's manifest");
            return MSI_E_WRONG_OBJECT;
        }
    std::vector<uint8_t> exclude(pool_slots_, 0);
    for (int32_t e : experts) {                 // listed objects already in the bank stay
        const int32_t r = resident_slot(layer, uint32_t(e));
        if (r >= 0)
            exclude[r] = 1;
    }
    for (int32_t e : experts) {
        if (ids->size() >= prefetch_slots_)
            break;
        if (resident_slot(layer, uint32_t(e)) >= 0)
            continue;                        // resident or already loading: nothing to do
        const int32_t v = choose_victim(layer, exclude, true);
        if (v < 0 || slot(layer, uint32_t(v)).consumers > 0)
            break;
        exclude[v] = 1;
        const int64_t id = new_fill(layer, uint32_t(v), uint32_t(e));
        slot(layer, uint32_t(v)).prefetched = true;
        stats_.prefetch_fills++;
        ids->push_back(id);
    }
    return MSI_OK;
}

int64_t PlanCore::new_fill(uint32_t layer, uint32_t s, uint32_t expert)
{
    Slot &sl = slot(layer, s);
    if (sl.state != SlotState::Vacant && sl.expert >= 0)
        stats_.evictions++;
    if (sl.fill_id >= 0) {
        // An earlier fill of this slot is superseded; the device layer orders
        // the new copy after it.  Its version was either read by a round of
        // this forward (published in stream order) or never visible.
        auto it = fills_.find(sl.fill_id);
        if (it != fills_.end() && !it->second.consumed)
            stats_.fills_discarded++;
        else
            stats_.fills_published++;
        if (it != fills_.end()) {
            if (it->second.window != SOURCE_WINDOW)
                window_busy_[it->second.window]--;
            fills_.erase(it);
        }
    }
    const ObjectInfo &o = objects_[size_t(layer) * n_experts_ + expert];
    FillRecord r;
    r.id = next_fill_++;
    r.layer = layer;
    r.slot = s;
    r.expert = expert;
    r.gen = ++sl.gen;
    r.epoch = epoch_;
    r.window = o.window;
    r.offset = o.offset;
    r.nbytes = o.nbytes;
    sl.expert = int32_t(expert);
    sl.epoch = epoch_;
    sl.state = SlotState::Loading;
    sl.fill_id = r.id;
    sl.prot = false;
    sl.prefetched = false;
    layer_version_[layer]++;
    sl.last_use = ++tick_;
    if (o.window != SOURCE_WINDOW)
        window_busy_[o.window]++;
    stats_.fills++;
    stats_.h2d_bytes += o.nbytes;
    fills_.emplace(r.id, r);
    return r.id;
}

void PlanCore::publish_state(Slot &sl)
{
    sl.state = (sl.consumers + sl.holds) > 0 ? SlotState::InUse : SlotState::DeviceReady;
}

msi_status PlanCore::request_fill(uint32_t layer, uint32_t expert, int32_t forced_slot, msi_ticket *t,
                                  int64_t *fill_id)
{
    *fill_id = -1;
    if (layer >= n_layers_) {
        stats_.rejections++;
        set_error(MSI_E_INVALID_ARG, "layer out of range");
        return MSI_E_INVALID_ARG;
    }
    if (!object(layer, expert) || (forced_slot >= 0 && uint32_t(forced_slot) >= pool_slots_) ||
        forced_slot < -1) {
        stats_.rejections++;
        set_error(MSI_E_WRONG_OBJECT, "object not in this layer's manifest or slot outside its pool");
        return MSI_E_WRONG_OBJECT;
    }
    const int32_t r = resident_slot(layer, expert);
    if (r >= 0 && (forced_slot < 0 || forced_slot == r)) {
        Slot &sl = slot(layer, uint32_t(r));
        touch(layer, uint32_t(r));
        stats_.hits++;
        *t = msi_ticket{layer, expert, r, sl.gen, sl.epoch, 1u};
        return MSI_OK;
    }
    int32_t s = forced_slot;
    if (s >= 0) {
        const Slot &sl = slot(layer, uint32_t(s));
        if (sl.holds > 0 || sl.consumers > 0) {
            stats_.rejections++;
            set_error(MSI_E_BUSY, "slot has live consumers; reuse is delayed");
            return MSI_E_BUSY;
        }
    } else {
        s = choose_victim(layer, {});
        if (s < 0) {
            stats_.rejections++;
            set_error(MSI_E_BUSY, "every slot of the layer has live consumers");
            return MSI_E_BUSY;
        }
    }
    // one version per object: forget an older copy held elsewhere (no consumers)
    for (uint32_t o = 0; o < pool_slots_; ++o) {
        Slot &sl = slot(layer, o);
        if (int32_t(o) != s && sl.expert == int32_t(expert) && sl.holds == 0 && sl.consumers == 0 &&
            sl.fill_id < 0) {
            sl.state = SlotState::Vacant;
            sl.expert = -1;
            layer_version_[layer]++;
        }
    }
    stats_.misses++;
    *fill_id = new_fill(layer, uint32_t(s), expert);
    const Slot &sl = slot(layer, uint32_t(s));
    *t = msi_ticket{layer, expert, s, sl.gen, sl.epoch, 0u};
    return MSI_OK;
}

void PlanCore::complete_fill(int64_t id)
{
    auto it = fills_.find(id);
    if (it == fills_.end())
        return;
    const FillRecord rec = it->second;
    fills_.erase(it);
    if (rec.window != SOURCE_WINDOW)
        window_busy_[rec.window]--;
    Slot &sl = slot(rec.layer, rec.slot);
    if (sl.fill_id != id)
        return;
    sl.fill_id = -1;
    layer_version_[rec.layer]++;
    if (sl.state == SlotState::Loading && sl.gen == rec.gen && rec.epoch == epoch_) {
        publish_state(sl);
        stats_.fills_published++;
    } else {
        // the ticket's epoch or generation is no longer current: never visible
        sl.state = SlotState::Vacant;
        sl.expert = -1;
        stats_.fills_discarded++;
    }
}

msi_status PlanCore::schedule_forward(uint32_t layer, const std::vector<int32_t> &demanded, Schedule *out)
{
    out->rounds.clear();
    if (layer >= n_layers_) {
        set_error(MSI_E_INVALID_ARG, "layer out of range");
        return MSI_E_INVALID_ARG;
    }
    std::vector<int32_t> hits, misses;
    for (int32_t e : demanded) {
        if (e < 0 || !object(layer, uint32_t(e))) {
            stats_.rejections++;
            set_error(MSI_E_WRONG_OBJECT, "demanded expert " + std::to_string(e) +
                                              " has no object in layer " + std::to_string(layer));
            return MSI_E_WRONG_OBJECT;
        }
        (resident_slot(layer, uint32_t(e)) >= 0 ? hits : misses).push_back(e);
    }
    // misses go in storage order (window, offset) for window-backed plans:
    // with victims handed out in slot order, objects stored one after another
    // then fill consecutive slots and their copies merge into one
    if (!source_backed_)
        std::stable_sort(misses.begin(), misses.end(), [&](int32_t a, int32_t b) {
            const ObjectInfo *oa = object(layer, uint32_t(a)), *ob = object(layer, uint32_t(b));
            return oa->window != ob->window ? oa->window < ob->window : oa->offset < ob->offset;
        });
    // rounds are sized by the demand bank: misses fill only there, hits in the
    // prefetch bank take no demand slot
    const uint32_t A = demand_slots();
    uint32_t eligible = 0;
    for (uint32_t s = 0; s < A; ++s)
        eligible += slot(layer, s).holds == 0;
    if (!misses.empty() && eligible == 0) {
        stats_.rejections++;
        set_error(MSI_E_BUSY, "no slot of the layer can be freed (all held)");
        return MSI_E_BUSY;
    }
    size_t n = misses.size();
    for (int32_t e : hits)
        n += !in_prefetch_bank(uint32_t(resident_slot(layer, uint32_t(e))));
    uint32_t R = n <= A ? A : std::max(1u, A / 2);
    R = std::max(1u, std::min(R, eligible ? eligible : A));

    size_t hi = 0, mi = 0;
    while (hi < hits.size() || mi < misses.size()) {
        SchedRound round;
        std::vector<uint8_t> exclude(pool_slots_, 0);
        uint32_t taken = 0;      // eligible slots this round occupies
        while (hi < hits.size()) {
            const int32_t s = resident_slot(layer, uint32_t(hits[hi]));
            const bool el = slot(layer, uint32_t(s)).holds == 0 && !in_prefetch_bank(uint32_t(s));
            if (el && taken + 1 > R)
                break;
            exclude[s] = 1;
            taken += el;
            round.items.push_back(SchedItem{hits[hi], s, slot(layer, uint32_t(s)).gen});
            stats_.hits++;
            ++hi;
        }
        while (hi == hits.size() && mi < misses.size() && taken + 1 <= R) {
            const int32_t v = choose_victim(layer, exclude);
            if (v < 0)
                break;
            const uint32_t e = uint32_t(misses[mi]);
            const int64_t id = new_fill(layer, uint32_t(v), e);
            fills_[id].consumed = true;
            exclude[v] = 1;
            taken++;
            round.fills.push_back(fills_[id]);
            round.items.push_back(SchedItem{int32_t(e), v, slot(layer, uint32_t(v)).gen});
            stats_.misses++;
            ++mi;
        }
        if (round.items.empty()) {   // cannot happen with eligible > 0; guard the loop
            set_error(MSI_E_BUSY, "scheduler made no progress");
            return MSI_E_BUSY;
        }
        for (const SchedItem &it : round.items) {
            Slot &sl = slot(layer, uint32_t(it.slot));
            sl.consumers++;
            const bool filled = std::any_of(round.fills.begin(), round.fills.end(),
                                            [&](const FillRecord &f) { return int32_t(f.slot) == it.slot; });
            if (filled)
                sl.last_use = ++tick_;
            else
                touch(layer, uint32_t(it.slot));     // a hit
            if (sl.state != SlotState::Loading)
                sl.state = SlotState::InUse;
        }
        stats_.rounds++;
        out->rounds.push_back(std::move(round));
    }
    stats_.forwards++;
    return MSI_OK;
}

void PlanCore::end_forward(uint32_t layer, const Schedule &s)
{
    for (const SchedRound &r : s.rounds)
        for (const SchedItem &it : r.items) {
            Slot &sl = slot(layer, uint32_t(it.slot));
            if (sl.consumers)
                sl.consumers--;
            if (sl.consumers + sl.holds == 0 &&
                (sl.state == SlotState::InUse || sl.state == SlotState::DeviceReady))
                sl.state = SlotState::Recyclable;
        }
    layer_version_[layer]++;
    if (zero_cache_)
        for (uint32_t s2 = 0; s2 < pool_slots_; ++s2) {
            Slot &sl = slot(layer, s2);
            if (sl.holds == 0 && sl.consumers == 0 && sl.fill_id < 0) {
                sl.state = SlotState::Vacant;
                sl.expert = -1;
            }
        }
}

void PlanCore::invalidate_read_slots(uint32_t layer, const Schedule &s)
{
    layer_version_[layer]++;
    for (const SchedRound &r : s.rounds)
        for (const SchedItem &it : r.items) {
            Slot &sl = slot(layer, uint32_t(it.slot));
            if (sl.fill_id < 0 && sl.holds == 0 && sl.consumers == 0) {
                sl.state = SlotState::Vacant;
                sl.expert = -1;
            }
        }
}

msi_status PlanCore::hold(uint32_t layer, uint32_t s)
{
    if (layer >= n_layers_ || s >= pool_slots_) {
        set_error(MSI_E_INVALID_ARG, "layer or slot out of range");
        return MSI_E_INVALID_ARG;
    }
    Slot &sl = slot(layer, s);
    sl.holds++;
    if (sl.state == SlotState::DeviceReady || sl.state == SlotState::Recyclable)
        sl.state = SlotState::InUse;
    return MSI_OK;
}

msi_status PlanCore::unhold(uint32_t layer, uint32_t s)
{
    if (layer >= n_layers_ || s >= pool_slots_) {
        set_error(MSI_E_INVALID_ARG, "layer or slot out of range");
        return MSI_E_INVALID_ARG;
    }
    Slot &sl = slot(layer, s);
    if (sl.holds == 0) {
        stats_.rejections++;
        set_error(MSI_E_STATE, "slot has no held consumer");
        return MSI_E_STATE;
    }
    sl.holds--;
    if (sl.holds + sl.consumers == 0 && sl.state == SlotState::InUse)
        sl.state = SlotState::Recyclable;
    return MSI_OK;
}

bool PlanCore::any_holds() const
{
    for (const Slot &s : slots_)
        if (s.holds)
            return true;
    return false;
}

msi_status PlanCore::reset()
{
    if (any_holds()) {
        stats_.rejections++;
        set_error(MSI_E_BUSY, "reset with a live held consumer");
        return MSI_E_BUSY;
    }
    epoch_++;
    return MSI_OK;
}

uint64_t PlanCore::fills_in_flight() const { return fills_.size(); }

uint64_t PlanCore::windows_busy() const
{
    uint64_t n = 0;
    for (uint32_t b : window_busy_)
        n += b > 0;
    return n;
}

uint64_t PlanCore::consumers_live() const
{
    uint64_t n = 0;
    for (const Slot &s : slots_)
        n += s.consumers + s.holds;
    return n;
}

}  // namespace msi
