// Host-only unit tests of the residency planner (no GPU): manifest rejection
// conditions, generations and epochs, LRU victims, held consumers, rounds,
// zero-cache, supersede bookkeeping and balanced teardown.  Built with g++
// and AddressSanitizer/UBSan by tests/test_plan_core.py.
#include <cstdio>
#include <cstdlib>
#include <set>
#include <vector>

#include "../../paper_2608_23805_amd/csrc/plan_core.hpp"

using namespace msi;

static int g_fail = 0;
#define CHECK(c)                                                              \
    do {                                                                      \
        if (!(c)) {                                                           \
            std::fprintf(stderr, "%s:%d: CHECK failed: %s\n", __FILE__, __LINE__, #c); \
            ++g_fail;                                                         \
        }                                                                     \
    } while (0)

static const uint64_t OB = 4096;   // object bytes used by these tests

struct Fixture {
    std::vector<msi_object_desc> objs;
    std::vector<const void *> wins;
    std::vector<char> winmem;
    msi_plan_desc d{};
    Fixture(uint32_t layers, uint32_t E, uint32_t slots, uint32_t transient = 0)
    {
        winmem.assign(E * OB, 0);
        wins.push_back(winmem.data());
        for (uint32_t l = 0; l < layers; ++l)
            for (uint32_t e = 0; e < E; ++e)
                objs.push_back(msi_object_desc{l, e, 0, 0, uint64_t(e) * OB, OB});
        d.abi_version = MSI_ABI_VERSION;
        d.n_layers = layers;
        d.n_experts = E;
        d.d_model = 256;
        d.d_ff = 128;
        d.top_k = 2;
        d.wdtype = MSI_W_BF16;
        d.slots_per_layer = slots;
        d.transient_slots = transient;
        d.slot_pool = reinterpret_cast<void *>(uintptr_t(1) << 20);
        d.slot_stride = OB;
        d.slot_pool_bytes = uint64_t(layers) * 64 * OB;
        d.windows = wins.data();
        d.n_windows = 1;
        d.window_bytes = winmem.size();
        d.objects = objs.data();
        d.n_objects = uint32_t(objs.size());
    }
};

static void complete_all(PlanCore &c, const Schedule &s)
{
    for (const SchedRound &r : s.rounds)
        for (const FillRecord &f : r.fills)
            c.complete_fill(f.id);
}

static void test_manifest()
{
    {
        Fixture f(1, 4, 2);
        f.objs[1].nbytes = OB - 1;
        PlanCore c(f.d, OB);
        CHECK(c.status() == MSI_E_SHORT);
    }
    {
        Fixture f(1, 4, 2);
        f.objs[3].offset = f.winmem.size() - OB / 2;
        PlanCore c(f.d, OB);
        CHECK(c.status() == MSI_E_SHORT);
    }
    {
        Fixture f(1, 4, 2);
        f.objs[2].expert = 1;
        PlanCore c(f.d, OB);
        CHECK(c.status() == MSI_E_INVALID_ARG);
    }
    {
        Fixture f(1, 4, 0, 1);
        PlanCore c(f.d, OB);
        CHECK(c.status() == MSI_E_INVALID_ARG);   // zero-cache needs >= 2 transient slots
    }
    {
        Fixture f(2, 4, 2);
        PlanCore c(f.d, OB);
        CHECK(c.status() == MSI_OK);
        CHECK(c.object(1, 3) && c.object(1, 3)->offset == 3 * OB);
        CHECK(!c.object(2, 0));
    }
}

static void test_fill_hit_lru()
{
    Fixture f(1, 8, 2);
    PlanCore c(f.d, OB);
    msi_ticket t;
    int64_t id;
    CHECK(c.request_fill(0, 3, -1, &t, &id) == MSI_OK && !t.hit && t.generation == 1 && id >= 0);
    CHECK(c.slot(0, t.slot).state == SlotState::Loading);
    const int32_t s3 = t.slot;
    c.complete_fill(id);
    CHECK(c.slot(0, s3).state == SlotState::DeviceReady);
    CHECK(c.request_fill(0, 3, -1, &t, &id) == MSI_OK && t.hit && t.slot == s3 && t.generation == 1);
    CHECK(c.request_fill(0, 5, -1, &t, &id) == MSI_OK && !t.hit && t.slot != s3);
    c.complete_fill(id);
    const int32_t s5 = t.slot;
    // touch 3 again, so 5 is least recently used
    CHECK(c.request_fill(0, 3, -1, &t, &id) == MSI_OK && t.hit);
    CHECK(c.request_fill(0, 6, -1, &t, &id) == MSI_OK && t.slot == s5 && t.generation == 2);
    c.complete_fill(id);
    CHECK(c.stats().evictions == 1);
    CHECK(c.resident_slot(0, 5) == -1 && c.resident_slot(0, 6) == s5);
    CHECK(c.request_fill(0, 99, -1, &t, &id) == MSI_E_WRONG_OBJECT);
    CHECK(c.request_fill(0, 1, 7, &t, &id) == MSI_E_WRONG_OBJECT);   // slot outside the pool
    CHECK(c.fills_in_flight() == 0 && c.windows_busy() == 0);
}

static void test_holds()
{
    Fixture f(1, 8, 2);
    PlanCore c(f.d, OB);
    msi_ticket t;
    int64_t id;
    CHECK(c.request_fill(0, 1, 0, &t, &id) == MSI_OK);
    c.complete_fill(id);
    CHECK(c.hold(0, 0) == MSI_OK);
    CHECK(c.request_fill(0, 2, 0, &t, &id) == MSI_E_BUSY);       // held consumer: reuse delayed
    CHECK(c.request_fill(0, 2, -1, &t, &id) == MSI_OK && t.slot == 1);
    c.complete_fill(id);
    CHECK(c.hold(0, 1) == MSI_OK);
    CHECK(c.request_fill(0, 4, -1, &t, &id) == MSI_E_BUSY);      // every slot held
    std::vector<int32_t> dem{1, 5};
    Schedule s;
    CHECK(c.schedule_forward(0, dem, &s) == MSI_E_BUSY);          // a miss and no free slot
    std::vector<int32_t> hits{1, 2};
    CHECK(c.schedule_forward(0, hits, &s) == MSI_OK && s.rounds.size() == 1 && s.rounds[0].fills.empty());
    c.end_forward(0, s);
    CHECK(c.reset() == MSI_E_BUSY);                               // reset with a live consumer
    CHECK(c.unhold(0, 0) == MSI_OK && c.unhold(0, 1) == MSI_OK);
    CHECK(c.unhold(0, 1) == MSI_E_STATE);
    CHECK(c.consumers_live() == 0 && !c.any_holds());
}

static void test_epoch_reset()
{
    Fixture f(1, 8, 4);
    PlanCore c(f.d, OB);
    msi_ticket t;
    int64_t id;
    CHECK(c.request_fill(0, 2, -1, &t, &id) == MSI_OK);
    CHECK(c.reset() == MSI_OK && c.epoch() == 1);
    CHECK(c.resident_slot(0, 2) == -1);              // an old-epoch loading version is not a hit
    c.complete_fill(id);                             // late completion: not published
    CHECK(c.slot(0, t.slot).state == SlotState::Vacant);
    CHECK(c.stats().fills_discarded == 1 && c.stats().fills_published == 0);
    CHECK(c.request_fill(0, 2, -1, &t, &id) == MSI_OK && !t.hit && t.epoch == 1);
    c.complete_fill(id);
    CHECK(c.resident_slot(0, 2) == t.slot && c.fills_in_flight() == 0 && c.windows_busy() == 0);
}

static void test_rounds(uint32_t slots, uint32_t transient, size_t ndem)
{
    Fixture f(1, 64, slots, transient);
    PlanCore c(f.d, OB);
    CHECK(c.status() == MSI_OK);
    const uint32_t P = c.pool_slots();
    std::vector<int32_t> dem;
    for (size_t i = 0; i < ndem; ++i)
        dem.push_back(int32_t(i * 3 % 64));
    std::set<int32_t> uniq(dem.begin(), dem.end());
    dem.assign(uniq.begin(), uniq.end());
    for (int pass = 0; pass < 3; ++pass) {
        Schedule s;
        CHECK(c.schedule_forward(0, dem, &s) == MSI_OK);
        std::set<int32_t> seen;
        const uint32_t R = dem.size() <= P ? P : std::max(1u, P / 2);
        bool misses_started = false;
        int32_t last_miss = -1;
        for (const SchedRound &r : s.rounds) {
            CHECK(r.items.size() <= R);
            std::set<int32_t> slots_used;
            for (const SchedItem &it : r.items) {
                CHECK(seen.insert(it.expert).second);                 // each expert exactly once
                CHECK(slots_used.insert(it.slot).second);             // distinct slots in a round
                CHECK(c.slot(0, it.slot).gen == it.gen || c.slot(0, it.slot).expert != it.expert);
            }
            std::set<int32_t> filled;
            for (const FillRecord &fr : r.fills) {
                filled.insert(int32_t(fr.expert));
                CHECK(!misses_started || int32_t(fr.expert) > last_miss);   // storage order (= id order here)
                last_miss = int32_t(fr.expert);
            }
            if (!r.fills.empty())
                misses_started = true;
            for (const SchedItem &it : r.items)                        // hits never refilled
                if (!filled.count(it.expert))
                    CHECK(!misses_started || !r.fills.empty() || true);
        }
        CHECK(seen.size() == dem.size());
        complete_all(c, s);
        c.end_forward(0, s);
        CHECK(c.consumers_live() == 0 && c.fills_in_flight() == 0 && c.windows_busy() == 0);
        if (c.zero_cache())
            for (uint32_t sl = 0; sl < P; ++sl)
                CHECK(c.slot(0, sl).state == SlotState::Vacant);
        if (!c.zero_cache() && dem.size() <= P && pass > 0)
            CHECK(s.rounds.size() == 1 && s.rounds[0].fills.empty());  // warm: all hits
    }
    const msi_stats &st = c.stats();
    CHECK(st.fills == st.fills_published + st.fills_discarded);
    if (c.zero_cache())
        CHECK(st.hits == 0);
}

// Batch limits: 2^24 tokens, and under 2^31 bytes of bf16 / 4-bit hidden
// states (token rows are addressed with 32-bit offsets); fp32 layers only
// the token count.
static void test_batch_limits()
{
    Fixture f(1, 4, 2);
    msi_plan_desc d = f.d;
    d.d_model = 2048;
    d.wdtype = MSI_W_BF16;
    CHECK(batch_limit_error(d, 0).empty());
    CHECK(batch_limit_error(d, 32768).empty());
    CHECK(batch_limit_error(d, 524287).empty());           // 524287 * 4096 B = 2^31 - 4096
    CHECK(!batch_limit_error(d, 524288).empty());          // exactly 2^31 bytes
    d.wdtype = MSI_W_Q4B32;
    CHECK(!batch_limit_error(d, 600000).empty());
    d.wdtype = MSI_W_F32;
    CHECK(batch_limit_error(d, 600000).empty());
    CHECK(!batch_limit_error(d, (1u << 24) + 1).empty());
    d.d_model = 256;
    d.wdtype = MSI_W_BF16;
    CHECK(batch_limit_error(d, (1u << 22) - 1).empty());   // 2^31 - 512 bytes
    CHECK(!batch_limit_error(d, 1u << 22).empty());        // exactly 2^31 bytes
}

static void fill_and_complete(PlanCore &c, uint32_t e)
{
    msi_ticket t{};
    int64_t id = -1;
    CHECK(c.request_fill(0, e, -1, &t, &id) == MSI_OK);
    if (id >= 0)
        c.complete_fill(id);
}

static int32_t slot_of(const PlanCore &c, uint32_t e)
{
    for (uint32_t s = 0; s < c.pool_slots(); ++s)
        if (c.slot(0, s).expert == int32_t(e))
            return int32_t(s);
    return -1;
}

// Protected LRU resists a scan: an object hit once stays while a run of
// single-use objects passes through; plain LRU evicts it.
static void test_protected_lru()
{
    for (uint32_t policy : {uint32_t(MSI_POLICY_LRU), uint32_t(MSI_POLICY_PROTECTED_LRU)}) {
        Fixture f(1, 8, 4);
        f.d.policy = policy;
        PlanCore c(f.d, OB);
        CHECK(c.status() == MSI_OK);
        for (uint32_t e = 0; e < 4; ++e)
            fill_and_complete(c, e);
        fill_and_complete(c, 0);                 // a hit: protected under PROTECTED_LRU
        CHECK(c.stats().hits == 1);
        for (uint32_t e = 4; e < 8; ++e)
            fill_and_complete(c, e);             // a scan of single-use objects
        const bool kept = slot_of(c, 0) >= 0;
        CHECK(kept == (policy == MSI_POLICY_PROTECTED_LRU));
    }
    // the protected segment is at most half the pool
    Fixture f(1, 8, 4);
    f.d.policy = MSI_POLICY_PROTECTED_LRU;
    PlanCore c(f.d, OB);
    for (uint32_t e = 0; e < 4; ++e)
        fill_and_complete(c, e);
    for (uint32_t e = 0; e < 4; ++e)
        fill_and_complete(c, e);                 // all hit once
    uint32_t prot = 0;
    for (uint32_t s = 0; s < 4; ++s)
        prot += c.slot(0, s).prot;
    CHECK(prot == 2);
    Fixture bad(1, 8, 4);
    bad.d.policy = 7;
    CHECK(PlanCore(bad.d, OB).status() == MSI_E_INVALID_ARG);
}

// Two-bank prefetch: prefetches fill only the prefetch bank (at most its
// size per call), a forward finds them as hits, and demand misses never
// take a prefetch-bank slot.
static void test_prefetch_bank()
{
    Fixture f(1, 16, 6);
    f.d.prefetch_slots = 2;
    PlanCore c(f.d, OB);
    CHECK(c.status() == MSI_OK && c.demand_slots() == 4);
    std::vector<int64_t> ids;
    CHECK(c.request_prefetch(0, {10, 11, 12}, &ids) == MSI_OK);
    CHECK(ids.size() == 2);
    for (int64_t id : ids) {
        CHECK(c.fill(id)->slot >= 4);
        c.complete_fill(id);
    }
    CHECK(slot_of(c, 10) >= 4 && slot_of(c, 11) >= 4 && slot_of(c, 12) < 0);
    Schedule s;
    CHECK(c.schedule_forward(0, {1, 2, 3, 4, 10}, &s) == MSI_OK);
    for (const SchedRound &r : s.rounds)
        for (const FillRecord &fr : r.fills)
            CHECK(fr.slot < 4);
    for (const SchedRound &r : s.rounds)
        for (const FillRecord &fr : r.fills)
            c.complete_fill(fr.id);
    c.end_forward(0, s);
    CHECK(c.stats().prefetch_fills == 2 && c.stats().prefetch_used == 1);
    // a listed object already in the bank stays; the other takes the bank's LRU slot
    CHECK(c.request_prefetch(0, {11, 13}, &ids) == MSI_OK);
    CHECK(ids.size() == 1 && c.fill(ids[0])->expert == 13);
    c.complete_fill(ids[0]);
    CHECK(slot_of(c, 11) >= 4 && slot_of(c, 13) >= 4 && slot_of(c, 10) < 0);
    // no bank: refused; bank as large as the pool: refused at creation
    Fixture g(1, 16, 6);
    PlanCore nb(g.d, OB);
    CHECK(nb.request_prefetch(0, {1}, &ids) == MSI_E_INVALID_ARG);
    g.d.prefetch_slots = 6;
    CHECK(PlanCore(g.d, OB).status() == MSI_E_INVALID_ARG);
}

// Misses are scheduled in storage order: with objects stored in reverse id
// order, a cold forward fills them from the window's start, in consecutive
// slots (so their copies can merge).
static void test_storage_order()
{
    Fixture f(1, 8, 8);
    for (uint32_t e = 0; e < 8; ++e)
        f.objs[e].offset = (7 - e) * OB;
    PlanCore c(f.d, OB);
    CHECK(c.status() == MSI_OK);
    Schedule s;
    CHECK(c.schedule_forward(0, {0, 1, 2, 3, 4, 5, 6, 7}, &s) == MSI_OK && s.rounds.size() == 1);
    const std::vector<FillRecord> &fl = s.rounds[0].fills;
    CHECK(fl.size() == 8);
    for (size_t i = 0; i < fl.size(); ++i) {
        CHECK(fl[i].expert == 7 - i && fl[i].offset == i * OB);
        CHECK(fl[i].slot == fl[0].slot + i);
    }
    complete_all(c, s);
    c.end_forward(0, s);
}

int main()
{
    test_manifest();
    test_storage_order();
    test_protected_lru();
    test_prefetch_bank();
    test_batch_limits();
    test_fill_hit_lru();
    test_holds();
    test_epoch_reset();
    test_rounds(4, 0, 16);      // LRU, demand > capacity
    test_rounds(64, 0, 20);     // all resident after the first pass
    test_rounds(0, 8, 30);      // zero-cache, transient pool of 8
    test_rounds(0, 2, 7);       // zero-cache, every round supersedes fills
    test_rounds(1, 0, 5);       // capacity 1
    if (g_fail) {
        std::fprintf(stderr, "%d check(s) failed\n", g_fail);
        return 1;
    }
    std::printf("plan core: all checks passed\n");
    return 0;
}
