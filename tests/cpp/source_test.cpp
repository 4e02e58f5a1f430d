// Host-only unit tests of the bounded source service (no GPU): covering
// reads of unaligned extents into aligned windows, the in-flight bound, the
// window state sequence, and the rejection conditions (short read, negative
// completion, stale ticket, extent overflow), held reads, and draining at
// destruction.  Built with g++ and AddressSanitizer/UBSan, and separately
// with ThreadSanitizer, by tests/test_plan_core.py.
#include <fcntl.h>
#include <unistd.h>

#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <memory>
#include <string>
#include <vector>

#include "../../paper_2608_23805_amd/csrc/source.hpp"

using namespace msi;

static int g_fail = 0;
#define CHECK(c)                                                                          \
    do {                                                                                  \
        if (!(c)) {                                                                       \
            std::fprintf(stderr, "%s:%d: CHECK failed: %s\n", __FILE__, __LINE__, #c);   \
            ++g_fail;                                                                     \
        }                                                                                 \
    } while (0)

static uint8_t pattern(uint64_t i) { return uint8_t((i * 131u + (i >> 9) * 7u + 3u) & 0xFFu); }

struct TempFile {
    std::string path;
    explicit TempFile(uint64_t bytes)
    {
        char tmpl[] = "/tmp/msi_source_testXXXXXX";
        const int fd = mkstemp(tmpl);
        path = tmpl;
        std::vector<uint8_t> buf(bytes);
        for (uint64_t i = 0; i < bytes; ++i)
            buf[i] = pattern(i);
        CHECK(write(fd, buf.data(), buf.size()) == ssize_t(buf.size()));
        close(fd);
    }
    ~TempFile() { unlink(path.c_str()); }
};

struct Windows {
    std::vector<void *> w;
    Windows(int n, uint64_t bytes)
    {
        for (int i = 0; i < n; ++i)
            w.push_back(std::aligned_alloc(4096, bytes));
    }
    ~Windows()
    {
        for (void *p : w)
            std::free(p);
    }
};

static auto always = [](uint64_t, uint32_t, uint32_t) { return true; };

static std::vector<SourceService::Done> wait_all(SourceService &S, size_t n)
{
    std::vector<SourceService::Done> out;
    const auto t0 = std::chrono::steady_clock::now();
    while (out.size() < n && std::chrono::steady_clock::now() - t0 < std::chrono::seconds(20)) {
        auto d = S.collect(50, always);
        out.insert(out.end(), d.begin(), d.end());
    }
    return out;
}

static void test_reads_and_layout()
{
    TempFile f(3 << 20);
    Windows W(4, 1 << 20);
    auto SP = std::make_unique<SourceService>(std::vector<std::string>{f.path}, W.w, 1 << 20, 2, 4096, true);
    SourceService &S = *SP;
    CHECK(S.ok());
    CHECK(S.file_size(0) == (3u << 20));
    const SourceExtent ext[3] = {{0, 1000, 100000}, {0, 300001, 123457}, {0, 2100000, 50000}};
    uint64_t place[3], phys = 0;
    CHECK(S.layout(ext, 3, place, &phys));
    CHECK(phys % 4096 == 0 && phys >= 100000 + 123457 + 50000);
    for (uint64_t tag = 0; tag < 4; ++tag)
        CHECK(S.submit(uint32_t(tag), ext, 3, tag, 0, 1));
    CHECK(!S.submit(0, ext, 3, 9, 0, 1));                 // window 0 is Reading, not Free
    CHECK(S.free_window() == -1 && S.busy_windows() == 4);
    auto done = wait_all(S, 4);
    CHECK(done.size() == 4);
    for (const auto &d : done) {
        CHECK(d.error == SourceError::None);
        CHECK(S.state(d.window) == WindowState::HostReady);
        const uint8_t *w = S.window(d.window);
        bool same = true;
        for (int i = 0; i < 3; ++i)
            for (uint64_t b = 0; b < ext[i].nbytes; b += 997)
                same &= w[place[i] + b] == pattern(ext[i].offset + b);
        CHECK(same);
        S.set_copying(d.window);
        CHECK(S.state(d.window) == WindowState::Copying);
        S.set_free(d.window);
        CHECK(S.state(d.window) == WindowState::Free);
    }
    const SourceStats st = S.stats();
    CHECK(st.reads_issued == 12 && st.reads_completed == 12 && st.reads_failed == 0);
    CHECK(st.peak_depth >= 1 && st.peak_depth <= 2);        // in-flight limit 2
    CHECK(st.logical_bytes == 4 * (100000u + 123457u + 50000u));
    CHECK(st.physical_bytes == 4 * phys && st.padding_bytes == st.physical_bytes - st.logical_bytes);
    CHECK(st.direct + st.buffered == 1);
    // overflow: extents that do not fit the window are refused, the window stays Free
    const SourceExtent big[2] = {{0, 0, 600000}, {0, 700000, 600000}};
    CHECK(!S.layout(big, 2, place, nullptr));
    CHECK(!S.submit(1, big, 2, 20, 0, 1) && S.state(1) == WindowState::Free);
}

static void test_rejections()
{
    TempFile f(1 << 20);
    Windows W(2, 1 << 20);
    auto SP = std::make_unique<SourceService>(std::vector<std::string>{f.path}, W.w, 1 << 20, 8, 4096, true);
    SourceService &S = *SP;
    CHECK(S.ok());
    // extent past the end of the file: a short read
    const SourceExtent past[1] = {{0, (1 << 20) - 5000, 10000}};
    CHECK(S.submit(0, past, 1, 1, 0, 1));
    auto d = wait_all(S, 1);
    CHECK(d.size() == 1 && d[0].error == SourceError::Short && S.state(0) == WindowState::Free);
    // an extent ending exactly at the file's end is whole
    const SourceExtent tail[1] = {{0, (1 << 20) - 5000, 5000}};
    CHECK(S.submit(0, tail, 1, 2, 0, 1));
    d = wait_all(S, 1);
    CHECK(d.size() == 1 && d[0].error == SourceError::None);
    S.set_free(0);
    // forced short read and EIO on one component of a bundle of three: the bundle fails
    const SourceExtent ext[3] = {{0, 10, 1000}, {0, 20000, 3000}, {0, 50000, 7000}};
    S.inject(3, 1, SourceFault::Short);
    CHECK(S.submit(0, ext, 3, 3, 0, 1));
    S.inject(4, 2, SourceFault::Eio);
    CHECK(S.submit(1, ext, 3, 4, 0, 1));
    d = wait_all(S, 2);
    CHECK(d.size() == 2);
    for (const auto &x : d) {
        CHECK(x.error == (x.tag == 3 ? SourceError::Short : SourceError::Io));
        if (x.tag == 4)
            CHECK(x.sys_errno == EIO);
        CHECK(S.state(x.window) == WindowState::Free);
    }
    // stale ticket at completion: judged by the caller's predicate
    CHECK(S.submit(0, ext, 3, 5, 7, 9));
    std::vector<SourceService::Done> got;
    const auto t0 = std::chrono::steady_clock::now();
    while (got.empty() && std::chrono::steady_clock::now() - t0 < std::chrono::seconds(20))
        got = S.collect(50, [](uint64_t tag, uint32_t ep, uint32_t gen) { return !(tag == 5 && ep == 7 && gen == 9); });
    CHECK(got.size() == 1 && got[0].error == SourceError::Stale && S.state(0) == WindowState::Free);
    const SourceStats st = S.stats();
    CHECK(st.requests_failed == 4 && st.requests_stale == 1 && st.requests_ready == 1);
    CHECK(S.outstanding() == 0 && S.busy_windows() == 0);
}

static void test_hold_and_drain()
{
    TempFile f(1 << 20);
    Windows W(2, 1 << 20);
    {
        auto SP = std::make_unique<SourceService>(std::vector<std::string>{f.path}, W.w, 1 << 20, 1, 4096, true);
        SourceService &S = *SP;
        const SourceExtent ext[1] = {{0, 4096, 8192}};
        S.inject(1, 0, SourceFault::Hold);
        CHECK(S.submit(0, ext, 1, 1, 0, 1));
        CHECK(S.submit(1, ext, 1, 2, 0, 1));            // behind the held read (one worker)
        CHECK(S.collect(100, always).empty());           // held: nothing completes
        CHECK(S.outstanding() == 2);
        S.release_holds();
        auto d = wait_all(S, 2);
        CHECK(d.size() == 2);
        // a release that comes before the worker reaches a held read lets it go too:
        // with one worker busy on held read 4, read 5 (also held) is still queued
        S.set_free(0);
        S.set_free(1);
        S.inject(4, 0, SourceFault::Hold);
        S.inject(5, 0, SourceFault::Hold);
        CHECK(S.submit(0, ext, 1, 4, 0, 1));
        CHECK(S.submit(1, ext, 1, 5, 0, 1));
        CHECK(S.collect(100, always).empty());
        const auto tr = std::chrono::steady_clock::now();
        S.release_holds();
        d = wait_all(S, 2);
        CHECK(d.size() == 2);
        CHECK(std::chrono::steady_clock::now() - tr < std::chrono::seconds(10));
        // a held read at destruction: the destructor lets it go and drains
        S.set_free(0);
        S.set_free(1);
        S.inject(3, 0, SourceFault::Hold);
        CHECK(S.submit(0, ext, 1, 3, 0, 1));
        const auto t0 = std::chrono::steady_clock::now();
        (void)t0;
    }
    // bad configurations
    Windows M(1, 1 << 20);
    std::vector<void *> mis{static_cast<uint8_t *>(M.w[0]) + 512};
    CHECK(!std::make_unique<SourceService>(std::vector<std::string>{f.path}, mis, 1 << 19, 1, 4096, true)->ok());
    CHECK(!std::make_unique<SourceService>(std::vector<std::string>{f.path}, M.w, 1 << 20, 9, 4096, true)->ok());
    CHECK(!std::make_unique<SourceService>(std::vector<std::string>{"/nonexistent/file"}, M.w, 1 << 20, 1, 4096,
                                           true)->ok());
}

// Reads staged through the workers' bounce buffers: the same bytes land in
// the windows, covering reads longer than one bounce buffer included.
static void test_bounce()
{
    TempFile f(12 << 20);
    Windows W(2, 12 << 20);
    auto SP = std::make_unique<SourceService>(std::vector<std::string>{f.path}, W.w, 12 << 20, 2, 4096, true);
    SourceService &S = *SP;
    S.use_bounce_buffers();
    const SourceExtent ext[2] = {{0, 777, 9 << 20}, {0, (9 << 20) + 5000, 1234567}};
    uint64_t place[2];
    CHECK(S.layout(ext, 2, place, nullptr));
    CHECK(S.submit(0, ext, 2, 1, 0, 1));
    auto d = wait_all(S, 1);
    CHECK(d.size() == 1 && d[0].error == SourceError::None);
    const uint8_t *w = S.window(0);
    bool same = true;
    for (int i = 0; i < 2; ++i)
        for (uint64_t b = 0; b < ext[i].nbytes; b += 1009)
            same &= w[place[i] + b] == pattern(ext[i].offset + b);
    same &= w[place[0] + ext[0].nbytes - 1] == pattern(ext[0].offset + ext[0].nbytes - 1);
    CHECK(same);
    CHECK(S.stats().bounced == 2);
}

int main()
{
    test_reads_and_layout();
    test_bounce();
    test_rejections();
    const auto t0 = std::chrono::steady_clock::now();
    test_hold_and_drain();
    const double dt = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
    CHECK(dt < 10.0);   // the held read at destruction did not wait for its 30 s limit
    if (g_fail) {
        std::fprintf(stderr, "%d check(s) failed\n", g_fail);
        return 1;
    }
    std::printf("source service: all checks passed\n");
    return 0;
}
