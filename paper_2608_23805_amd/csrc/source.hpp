// source.hpp -- bounded source service: canonical expert bytes read from
// files into a fixed set of aligned host windows (the paper's Design
// section, "Bounded Source Service" and "Separate Window and GPU-Slot
// Lifecycles").
//
// Pure C++17, no HIP.  The service opens the canonical files for direct I/O
// (O_DIRECT; buffered reads only where the caller allows the fallback and the
// file system refuses direct I/O), owns no window memory (the caller passes
// N_w windows of W bytes, aligned to the direct-I/O block), and runs at most
// `inflight` reads at a time on a fixed set of I/O worker threads, so the
// source's memory is bounded by N_w * W plus its queue and metadata (and,
// when the windows' pages cannot take direct reads, one 4 MiB bounce buffer
// per I/O worker).
//
// A request assembles one logical object from up to MAX_EXTENTS extents (the
// components of one bundle: gate, up, down).  Each extent is read with one
// covering read, aligned down / up to the block size, into its own aligned
// region of the window; the logical bytes of extent i then sit at
// window + place[i].  Window states: Free -> Reading -> HostReady ->
// Copying -> Free.  A window becomes HostReady only after every extent of its
// request completed with the whole covering length (or the file's end past
// the extent's last byte) and the request's ticket (object, epoch,
// generation) is still current; a short read, a negative completion or a
// stale ticket makes the request Failed, and its window returns to Free
// without ever becoming HostReady (nothing from it may be published).
#pragma once

#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdint>
#include <deque>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

namespace msi {

enum class WindowState : uint32_t { Free = 0, Reading = 1, HostReady = 2, Copying = 3 };

struct SourceExtent {
    uint32_t file = 0;
    uint64_t offset = 0;       // byte offset of the logical extent in the file
    uint64_t nbytes = 0;       // logical bytes
};

// Why a request failed (the rejection conditions of the service).
enum class SourceError : uint32_t {
    None = 0,
    Short = 1,       // a read returned fewer bytes than the extent needs
    Io = 2,          // a read completed with a negative status (errno)
    Stale = 3,       // the request's ticket was no longer current at completion
    Overflow = 4,    // the extents do not fit the window
};

// Test hooks: what the next read of an object's given extent does instead.
enum class SourceFault : uint32_t { None = 0, Short = 1, Eio = 2, Hold = 3 };

struct SourceStats {
    uint64_t reads_issued = 0, reads_completed = 0, reads_failed = 0;
    uint64_t requests = 0, requests_ready = 0, requests_failed = 0, requests_stale = 0;
    uint64_t logical_bytes = 0, physical_bytes = 0, padding_bytes = 0;
    uint64_t peak_depth = 0;          // most reads in flight at once
    double read_seconds = 0.0;        // summed read latency
    uint32_t direct = 0;              // files opened for direct I/O
    uint32_t buffered = 0;            // files read through the page cache (fallback)
    uint64_t bounced = 0;             // reads that went through a worker's bounce buffer
};

class SourceService {
public:
    static constexpr int MAX_EXTENTS = 4;
    static constexpr int MAX_INFLIGHT = 8;

    // files: canonical file paths; windows: n host buffers of window_bytes,
    // each aligned to `align` (a power of two >= 512); inflight in
    // [1, MAX_INFLIGHT].  On failure ok() is false and error() says why.
    SourceService(const std::vector<std::string> &files, const std::vector<void *> &windows, uint64_t window_bytes,
                  uint32_t inflight, uint32_t align, bool allow_buffered);
    ~SourceService();   // drains every read in flight, then closes the files
    SourceService(const SourceService &) = delete;
    SourceService &operator=(const SourceService &) = delete;

    bool ok() const { return err_.empty(); }
    const std::string &error() const { return err_; }
    uint32_t n_windows() const { return uint32_t(windows_.size()); }
    uint64_t file_size(uint32_t f) const { return f < sizes_.size() ? sizes_[f] : 0; }
    uint32_t inflight_limit() const { return inflight_; }

    // Covering-read layout of a request: false (Overflow) if it does not fit a window.
    bool layout(const SourceExtent *ext, int n, uint64_t *place, uint64_t *physical) const;

    // Start a request into Free window w; the ticket (tag, epoch, gen) comes
    // back with the completion.  Returns false if w is not Free or the
    // extents do not fit (the window stays Free).
    bool submit(uint32_t w, const SourceExtent *ext, int n, uint64_t tag, uint32_t epoch, uint32_t gen);

    struct Done {
        uint32_t window;
        uint64_t tag;
        uint32_t epoch, gen;
        SourceError error;
        int sys_errno;
    };
    // Requests whose reads have all completed since the last call; `current`
    // judges each ticket (false: Stale).  Ready requests leave their window
    // HostReady; failed ones leave it Free.  With wait_ms > 0, blocks until at
    // least one request completes, none is outstanding, or wait_ms passed.
    template <typename Current>
    std::vector<Done> collect(int wait_ms, Current current);

    void set_copying(uint32_t w);      // HostReady -> Copying (the H2D copy was enqueued)
    void set_free(uint32_t w);         // Copying (or HostReady) -> Free
    WindowState state(uint32_t w) const;
    const uint8_t *window(uint32_t w) const { return static_cast<const uint8_t *>(windows_[w]); }
    int free_window() const;           // a Free window, -1 if none
    uint32_t busy_windows() const;     // windows not Free
    uint32_t outstanding() const;      // requests still reading
    SourceStats stats() const;

    // Read through the workers' bounce buffers from now on (what the service
    // switches to by itself when a direct read into a window returns EFAULT).
    void use_bounce_buffers() { bounce_.store(true, std::memory_order_relaxed); }

    // Test hook: the next read of extent `extent` of the request tagged `tag`
    // is cut short, fails with EIO, or is held until release_holds(), which
    // lets go every submitted held read, running or still queued.
    void inject(uint64_t tag, int extent, SourceFault f);
    void release_holds();

private:
    struct Read {
        uint32_t req;          // request slot (= window)
        int extent;
        int fd;
        uint64_t file_off, len;   // covering read
        uint64_t need;            // bytes of the covering read the extent needs
        uint8_t *dst;
        SourceFault fault;
    };
    struct Request {
        uint64_t tag = 0;
        uint32_t epoch = 0, gen = 0;
        int pending = 0;
        SourceError error = SourceError::None;
        int sys_errno = 0;
        bool active = false;
    };
    struct Fault {
        uint64_t tag;
        int extent;
        SourceFault f;
    };

    void worker();

    std::string err_;
    std::vector<int> fds_;
    std::vector<uint64_t> sizes_;
    std::vector<void *> windows_;
    uint64_t window_bytes_ = 0;
    uint32_t inflight_ = 1, align_ = 4096;

    mutable std::mutex mu_;
    std::condition_variable work_cv_, done_cv_, hold_cv_;
    std::deque<Read> queue_;
    std::vector<Request> req_;
    std::vector<WindowState> wstate_;
    std::vector<uint32_t> completed_;     // requests whose last read finished, not yet collected
    std::vector<Fault> faults_;
    uint64_t hold_epoch_ = 0;
    uint32_t depth_ = 0;
    bool stop_ = false, draining_ = false;
    std::atomic<bool> bounce_{false};     // windows refuse direct reads: read via bounce buffers
    SourceStats st_;
    std::vector<std::thread> threads_;
};

template <typename Current>
std::vector<SourceService::Done> SourceService::collect(int wait_ms, Current current)
{
    std::vector<Done> out;
    std::unique_lock<std::mutex> lk(mu_);
    if (wait_ms > 0)
        done_cv_.wait_until(lk, std::chrono::system_clock::now() + std::chrono::milliseconds(wait_ms), [&] {
            if (!completed_.empty())
                return true;
            for (const Request &r : req_)
                if (r.active)
                    return false;
            return true;
        });
    for (uint32_t w : completed_) {
        Request &r = req_[w];
        Done d{w, r.tag, r.epoch, r.gen, r.error, r.sys_errno};
        if (d.error == SourceError::None && !current(r.tag, r.epoch, r.gen))
            d.error = SourceError::Stale;
        r.active = false;
        if (d.error == SourceError::None) {
            wstate_[w] = WindowState::HostReady;
            st_.requests_ready++;
        } else {
            wstate_[w] = WindowState::Free;
            st_.requests_failed++;
            if (d.error == SourceError::Stale)
                st_.requests_stale++;
        }
        out.push_back(d);
    }
    completed_.clear();
    return out;
}

}  // namespace msi
