// source.cpp -- bounded source service (see source.hpp).
#include "source.hpp"

#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <cerrno>
#include <cstdlib>
#include <chrono>
#include <cstring>

namespace msi {

namespace {
constexpr auto HOLD_LIMIT = std::chrono::seconds(30);   // a held read completes by itself after this
constexpr uint64_t BOUNCE_BYTES = 4u << 20;             // per-worker bounce buffer
}

SourceService::SourceService(const std::vector<std::string> &files, const std::vector<void *> &windows,
                             uint64_t window_bytes, uint32_t inflight, uint32_t align, bool allow_buffered)
    : windows_(windows), window_bytes_(window_bytes), inflight_(inflight), align_(align)
{
    if (files.empty())
        { err_ = "no source files"; return; }
    if (windows.empty() || window_bytes == 0)
        { err_ = "no source windows"; return; }
    if (inflight < 1 || inflight > MAX_INFLIGHT)
        { err_ = "in-flight limit must be in [1, 8]"; return; }
    if (align < 512 || (align & (align - 1)) || window_bytes % align)
        { err_ = "alignment must be a power of two >= 512 dividing the window size"; return; }
    for (void *w : windows)
        if (!w || reinterpret_cast<uintptr_t>(w) % align)
            { err_ = "source windows must be non-null and aligned to the direct-I/O block"; return; }
    for (const std::string &f : files) {
        int fd = ::open(f.c_str(), O_RDONLY | O_DIRECT | O_CLOEXEC);
        if (fd >= 0) {
            st_.direct++;
        } else if (allow_buffered && errno == EINVAL) {
            fd = ::open(f.c_str(), O_RDONLY | O_CLOEXEC);
            if (fd >= 0)
                st_.buffered++;
        }
        if (fd < 0) {
            err_ = "cannot open source file " + f + ": " + std::strerror(errno);
            return;
        }
        struct stat sb{};
        if (::fstat(fd, &sb) != 0) {
            err_ = "cannot stat source file " + f;
            ::close(fd);
            return;
        }
        fds_.push_back(fd);
        sizes_.push_back(uint64_t(sb.st_size));
    }
    req_.assign(windows.size(), Request{});
    wstate_.assign(windows.size(), WindowState::Free);
    for (uint32_t i = 0; i < inflight_; ++i)
        threads_.emplace_back([this] { worker(); });
}

SourceService::~SourceService()
{
    {
        std::unique_lock<std::mutex> lk(mu_);
        draining_ = true;               // held reads complete now, and no new read is held
        hold_epoch_++;
        hold_cv_.notify_all();
        // drain: every queued and running read completes
        done_cv_.wait(lk, [&] { return queue_.empty() && depth_ == 0; });
        stop_ = true;
    }
    work_cv_.notify_all();
    for (std::thread &t : threads_)
        t.join();
    for (int fd : fds_)
        ::close(fd);
}

bool SourceService::layout(const SourceExtent *ext, int n, uint64_t *place, uint64_t *physical) const
{
    if (n < 1 || n > MAX_EXTENTS)
        return false;
    uint64_t off = 0, phys = 0;
    for (int i = 0; i < n; ++i) {
        const uint64_t a0 = ext[i].offset / align_ * align_;
        const uint64_t a1 = (ext[i].offset + ext[i].nbytes + align_ - 1) / align_ * align_;
        place[i] = off + (ext[i].offset - a0);
        off += a1 - a0;
        phys += a1 - a0;
    }
    if (physical)
        *physical = phys;
    return off <= window_bytes_;
}

bool SourceService::submit(uint32_t w, const SourceExtent *ext, int n, uint64_t tag, uint32_t epoch, uint32_t gen)
{
    uint64_t place[MAX_EXTENTS], phys = 0;
    if (w >= windows_.size() || !layout(ext, n, place, &phys))
        return false;
    for (int i = 0; i < n; ++i)
        if (ext[i].file >= fds_.size())
            return false;
    std::lock_guard<std::mutex> lk(mu_);
    if (wstate_[w] != WindowState::Free || req_[w].active)
        return false;
    Request &r = req_[w];
    r = Request{tag, epoch, gen, n, SourceError::None, 0, true};
    wstate_[w] = WindowState::Reading;
    st_.requests++;
    uint64_t dst = 0;
    for (int i = 0; i < n; ++i) {
        const uint64_t a0 = ext[i].offset / align_ * align_;
        const uint64_t a1 = (ext[i].offset + ext[i].nbytes + align_ - 1) / align_ * align_;
        Read rd{w, i, fds_[ext[i].file], a0, a1 - a0, ext[i].offset + ext[i].nbytes - a0,
                static_cast<uint8_t *>(windows_[w]) + dst, SourceFault::None};
        for (auto it = faults_.begin(); it != faults_.end(); ++it)
            if (it->tag == tag && it->extent == i) {
                rd.fault = it->f;
                faults_.erase(it);
                break;
            }
        dst += a1 - a0;
        st_.logical_bytes += ext[i].nbytes;
        st_.physical_bytes += a1 - a0;
        st_.padding_bytes += (a1 - a0) - ext[i].nbytes;
        queue_.push_back(rd);
    }
    work_cv_.notify_all();
    return true;
}

// A direct read needs destination pages the kernel can pin; pinned host
// memory that is mapped from a device file (as GPU runtimes' page-locked
// allocations can be) refuses that with EFAULT.  The service then reads
// through a small aligned bounce buffer per worker and copies each piece into
// the window: still no page cache, one host copy more, and at most
// inflight * BOUNCE_BYTES of extra memory.
static uint64_t read_covering(int fd, uint8_t *dst, uint64_t len, uint64_t off, uint8_t *bounce, bool use_bounce,
                              int &err)
{
    uint64_t got = 0;
    err = 0;
    while (got < len) {
        const uint64_t want = use_bounce ? std::min<uint64_t>(BOUNCE_BYTES, len - got) : len - got;
        const ssize_t r = ::pread(fd, use_bounce ? bounce : dst + got, want, off_t(off + got));
        if (r < 0) {
            if (errno == EINTR)
                continue;
            err = errno;
            break;
        }
        if (r == 0)
            break;               // end of file
        if (use_bounce)
            std::memcpy(dst + got, bounce, size_t(r));
        got += uint64_t(r);
    }
    return got;
}

void SourceService::worker()
{
    uint8_t *bounce = static_cast<uint8_t *>(std::aligned_alloc(align_, BOUNCE_BYTES));
    std::unique_lock<std::mutex> lk(mu_);
    for (;;) {
        work_cv_.wait(lk, [&] { return stop_ || !queue_.empty(); });
        if (stop_ && queue_.empty()) {
            lk.unlock();
            std::free(bounce);
            return;
        }
        const bool use_bounce = bounce_.load(std::memory_order_relaxed) && bounce;
        Read rd = queue_.front();
        queue_.pop_front();
        depth_++;
        st_.reads_issued++;
        st_.peak_depth = std::max<uint64_t>(st_.peak_depth, depth_);
        if (rd.fault == SourceFault::Hold && !draining_) {
            const uint64_t e = hold_epoch_;
            // (timed waits take a system-clock deadline: pthread_cond_timedwait)
            hold_cv_.wait_until(lk, std::chrono::system_clock::now() + HOLD_LIMIT, [&] { return hold_epoch_ != e; });
        }
        lk.unlock();
        const auto t0 = std::chrono::steady_clock::now();
        // one covering read; a read may return in pieces, so continue until
        // the length is covered, the file ends, or an error occurs
        uint64_t got = 0;
        int err = 0;
        bool bounced = use_bounce;
        if (rd.fault == SourceFault::Eio) {
            err = EIO;
        } else {
            got = read_covering(rd.fd, rd.dst, rd.len, rd.file_off, bounce, use_bounce, err);
            if (err == EFAULT && !use_bounce && bounce) {
                // the window's pages cannot take a direct read: bounce from now on
                bounce_.store(true, std::memory_order_relaxed);
                bounced = true;
                got = read_covering(rd.fd, rd.dst, rd.len, rd.file_off, bounce, true, err);
            }
            if (rd.fault == SourceFault::Short && got > 0)
                got = rd.need > 1 ? rd.need - 1 : 0;
        }
        const double dt = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
        lk.lock();
        st_.read_seconds += dt;
        st_.reads_completed++;
        st_.bounced += bounced;
        Request &q = req_[rd.req];
        if (err) {
            st_.reads_failed++;
            if (q.error == SourceError::None) {
                q.error = SourceError::Io;
                q.sys_errno = err;
            }
        } else if (got < rd.need) {
            st_.reads_failed++;
            if (q.error == SourceError::None)
                q.error = SourceError::Short;
        }
        depth_--;
        if (--q.pending == 0)
            completed_.push_back(rd.req);
        done_cv_.notify_all();
    }
}

void SourceService::set_copying(uint32_t w)
{
    std::lock_guard<std::mutex> lk(mu_);
    if (w < wstate_.size() && wstate_[w] == WindowState::HostReady)
        wstate_[w] = WindowState::Copying;
}

void SourceService::set_free(uint32_t w)
{
    std::lock_guard<std::mutex> lk(mu_);
    if (w < wstate_.size() && (wstate_[w] == WindowState::Copying || wstate_[w] == WindowState::HostReady))
        wstate_[w] = WindowState::Free;
}

WindowState SourceService::state(uint32_t w) const
{
    std::lock_guard<std::mutex> lk(mu_);
    return w < wstate_.size() ? wstate_[w] : WindowState::Free;
}

int SourceService::free_window() const
{
    std::lock_guard<std::mutex> lk(mu_);
    for (uint32_t w = 0; w < wstate_.size(); ++w)
        if (wstate_[w] == WindowState::Free && !req_[w].active)
            return int(w);
    return -1;
}

uint32_t SourceService::busy_windows() const
{
    std::lock_guard<std::mutex> lk(mu_);
    uint32_t n = 0;
    for (WindowState s : wstate_)
        n += s != WindowState::Free;
    return n;
}

uint32_t SourceService::outstanding() const
{
    std::lock_guard<std::mutex> lk(mu_);
    uint32_t n = 0;
    for (const Request &r : req_)
        n += r.active;
    return n;
}

SourceStats SourceService::stats() const
{
    std::lock_guard<std::mutex> lk(mu_);
    return st_;
}

void SourceService::inject(uint64_t tag, int extent, SourceFault f)
{
    std::lock_guard<std::mutex> lk(mu_);
    faults_.push_back(Fault{tag, extent, f});
}

void SourceService::release_holds()
{
    std::lock_guard<std::mutex> lk(mu_);
    // held reads still queued are let go too: a worker checks the hold under
    // this lock, so every held read is either waiting (woken by the epoch) or
    // not yet taken (its hold cleared here)
    for (Read &r : queue_)
        if (r.fault == SourceFault::Hold)
            r.fault = SourceFault::None;
    hold_epoch_++;
    hold_cv_.notify_all();
}

}  // namespace msi
