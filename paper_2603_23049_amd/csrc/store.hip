// SSD tier of the KV-chunk cache: an asynchronous chunk store (Sec. 4.4: the
// prefetcher loads chunks of waiting requests from SSD into DRAM without blocking
// the serving loop, and newly computed chunks are written back to SSD
// asynchronously; Sec. 5: a dedicated prefetch thread).
//
// Host code only. One file holds every chunk at offset chunk_id * chunk_bytes. A
// pool of I/O threads serves a FIFO of read and write tasks with positional I/O
// (pread/pwrite), opening the file with O_DIRECT when the chunk size and the
// caller's buffers are page-aligned, so reads measure the device rather than the
// page cache. Completion is tracked per chunk id. Tasks of one chunk run one at a
// time in submission order: submitting a read or a write of a chunk first waits
// (in the submitting thread) until every earlier task of that chunk is done, so
// with several I/O threads a read never sees a half-written chunk and two writes
// of a chunk land in the order they were submitted. Tasks of different chunks
// run concurrently.
#include <errno.h>
#include <stdio.h>
#include <fcntl.h>
#include <string.h>
#include <sys/stat.h>
#include <unistd.h>

#include <condition_variable>
#include <deque>
#include <mutex>
#include <thread>
#include <unordered_map>
#include <vector>

#include "pcr_internal.h"

struct pcr_chunk_store {
    int fd = -1;
    int fd_direct = -1;
    int64_t chunk_bytes = 0;
    std::mutex mu;
    std::condition_variable cv_task, cv_done;
    struct Task {
        bool write;
        int64_t id;
        void *buf;
    };
    std::deque<Task> queue;
    std::unordered_map<int64_t, int> pending;     // outstanding tasks per chunk id
    std::unordered_map<int64_t, int64_t> written;  // chunk ids on the device (value unused)
    int64_t total_pending = 0;
    int io_errors = 0;
    char first_error[256] = "";
    bool stop = false;
    std::vector<std::thread> workers;
    int64_t bytes_read = 0, bytes_written = 0;
    int64_t direct_fallbacks = 0;   // transfers that O_DIRECT refused and the page cache served
};

namespace {

bool page_aligned(const void *p, int64_t n)
{
    const long pg = sysconf(_SC_PAGESIZE);
    return ((uintptr_t)p % (uintptr_t)pg) == 0 && n % pg == 0;
}

// Full positional transfer (loops over short reads and writes).
bool xfer(int fd, bool write, void *buf, int64_t n, int64_t off)
{
    char *p = static_cast<char *>(buf);
    while (n > 0) {
        const ssize_t r = write ? pwrite(fd, p, (size_t)n, off) : pread(fd, p, (size_t)n, off);
        if (r < 0 && errno == EINTR) continue;
        if (r <= 0) return false;
        p += r;
        off += r;
        n -= r;
    }
    return true;
}

void worker(pcr_chunk_store *st)
{
    for (;;) {
        pcr_chunk_store::Task t;
        {
            std::unique_lock<std::mutex> lk(st->mu);
            st->cv_task.wait(lk, [&] { return st->stop || !st->queue.empty(); });
            if (st->queue.empty()) return;            // stop requested and nothing left
            t = st->queue.front();
            st->queue.pop_front();
        }
        const int64_t off = t.id * st->chunk_bytes;
        const int fd = (st->fd_direct >= 0 && page_aligned(t.buf, st->chunk_bytes)) ? st->fd_direct : st->fd;
        bool ok = xfer(fd, t.write, t.buf, st->chunk_bytes, off);
        int err = errno;
        bool fell_back = false;
        if (!ok && fd == st->fd_direct && (err == EFAULT || err == EINVAL)) {
            // Direct I/O pins the buffer's pages, which fails for host memory the GPU driver
            // mapped (pinned memory from hipHostMalloc): such buffers go through the page
            // cache instead (the kernel keeps the two kinds of access to the file coherent).
            ok = xfer(st->fd, t.write, t.buf, st->chunk_bytes, off);
            err = errno;
            fell_back = true;
        }
        {
            std::lock_guard<std::mutex> lk(st->mu);
            st->direct_fallbacks += fell_back;
            if (!ok) {
                if (!st->io_errors++)
                    snprintf(st->first_error, sizeof st->first_error, "%s of chunk %lld failed: %s",
                             t.write ? "write" : "read", (long long)t.id, strerror(err));
            } else if (t.write) {
                st->written[t.id] = 1;
                st->bytes_written += st->chunk_bytes;
            } else {
                st->bytes_read += st->chunk_bytes;
            }
            if (--st->pending[t.id] == 0) st->pending.erase(t.id);
            --st->total_pending;
        }
        st->cv_done.notify_all();
    }
}

pcr_status submit(pcr_chunk_store *st, bool write, int64_t id, void *buf, const char *who)
{
    if (!st) return pcr::fail(PCR_ERR_INVALID_ARG, "%s: NULL store", who);
    if (id < 0) return pcr::fail(PCR_ERR_INVALID_ARG, "%s: negative chunk id", who);
    if (!buf) return pcr::fail(PCR_ERR_INVALID_ARG, "%s: NULL buffer", who);
    if (id > INT64_MAX / st->chunk_bytes - 1) return pcr::fail(PCR_ERR_INVALID_ARG, "%s: chunk id too large", who);
    std::unique_lock<std::mutex> lk(st->mu);
    // One task per chunk at a time: wait for the chunk's earlier reads and writes.
    st->cv_done.wait(lk, [&] { return st->pending.find(id) == st->pending.end(); });
    if (!write && st->written.find(id) == st->written.end())
        return pcr::fail(PCR_ERR_INVALID_ARG, "%s: chunk %lld was never written", who, (long long)id);
    st->queue.push_back({write, id, buf});
    ++st->pending[id];
    ++st->total_pending;
    lk.unlock();
    st->cv_task.notify_one();
    return PCR_OK;
}

}  // namespace

extern "C" {

pcr_status pcr_store_open(const char *path, int64_t chunk_bytes, int32_t io_threads, pcr_chunk_store **out)
{
    const char *who = "pcr_store_open";
    if (!out) return pcr::fail(PCR_ERR_INVALID_ARG, "%s: NULL out", who);
    *out = nullptr;
    if (!path || chunk_bytes <= 0 || io_threads <= 0 || io_threads > 64)
        return pcr::fail(PCR_ERR_INVALID_ARG, "%s: bad path, chunk size or thread count", who);
    auto *st = new pcr_chunk_store();
    st->chunk_bytes = chunk_bytes;
    st->fd = open(path, O_RDWR | O_CREAT | O_TRUNC, 0600);
    if (st->fd < 0) {
        pcr::fail(PCR_ERR_INVALID_ARG, "%s: cannot open %s: %s", who, path, strerror(errno));
        delete st;
        return PCR_ERR_INVALID_ARG;
    }
    if (chunk_bytes % sysconf(_SC_PAGESIZE) == 0) st->fd_direct = open(path, O_RDWR | O_DIRECT);
    for (int i = 0; i < io_threads; ++i) st->workers.emplace_back(worker, st);
    *out = st;
    return PCR_OK;
}

pcr_status pcr_store_write_async(pcr_chunk_store *st, int64_t chunk_id, const void *src)
{
    return submit(st, true, chunk_id, const_cast<void *>(src), "pcr_store_write_async");
}

pcr_status pcr_store_read_async(pcr_chunk_store *st, int64_t chunk_id, void *dst)
{
    return submit(st, false, chunk_id, dst, "pcr_store_read_async");
}

pcr_status pcr_store_wait(pcr_chunk_store *st, int64_t chunk_id)
{
    if (!st) return pcr::fail(PCR_ERR_INVALID_ARG, "pcr_store_wait: NULL store");
    std::unique_lock<std::mutex> lk(st->mu);
    if (chunk_id < 0)
        st->cv_done.wait(lk, [&] { return st->total_pending == 0; });
    else
        st->cv_done.wait(lk, [&] { return st->pending.find(chunk_id) == st->pending.end(); });
    if (st->io_errors) return pcr::fail(PCR_ERR_INVALID_ARG, "pcr_store: %s", st->first_error);
    return PCR_OK;
}

pcr_status pcr_store_poll(pcr_chunk_store *st, int64_t chunk_id, int32_t *done)
{
    if (!st || !done) return pcr::fail(PCR_ERR_INVALID_ARG, "pcr_store_poll: NULL argument");
    std::lock_guard<std::mutex> lk(st->mu);
    *done = chunk_id < 0 ? st->total_pending == 0 : st->pending.find(chunk_id) == st->pending.end();
    return PCR_OK;
}

pcr_status pcr_store_stats(pcr_chunk_store *st, int64_t *bytes_read, int64_t *bytes_written, int32_t *direct,
                           int64_t *direct_fallbacks)
{
    if (!st) return pcr::fail(PCR_ERR_INVALID_ARG, "pcr_store_stats: NULL store");
    std::lock_guard<std::mutex> lk(st->mu);
    if (bytes_read) *bytes_read = st->bytes_read;
    if (bytes_written) *bytes_written = st->bytes_written;
    if (direct) *direct = st->fd_direct >= 0;
    if (direct_fallbacks) *direct_fallbacks = st->direct_fallbacks;
    return PCR_OK;
}

pcr_status pcr_store_close(pcr_chunk_store *st)
{
    if (!st) return PCR_OK;
    {
        std::lock_guard<std::mutex> lk(st->mu);
        st->stop = true;
    }
    st->cv_task.notify_all();
    for (auto &t : st->workers) t.join();           // the queue drains before the workers exit
    const int errs = st->io_errors;
    if (st->fd_direct >= 0) close(st->fd_direct);
    if (st->fd >= 0) close(st->fd);
    delete st;
    return errs ? pcr::fail(PCR_ERR_INVALID_ARG, "pcr_store_close: %d I/O errors", errs) : PCR_OK;
}

}  // extern "C"
