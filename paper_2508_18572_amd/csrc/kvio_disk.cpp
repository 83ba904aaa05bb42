// kvio_disk.cpp -- storage tier of the paged-KV cache (Strata Sec. 4.2.1):
// whole-page transfers between a disk store and a pinned host chunk, as
// parallel positioned reads / writes of merged contiguous pieces.
#include <errno.h>
#include <fcntl.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#include <algorithm>
#include <memory>
#include <new>
#include <system_error>
#include <atomic>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "kvio.h"

kvio_status kvio_sched_fail(kvio_status st, const char *msg);   // kvio_api.cpp

namespace {

// One transfer of `len` bytes between the file at file_off and the host chunk
// at host_off.  Pieces of one page are whole (page, layer, K|V) runs or whole
// pages; merging joins pieces contiguous on both sides, which may belong to
// different context pages, so every piece keeps its pages as `parts`.
struct Piece {
    int64_t file_off;
    int64_t host_off;
    int64_t len;
    int32_t part_begin, part_end;   // [begin, end) into Job::parts, in host order
};

struct Part {
    int32_t page;                   // context page index
    int64_t len;
};

kvio_status build(const kvio_disk_store *st, const int64_t *pages, int32_t n, int64_t host_tokens,
                  int32_t host_layout, std::vector<Piece> *out, std::vector<Part> *parts, const char *fn,
                  std::string *err) {
    if (st == nullptr || n < 0 || (n > 0 && pages == nullptr)) { *err = std::string(fn) + ": null argument"; return KVIO_EINVAL; }
    if (st->fd < 0 || st->num_layers < 1 || st->page_size < 1 || st->row_bytes < 1 || st->num_disk_pages < 0 ||
        (st->disk_layout != KVIO_DISK_PAGE_FIRST && st->disk_layout != KVIO_DISK_LAYER_FIRST)) {
        *err = std::string(fn) + ": bad disk store"; return KVIO_EINVAL;
    }
    if (host_layout != KVIO_HOST_TOKEN_MAJOR && host_layout != KVIO_HOST_PAGE_FIRST) {
        *err = std::string(fn) + ": host layout must be token-major or page-first"; return KVIO_EINVAL;
    }
    const int64_t L = st->num_layers, P = st->page_size, R = st->row_bytes;
    if (host_tokens < int64_t(n) * P) { *err = std::string(fn) + ": host_tokens below n_pages * page_size"; return KVIO_EINVAL; }
    if (host_layout == KVIO_HOST_PAGE_FIRST && host_tokens % P != 0) {
        *err = std::string(fn) + ": page-first chunks hold whole pages"; return KVIO_EINVAL;
    }
    struct Raw { int64_t file_off, host_off, len; int32_t page; };
    std::vector<Raw> raw;
    const bool whole = st->disk_layout == KVIO_DISK_PAGE_FIRST && host_layout == KVIO_HOST_PAGE_FIRST;
    raw.reserve(size_t(n) * (whole ? 1 : size_t(2 * L)));
    const int64_t seg = P * R;                    // one (page, layer, K|V) run
    for (int32_t j = 0; j < n; ++j) {
        const int64_t p = pages[j];
        if (p < 0 || p >= st->num_disk_pages) { *err = std::string(fn) + ": disk page out of range"; return KVIO_EINVAL; }
        if (whole) {
            raw.push_back({p * L * 2 * seg, int64_t(j) * L * 2 * seg, L * 2 * seg, j});
            continue;
        }
        for (int64_t l = 0; l < L; ++l) {
            for (int64_t kv = 0; kv < 2; ++kv) {
                const int64_t f = st->disk_layout == KVIO_DISK_PAGE_FIRST ? ((p * L + l) * 2 + kv) * seg
                                                                          : ((l * 2 + kv) * st->num_disk_pages + p) * seg;
                const int64_t h = host_layout == KVIO_HOST_PAGE_FIRST ? ((int64_t(j) * L + l) * 2 + kv) * seg
                                                                      : ((l * 2 + kv) * host_tokens + int64_t(j) * P) * R;
                raw.push_back({f, h, seg, j});
            }
        }
    }
    // Merge pieces contiguous on both sides (e.g. consecutive disk pages).
    std::sort(raw.begin(), raw.end(), [](const Raw &a, const Raw &b) { return a.host_off < b.host_off; });
    out->clear();
    parts->clear();
    parts->reserve(raw.size());
    for (const Raw &x : raw) {
        if (!out->empty() && out->back().host_off + out->back().len == x.host_off &&
            out->back().file_off + out->back().len == x.file_off) {
            out->back().len += x.len;
        } else {
            const int32_t at = int32_t(parts->size());
            out->push_back({x.file_off, x.host_off, x.len, at, at});
        }
        parts->push_back({x.page, x.len});
        out->back().part_end = int32_t(parts->size());
    }
    return KVIO_OK;
}

// Host memory the kernel cannot pin for direct I/O (the HIP runtime's pinned
// allocations are device-file mappings) makes an O_DIRECT transfer fail with
// EFAULT.  On O_DIRECT descriptors such transfers are staged through an
// aligned bounce buffer per worker thread instead.
constexpr size_t kBounceBytes = size_t(16) << 20;

struct Bounce {
    uint8_t *p = nullptr;
    ~Bounce() { free(p); }
    bool ready() { return p != nullptr || posix_memalign(reinterpret_cast<void **>(&p), 4096, kBounceBytes) == 0; }
};

// One transfer of up to len bytes between host + off and the file at file_off;
// returns what pread/pwrite return.
ssize_t transfer(int fd, uint8_t *host, int64_t len, int64_t file_off, bool to_host, Bounce *bounce) {
    if (bounce == nullptr)
        return to_host ? pread(fd, host, size_t(len), file_off) : pwrite(fd, host, size_t(len), file_off);
    const size_t n = std::min<size_t>(size_t(len), kBounceBytes);
    if (to_host) {
        const ssize_t r = pread(fd, bounce->p, n, file_off);
        if (r > 0) memcpy(host, bounce->p, size_t(r));
        return r;
    }
    memcpy(bounce->p, host, n);
    return pwrite(fd, bounce->p, n, file_off);
}

}  // namespace

// A set of page transfers run by worker threads.  Every page counts its bytes
// still to move; a page is complete when its count reaches zero.  Workers
// stop taking work after a failure or a cancellation request, at the next
// transfer boundary (at most one piece, or one bounce buffer, per worker).
struct kvio_prefetch {
    int fd = -1;
    bool direct = false;
    bool to_host = true;
    uint8_t *host = nullptr;
    const char *fn = "";
    std::vector<Piece> pieces;
    std::vector<Part> parts;
    int32_t n_pages = 0;
    std::unique_ptr<std::atomic<int64_t>[]> remaining;
    std::atomic<size_t> next{0};
    std::atomic<int> failed{0};
    std::atomic<bool> staged{false};   // set once a direct transfer reported EFAULT
    std::atomic<bool> cancel{false};
    std::mutex mu;
    std::string err;
    std::vector<std::thread> workers;

    void fail(const std::string &why) {
        std::lock_guard<std::mutex> g(mu);
        if (!failed.exchange(1)) err = std::string(fn) + ": " + why;
    }

    void work() {
        Bounce bounce;
        for (;;) {
            const size_t i = next.fetch_add(1);
            if (i >= pieces.size() || failed.load() || cancel.load()) return;
            const Piece &pc = pieces[i];
            int64_t done = 0, credited = 0;
            int32_t part = pc.part_begin;
            while (done < pc.len) {
                if (cancel.load()) return;
                Bounce *b = nullptr;
                if (staged.load()) {
                    if (!bounce.ready()) return fail("cannot allocate a bounce buffer");
                    b = &bounce;
                }
                const ssize_t r = transfer(fd, host + pc.host_off + done, pc.len - done, pc.file_off + done, to_host, b);
                if (r < 0 && errno == EINTR) continue;
                if (r < 0 && errno == EFAULT && direct && b == nullptr) {
                    staged.store(true);
                    continue;
                }
                if (r <= 0) return fail(r < 0 ? std::string(strerror(errno)) : std::string("short transfer at end of file"));
                done += r;
                // credit the parts this piece has now covered in full
                while (part < pc.part_end && credited + parts[size_t(part)].len <= done) {
                    credited += parts[size_t(part)].len;
                    remaining[size_t(parts[size_t(part)].page)].fetch_sub(parts[size_t(part)].len);
                    ++part;
                }
            }
        }
    }

    int32_t pages_done() const {
        int32_t c = 0;
        for (int32_t j = 0; j < n_pages; ++j) c += remaining[size_t(j)].load() == 0;
        return c;
    }
};

namespace {

kvio_status start(const kvio_disk_store *store, const int64_t *disk_pages, int32_t n_pages, uint8_t *host,
                  int64_t host_tokens, int32_t host_layout, int32_t threads, bool to_host, const char *fn,
                  kvio_prefetch **out, std::string *err) {
    std::unique_ptr<kvio_prefetch> job(new (std::nothrow) kvio_prefetch());
    if (!job) { *err = std::string(fn) + ": out of host memory"; return KVIO_ENOMEM; }
    kvio_status st = build(store, disk_pages, n_pages, host_tokens, host_layout, &job->pieces, &job->parts, fn, err);
    if (st != KVIO_OK) return st;
    if (n_pages > 0 && host == nullptr) { *err = std::string(fn) + ": null host chunk"; return KVIO_EINVAL; }
    const int fl = fcntl(store->fd, F_GETFL);
    if (fl < 0) { *err = std::string(fn) + ": bad file descriptor"; return KVIO_EINVAL; }
    job->fd = store->fd;
    job->direct = (fl & O_DIRECT) != 0;
    job->to_host = to_host;
    job->host = host;
    job->fn = fn;
    job->n_pages = n_pages;
    job->remaining.reset(new std::atomic<int64_t>[size_t(std::max(n_pages, 1))]);
    const int64_t page_bytes = int64_t(store->num_layers) * 2 * store->page_size * store->row_bytes;
    for (int32_t j = 0; j < n_pages; ++j) job->remaining[size_t(j)].store(page_bytes);
    const int32_t nt = std::max<int32_t>(1, std::min<int32_t>(threads, int32_t(job->pieces.size())));
    try {
        for (int32_t t = 0; t < nt && !job->pieces.empty(); ++t) job->workers.emplace_back(&kvio_prefetch::work, job.get());
    } catch (const std::system_error &) {
        job->cancel.store(true);
        for (auto &w : job->workers) w.join();
        *err = std::string(fn) + ": cannot start worker threads";
        return KVIO_ENOMEM;
    }
    *out = job.release();
    return KVIO_OK;
}

kvio_status finish(kvio_prefetch *job, bool cancel, uint8_t *page_done, int32_t *pages_done, std::string *err) {
    if (cancel) job->cancel.store(true);
    for (auto &w : job->workers) w.join();
    if (page_done != nullptr)
        for (int32_t j = 0; j < job->n_pages; ++j) page_done[j] = job->remaining[size_t(j)].load() == 0;
    if (pages_done != nullptr) *pages_done = job->pages_done();
    const kvio_status st = job->failed.load() ? KVIO_EIO : KVIO_OK;
    if (st != KVIO_OK) *err = job->err;
    delete job;
    return st;
}

kvio_status run_sync(const kvio_disk_store *store, const int64_t *disk_pages, int32_t n_pages, uint8_t *host,
                     int64_t host_tokens, int32_t host_layout, int32_t threads, bool to_host, const char *fn) {
    std::string err;
    kvio_prefetch *job = nullptr;
    kvio_status st = start(store, disk_pages, n_pages, host, host_tokens, host_layout, threads, to_host, fn, &job, &err);
    if (st == KVIO_OK) st = finish(job, false, nullptr, nullptr, &err);
    return st == KVIO_OK ? kvio_sched_fail(KVIO_OK, "") : kvio_sched_fail(st, err.c_str());
}

}  // namespace

extern "C" kvio_status kvio_disk_prefetch(const kvio_disk_store *store, const int64_t *disk_pages, int32_t n_pages,
                                          void *host, int64_t host_tokens, int32_t host_layout, int32_t threads) {
    return run_sync(store, disk_pages, n_pages, static_cast<uint8_t *>(host), host_tokens, host_layout, threads, true,
                    "kvio_disk_prefetch");
}

extern "C" kvio_status kvio_disk_store_pages(const kvio_disk_store *store, const int64_t *disk_pages, int32_t n_pages,
                                             const void *host, int64_t host_tokens, int32_t host_layout,
                                             int32_t threads) {
    return run_sync(store, disk_pages, n_pages, const_cast<uint8_t *>(static_cast<const uint8_t *>(host)), host_tokens,
                    host_layout, threads, false, "kvio_disk_store_pages");
}

extern "C" kvio_status kvio_disk_prefetch_start(const kvio_disk_store *store, const int64_t *disk_pages,
                                                int32_t n_pages, void *host, int64_t host_tokens, int32_t host_layout,
                                                int32_t threads, kvio_prefetch_t *out) {
    if (out == nullptr) return kvio_sched_fail(KVIO_EINVAL, "kvio_disk_prefetch_start: null handle pointer");
    *out = nullptr;
    std::string err;
    const kvio_status st = start(store, disk_pages, n_pages, static_cast<uint8_t *>(host), host_tokens, host_layout,
                                 threads, true, "kvio_disk_prefetch_start", out, &err);
    return st == KVIO_OK ? kvio_sched_fail(KVIO_OK, "") : kvio_sched_fail(st, err.c_str());
}

extern "C" kvio_status kvio_disk_prefetch_progress(kvio_prefetch_t job, int32_t *pages_done) {
    if (job == nullptr || pages_done == nullptr)
        return kvio_sched_fail(KVIO_EINVAL, "kvio_disk_prefetch_progress: null argument");
    *pages_done = job->pages_done();
    return kvio_sched_fail(KVIO_OK, "");
}

extern "C" kvio_status kvio_disk_prefetch_finish(kvio_prefetch_t job, int32_t cancel, uint8_t *page_done,
                                                 int32_t *pages_done) {
    if (job == nullptr) return kvio_sched_fail(KVIO_EINVAL, "kvio_disk_prefetch_finish: null handle");
    std::string err;
    const kvio_status st = finish(job, cancel != 0, page_done, pages_done, &err);
    return st == KVIO_OK ? kvio_sched_fail(KVIO_OK, "") : kvio_sched_fail(st, err.c_str());
}
