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
#include <atomic>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "kvio.h"

kvio_status kvio_sched_fail(kvio_status st, const char *msg);   // kvio_api.cpp

namespace {

struct Piece {
    int64_t file_off;
    int64_t host_off;
    int64_t len;
};

kvio_status build(const kvio_disk_store *st, const int64_t *pages, int32_t n, int64_t host_tokens,
                  int32_t host_layout, std::vector<Piece> *out, const char *fn, std::string *err) {
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
    out->clear();
    out->reserve(size_t(n) * (st->disk_layout == KVIO_DISK_PAGE_FIRST && host_layout == KVIO_HOST_PAGE_FIRST
                                  ? 1 : size_t(2 * L)));
    const int64_t seg = P * R;                    // one (page, layer, K|V) run
    for (int32_t j = 0; j < n; ++j) {
        const int64_t p = pages[j];
        if (p < 0 || p >= st->num_disk_pages) { *err = std::string(fn) + ": disk page out of range"; return KVIO_EINVAL; }
        if (st->disk_layout == KVIO_DISK_PAGE_FIRST && host_layout == KVIO_HOST_PAGE_FIRST) {
            out->push_back({p * L * 2 * seg, int64_t(j) * L * 2 * seg, L * 2 * seg});
            continue;
        }
        for (int64_t l = 0; l < L; ++l) {
            for (int64_t kv = 0; kv < 2; ++kv) {
                const int64_t f = st->disk_layout == KVIO_DISK_PAGE_FIRST ? ((p * L + l) * 2 + kv) * seg
                                                                          : ((l * 2 + kv) * st->num_disk_pages + p) * seg;
                const int64_t h = host_layout == KVIO_HOST_PAGE_FIRST ? ((int64_t(j) * L + l) * 2 + kv) * seg
                                                                      : ((l * 2 + kv) * host_tokens + int64_t(j) * P) * R;
                out->push_back({f, h, seg});
            }
        }
    }
    // Merge pieces contiguous on both sides (e.g. consecutive disk pages).
    std::sort(out->begin(), out->end(), [](const Piece &a, const Piece &b) { return a.host_off < b.host_off; });
    std::vector<Piece> merged;
    merged.reserve(out->size());
    for (const Piece &x : *out) {
        if (!merged.empty() && merged.back().host_off + merged.back().len == x.host_off &&
            merged.back().file_off + merged.back().len == x.file_off)
            merged.back().len += x.len;
        else
            merged.push_back(x);
    }
    out->swap(merged);
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

kvio_status run(int fd, const std::vector<Piece> &pieces, uint8_t *host, bool to_host, int32_t threads,
                const char *fn, std::string *err) {
    const int fl = fcntl(fd, F_GETFL);
    if (fl < 0) {
        *err = std::string(fn) + ": bad file descriptor";
        return KVIO_EINVAL;
    }
    const bool direct = (fl & O_DIRECT) != 0;
    std::atomic<size_t> next{0};
    std::atomic<int> failed{0};
    std::atomic<bool> staged{false};   // set once a direct transfer reported EFAULT
    std::mutex mu;
    auto fail = [&](const std::string &why) {
        std::lock_guard<std::mutex> g(mu);
        if (!failed.exchange(1)) *err = std::string(fn) + ": " + why;
    };
    auto worker = [&]() {
        Bounce bounce;
        for (;;) {
            const size_t i = next.fetch_add(1);
            if (i >= pieces.size() || failed.load()) return;
            const Piece &pc = pieces[i];
            int64_t done = 0;
            while (done < pc.len) {
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
            }
        }
    };
    const int32_t nt = std::max<int32_t>(1, std::min<int32_t>(threads, int32_t(pieces.size())));
    std::vector<std::thread> pool;
    for (int32_t t = 1; t < nt; ++t) pool.emplace_back(worker);
    worker();
    for (auto &t : pool) t.join();
    return failed.load() ? KVIO_EIO : KVIO_OK;
}

}  // namespace

extern "C" kvio_status kvio_disk_prefetch(const kvio_disk_store *store, const int64_t *disk_pages, int32_t n_pages,
                                          void *host, int64_t host_tokens, int32_t host_layout, int32_t threads) {
    std::vector<Piece> pieces;
    std::string err;
    kvio_status st = build(store, disk_pages, n_pages, host_tokens, host_layout, &pieces, "kvio_disk_prefetch", &err);
    if (st == KVIO_OK && n_pages > 0 && host == nullptr) { st = KVIO_EINVAL; err = "kvio_disk_prefetch: null host chunk"; }
    if (st == KVIO_OK) st = run(store->fd, pieces, static_cast<uint8_t *>(host), true, threads, "kvio_disk_prefetch", &err);
    return st == KVIO_OK ? kvio_sched_fail(KVIO_OK, "") : kvio_sched_fail(st, err.c_str());
}

extern "C" kvio_status kvio_disk_store_pages(const kvio_disk_store *store, const int64_t *disk_pages, int32_t n_pages,
                                             const void *host, int64_t host_tokens, int32_t host_layout,
                                             int32_t threads) {
    std::vector<Piece> pieces;
    std::string err;
    kvio_status st = build(store, disk_pages, n_pages, host_tokens, host_layout, &pieces, "kvio_disk_store_pages", &err);
    if (st == KVIO_OK && n_pages > 0 && host == nullptr) { st = KVIO_EINVAL; err = "kvio_disk_store_pages: null host chunk"; }
    if (st == KVIO_OK)
        st = run(store->fd, pieces, const_cast<uint8_t *>(static_cast<const uint8_t *>(host)), false, threads,
                 "kvio_disk_store_pages", &err);
    return st == KVIO_OK ? kvio_sched_fail(KVIO_OK, "") : kvio_sched_fail(st, err.c_str());
}
