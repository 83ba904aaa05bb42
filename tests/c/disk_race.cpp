// Storage-tier thread pool under ThreadSanitizer / AddressSanitizer: built
// with g++ from kvio_disk.cpp alone (host code, no GPU), it runs synchronous
// prefetches and stores, background prefetches polled from another thread
// and cancelled at various points, and checks that complete pages hold the
// bytes a synchronous prefetch of the same pages produced.
#include <fcntl.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#include <atomic>
#include <thread>
#include <vector>

#include "kvio.h"

// kvio_api.cpp (which needs the HIP runtime) provides this in the library.
kvio_status kvio_sched_fail(kvio_status st, const char *) { return st; }

#define CHECK(x)                                                             \
    do {                                                                     \
        if (!(x)) {                                                          \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #x); \
            return 1;                                                        \
        }                                                                    \
    } while (0)

int main(int argc, char **argv) {
    const char *path = argc > 1 ? argv[1] : "disk_race.bin";
    const int32_t L = 3, P = 8;
    const int64_t R = 512, N = 96, page_bytes = int64_t(L) * 2 * P * R;
    std::vector<uint8_t> data(size_t(N * page_bytes));
    uint32_t x = 12345;
    for (auto &b : data) { x = x * 1664525u + 1013904223u; b = uint8_t(x >> 24); }
    int fd = open(path, O_RDWR | O_CREAT | O_TRUNC, 0600);
    CHECK(fd >= 0);
    CHECK(write(fd, data.data(), data.size()) == ssize_t(data.size()));
    std::vector<int64_t> pages;
    for (int64_t p = N - 1; p >= 0; p -= 2) pages.push_back(p);
    pages.push_back(0);
    pages.push_back(2);
    const int32_t n = int32_t(pages.size());
    const int64_t T = int64_t(n) * P;
    const size_t chunk = size_t(L) * 2 * size_t(T) * size_t(R);
    for (int32_t layout = 0; layout < 2; ++layout) {
        kvio_disk_store st = {fd, layout, N, L, P, R};
        for (int32_t host_layout = 0; host_layout < 2; ++host_layout) {
            std::vector<uint8_t> ref(chunk), got(chunk);
            CHECK(kvio_disk_prefetch(&st, pages.data(), n, ref.data(), T, host_layout, 1) == KVIO_OK);
            for (int32_t threads : {1, 3, 8}) {
                for (int stop_after : {-1, 0, 4, 20}) {
                    std::fill(got.begin(), got.end(), uint8_t(0));
                    kvio_prefetch_t job = nullptr;
                    CHECK(kvio_disk_prefetch_start(&st, pages.data(), n, got.data(), T, host_layout, threads, &job) ==
                          KVIO_OK);
                    std::atomic<bool> stop{false};
                    std::thread poller([&] {
                        int32_t d = 0;
                        while (!stop.load()) {
                            if (kvio_disk_prefetch_progress(job, &d) != KVIO_OK || d < 0 || d > n) abort();
                            std::this_thread::yield();
                        }
                    });
                    int32_t d = 0;
                    while (stop_after > 0 && d < stop_after) {
                        CHECK(kvio_disk_prefetch_progress(job, &d) == KVIO_OK);
                        if (d >= n) break;
                    }
                    stop.store(true);
                    poller.join();
                    std::vector<uint8_t> done(static_cast<size_t>(n));
                    int32_t n_done = -1;
                    CHECK(kvio_disk_prefetch_finish(job, stop_after >= 0, done.data(), &n_done) == KVIO_OK);
                    int32_t count = 0;
                    for (int32_t j = 0; j < n; ++j) count += done[size_t(j)];
                    CHECK(count == n_done);
                    if (stop_after < 0) CHECK(n_done == n);
                    if (stop_after > 0) CHECK(n_done >= stop_after);
                    if (n_done == n) CHECK(memcmp(got.data(), ref.data(), chunk) == 0);
                }
            }
            // store the chunk back under other pages, then read it again
            std::vector<int64_t> back(pages.rbegin(), pages.rend());
            CHECK(kvio_disk_store_pages(&st, back.data(), n, ref.data(), T, host_layout, 4) == KVIO_OK);
            std::vector<uint8_t> again(chunk);
            CHECK(kvio_disk_prefetch(&st, back.data(), n, again.data(), T, host_layout, 4) == KVIO_OK);
            CHECK(memcmp(again.data(), ref.data(), chunk) == 0);
            CHECK(pwrite(fd, data.data(), data.size(), 0) == ssize_t(data.size()));
        }
    }
    close(fd);
    unlink(path);
    printf("disk race checks passed\n");
    return 0;
}
