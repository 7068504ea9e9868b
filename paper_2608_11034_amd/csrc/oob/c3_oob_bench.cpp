// Cost of the progress path of out-of-band hang localization (Sec. 7):
// nanoseconds per publication (the only work the trainer does), per
// snapshot while idle and while a second thread publishes continuously,
// and per classification of a 64-rank record table.  Prints one JSON
// object.  Usage: c3_oob_bench [iterations]
#include <stdio.h>
#include <stdlib.h>
#include <time.h>
#include <unistd.h>

#include <atomic>
#include <thread>

#include "../../../include/c3_oob.h"

static double now_s() {
    timespec ts;
    clock_gettime(CLOCK_MONOTONIC, &ts);
    return (double)ts.tv_sec + 1e-9 * (double)ts.tv_nsec;
}

int main(int argc, char** argv) {
    const long iters = argc > 1 ? atol(argv[1]) : 2000000;
    char name[64];
    snprintf(name, sizeof(name), "/c3_oob_bench_%d", (int)getpid());
    c3_progress_seg_t* seg = nullptr;
    if (c3_progress_open(name, 2, 1, &seg) != C3_OOB_OK) {
        fprintf(stderr, "c3_progress_open failed\n");
        return 1;
    }
    // publication, single writer, nothing reading
    double t0 = now_s();
    for (long i = 0; i < iters; ++i) c3_progress_publish(seg, 0, (uint64_t)i, 3, 0x1234, 1);
    const double pub_ns = (now_s() - t0) / (double)iters * 1e9;
    // snapshot, idle writer
    c3_progress_t p;
    uint64_t sink = 0;
    t0 = now_s();
    for (long i = 0; i < iters; ++i) {
        c3_progress_read(seg, 0, &p);
        sink += p.step;
    }
    const double read_ns = (now_s() - t0) / (double)iters * 1e9;
    // snapshot while another thread publishes back to back into the same slot
    std::atomic<bool> stop(false);
    std::atomic<long> published(0);
    std::thread w([&] {
        long n = 0;
        while (!stop.load(std::memory_order_relaxed)) {
            c3_progress_publish(seg, 1, (uint64_t)n, (uint64_t)(3 * n + 1), 0x5678, 0);
            ++n;
        }
        published.store(n);
    });
    long torn = 0, busy = 0;
    t0 = now_s();
    for (long i = 0; i < iters; ++i) {
        const int rc = c3_progress_read(seg, 1, &p);
        if (rc != C3_OOB_OK) {
            ++busy;
            continue;
        }
        if (p.publishes != 0 && p.op_id != 3 * p.step + 1) ++torn;
    }
    const double t_read = now_s() - t0;
    stop.store(true);
    w.join();
    const double read_contended_ns = t_read / (double)iters * 1e9;
    // classification of 64 gathered records
    c3_progress_t recs[64];
    for (int i = 0; i < 64; ++i) {
        recs[i] = p;
        recs[i].step = i == 17 ? 41 : 42;
    }
    c3_hang_verdict_t v;
    const long citers = iters / 20 + 1;
    t0 = now_s();
    for (long i = 0; i < citers; ++i) {
        recs[5].op_id = (uint64_t)i;
        c3_hang_classify(recs, 64, &v);
        sink += v.bitmap;
    }
    const double classify_ns = (now_s() - t0) / (double)citers * 1e9;
    c3_progress_close(seg, 1);
    printf("{\"publish_ns\": %.1f, \"read_ns\": %.1f, \"read_contended_ns\": %.1f, "
           "\"contended_reads\": %ld, \"torn\": %ld, \"busy\": %ld, \"writer_publications\": %ld, "
           "\"classify_64_ranks_ns\": %.1f, \"iterations\": %ld, \"sink\": %llu}\n",
           pub_ns, read_ns, read_contended_ns, iters, torn, busy, published.load(), classify_ns,
           iters, (unsigned long long)(sink & 1));
    return torn == 0 ? 0 : 2;
}
