// Host stress driver for the coordinator on the simulated device (FAKE backend), built with a
// host sanitizer (thread or address) by tests/test_sanitizers.py.  No GPU is touched: ops are
// created over placeholder device addresses and only the simulated backend launches.
//
// Threads: several submitters (critical and normal requests, some timed), a poller, a reader
// of statistics and the launch log, all running against the dispatcher thread; then a drain,
// a shutdown, and a second coordinator whose fifth launch fails (the failure path ends one
// request and clears its ops' counters).  Exits 0 when every request completed exactly once.
#include <atomic>
#include <cstdio>
#include <cstring>
#include <thread>
#include <vector>

#include "miriam.h"

static miriam_op *make_gemm(int tiles) {
    miriam_op_desc d;
    std::memset(&d, 0, sizeof(d));
    d.kind = MIRIAM_OP_GEMM;
    d.dtype = MIRIAM_F16;
    d.m = 64 * tiles;
    d.nn = 64;
    d.kk = 64;
    d.tile = 2;
    const uintptr_t fake = 0x100000;
    d.x = reinterpret_cast<const void *>(fake);
    d.wt = reinterpret_cast<const void *>(fake);
    d.y = reinterpret_cast<void *>(fake);
    miriam_op *op = nullptr;
    if (miriam_op_create(&d, &op) != MIRIAM_OK) {
        std::fprintf(stderr, "op create: %s\n", miriam_last_error());
        return nullptr;
    }
    return op;
}

static miriam_config base_config(int policy, int fail_at) {
    miriam_config c;
    std::memset(&c, 0, sizeof(c));
    c.policy = policy;
    c.backend = MIRIAM_BACKEND_FAKE;
    c.n_be_streams = 2;
    c.inflight_depth = 2;
    c.top_frac = 0.2;
    c.max_blk_frac = 0.1;
    c.max_pt_frac = 0.1;
    c.quantum_us = 10.0;
    c.log_launches = 1;
    c.profile_reps = 1;
    c.fake_n_cu = 8;
    c.fake_slots_per_cu = 2;
    c.fake_tile_ns = 500.0;
    c.fake_launch_ns = 1000.0;
    c.graphs = 1;
    c.fake_fail_launch = fail_at;
    return c;
}

static int run(int policy, int fail_at, int per_thread) {
    miriam_config cfg = base_config(policy, fail_at);
    if (miriam_init(&cfg) != MIRIAM_OK) {
        std::fprintf(stderr, "init: %s\n", miriam_last_error());
        return 1;
    }
    std::vector<miriam_op *> crit_ops = {make_gemm(3), make_gemm(5)};
    std::vector<miriam_op *> be_ops = {make_gemm(17), make_gemm(4), make_gemm(9)};
    for (miriam_op *o : crit_ops) if (!o) return 1;
    for (miriam_op *o : be_ops) if (!o) return 1;
    miriam_task *crit = nullptr, *be = nullptr;
    if (miriam_task_create(crit_ops.data(), (int)crit_ops.size(), &crit) != MIRIAM_OK ||
        miriam_task_create(be_ops.data(), (int)be_ops.size(), &be) != MIRIAM_OK) {
        std::fprintf(stderr, "task: %s\n", miriam_last_error());
        return 1;
    }
    const int n_sub = 4;
    std::atomic<int> submitted{0}, failed_submit{0};
    std::atomic<bool> done{false};
    std::atomic<long> completed{0}, bad{0};
    std::vector<std::thread> th;
    for (int k = 0; k < n_sub; ++k)
        th.emplace_back([&, k] {
            for (int i = 0; i < per_thread; ++i) {
                uint64_t t = 0;
                const int critical = (k == 0 && i % 4 == 0) ? 1 : 0;
                const int64_t rel = (i % 7 == 0) ? miriam_now_ns() + 200000 : 0;
                if (miriam_submit(critical ? crit : be, critical, rel, 0, &t) == MIRIAM_OK) submitted++;
                else failed_submit++;
            }
        });
    std::thread poller([&] {
        miriam_completion buf[64];
        while (!done.load() || completed.load() < submitted.load()) {
            const int n = miriam_poll(buf, 64);
            if (n < 0) break;
            for (int i = 0; i < n; ++i) {
                completed++;
                if (buf[i].status != MIRIAM_OK) bad++;
            }
            if (n == 0) std::this_thread::yield();
        }
    });
    std::thread reader([&] {
        miriam_launch_record rec[32];
        miriam_stats st;
        while (!done.load()) {
            (void)miriam_stats_get(&st);
            (void)miriam_launch_log(rec, 32);
            std::this_thread::yield();
        }
    });
    for (auto &t : th) t.join();
    done = true;
    const int drc = miriam_drain(30000);
    poller.join();
    reader.join();
    miriam_stats st;
    (void)miriam_stats_get(&st);
    const int src = miriam_shutdown();
    (void)miriam_task_destroy(crit);
    (void)miriam_task_destroy(be);
    for (miriam_op *o : crit_ops) (void)miriam_op_destroy(o);
    for (miriam_op *o : be_ops) (void)miriam_op_destroy(o);
    std::printf("policy %d fail_at %d: submitted %d completed %ld failed %ld (stats %lld / %lld) drain %d shutdown %d\n",
                policy, fail_at, submitted.load(), completed.load(), bad.load(), (long long)st.completed,
                (long long)st.failed_requests, drc, src);
    if (failed_submit.load() != 0 || drc != MIRIAM_OK || src != MIRIAM_OK) return 1;
    if (completed.load() != submitted.load() || st.completed != submitted.load()) return 1;
    if (bad.load() != (fail_at > 0 ? 1 : 0) || st.failed_requests != bad.load()) return 1;
    return 0;
}

int main() {
    int rc = 0;
    rc |= run(MIRIAM_POLICY_ELASTIC, 0, 300);
    rc |= run(MIRIAM_POLICY_SEQUENTIAL, 0, 40);
    rc |= run(MIRIAM_POLICY_IB, 0, 40);
    rc |= run(MIRIAM_POLICY_ELASTIC, 5, 40);
    rc |= run(MIRIAM_POLICY_MULTISTREAM, 3, 40);
    std::printf(rc ? "FAILED\n" : "OK\n");
    return rc;
}
