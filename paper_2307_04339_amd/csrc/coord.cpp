// Runtime dynamic kernel coordinator (§5.2, §7).
//
// Two queues of inference requests: critical and normal.  One dispatcher thread
// owns every launch.  Critical requests run unsharded, in order, on the
// critical stream.  Normal requests run as elastic shards on one stream per
// normal task; each shard is the head node of the op's shaded binary tree
// (§7), sized either to the whole GPU (no critical work in flight, greedy
// policy) or to the resources the running critical kernel leaves free, by the
// Eq. (2) limiters and the WIScore x OScore ranking with the top fraction kept
// (§6.3).  A bounded number of shards per normal stream is in flight, so a
// newly released critical request waits at most for the shards already on the
// GPU.  All streams keep the default priority: the coordinator, not the
// hardware queue priority, decides what may occupy the GPU.
//
// Baseline policies for comparison (§8.1.3): SEQUENTIAL runs one request at a
// time on one stream, critical first; MULTISTREAM launches every request's
// kernels unsharded on its task's stream; IB (inter-stream barrier) advances the
// tasks' unsharded kernels in lockstep groups, one kernel per task and stream,
// each stream waiting on the device for the previous group's kernels.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <condition_variable>
#include <cstring>
#include <ctime>
#include <deque>
#include <functional>
#include <mutex>
#include <new>
#include <queue>
#include <shared_mutex>
#include <sys/prctl.h>
#include <thread>
#include <vector>

#include "internal.h"

namespace miriam {

static int64_t mono_ns() {
    timespec ts;
    clock_gettime(CLOCK_MONOTONIC, &ts);
    return (int64_t)ts.tv_sec * 1000000000LL + ts.tv_nsec;
}

// ------------------------------------------------------------------ backends
// Ops [i0, i1) of a task, each launched unsharded (grid = T, block 256), recorded once and
// replayed as a unit.
struct Captured {
    virtual ~Captured() {}
};

struct Backend {
    virtual ~Backend() {}
    // Create the streams: 0 critical, 1 .. n-1 normal; with cu_reserve > 0 the normal streams
    // leave out the top cu_reserve of n_cu compute units, and with crit_exclusive the critical
    // stream has only those.
    virtual int start(int n_streams, int n_cu, int cu_reserve, bool crit_exclusive) = 0;
    virtual int launch(const miriam_op *op, int64_t b, int64_t l, int grid, int block, int stream) = 0;
    virtual int record(int stream) = 0;       // event id >= 0, or < 0 error
    virtual int query(int ev) = 0;            // 1 done, 0 pending, < 0 error
    virtual void release(int ev) = 0;
    virtual double time_us(const miriam_op *op, int64_t b, int64_t l, int grid, int block, int reps) = 0;
    virtual double launch_gap_us(const miriam_op *op, int reps) = 0;
    // Record the unsharded launch sequence of `ops` (grid = T, block 256 each) as one
    // replayable unit; nullptr where the backend has none (then requests launch per op).
    virtual Captured *capture(const std::vector<miriam_op *> &ops, size_t i0, size_t i1) {
        (void)ops; (void)i0; (void)i1;
        return nullptr;
    }
    virtual int launch_captured(Captured *unit, int stream) { (void)unit; (void)stream; return MIRIAM_ESTATE; }
    // Run the cache-warming kernel over a device table of ranges on `stream`, after the
    // recorded events `waits` (work already queued on other streams) have completed.
    virtual int warm(const WarmRange *table, int n, int grid, int *sink, int stream, const std::vector<int> &waits) {
        (void)table; (void)n; (void)grid; (void)sink; (void)stream; (void)waits;
        return MIRIAM_OK;
    }
    // Queue a gate on `stream`: the stream's later work waits until open_gates(>= seq) or
    // until limit_ns have passed.  A simulated device models the gate as ending at release_ns.
    virtual int gate(uint64_t seq, int64_t release_ns, int64_t limit_ns, int stream) {
        (void)seq; (void)release_ns; (void)limit_ns; (void)stream;
        return MIRIAM_ESTATE;
    }
    virtual void open_gates(uint64_t seq) { (void)seq; }
    // Clear, in the order of `stream`, the split-K arrival counters of `op` after a pass over it
    // that may have stopped part-way (a failed launch ended its request).
    virtual int reset_op(const miriam_op *op, int stream) = 0;
    // Make later work on `stream` wait, on the device, for recorded event `ev`.
    virtual int wait_event(int stream, int ev) {
        (void)stream; (void)ev;
        return MIRIAM_ESTATE;
    }
    virtual void stop() = 0;
};

// An instantiated HIP graph.
struct HipGraphUnit : Captured {
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    ~HipGraphUnit() override {
        if (exec) (void)hipGraphExecDestroy(exec);
        if (graph) (void)hipGraphDestroy(graph);
    }
};

struct HipBackend : Backend {
    int dev = 0;
    std::vector<hipStream_t> streams;
    std::vector<hipEvent_t> events;
    std::vector<int> free_ev;
    hipStream_t prof = nullptr;
    hipStream_t cap = nullptr;  // capture stream for task graphs (never executes work)
    std::mutex cap_mu;
    uint64_t *gate_host = nullptr;  // gate flag in coherent host memory, and its device address
    uint64_t *gate_dev = nullptr;
    int wall_khz = 0;               // device wall-clock rate

    int start(int n, int n_cu, int cu_reserve, bool crit_exclusive) override {
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
        std::vector<uint32_t> normal_mask((size_t)(n_cu + 31) / 32, 0u), crit_mask(normal_mask.size(), 0u);
        for (int i = 0; i < n_cu; ++i) {
            std::vector<uint32_t> &m = i < n_cu - cu_reserve ? normal_mask : crit_mask;
            m[(size_t)i / 32] |= 1u << (i % 32);
        }
        for (int i = 0; i < n; ++i) {
            hipStream_t s;
            if (cu_reserve > 0 && (i > 0 || crit_exclusive)) {
                const std::vector<uint32_t> &mask = i > 0 ? normal_mask : crit_mask;
                e = hipExtStreamCreateWithCUMask(&s, (uint32_t)mask.size(), mask.data());
                if (e != hipSuccess) return hip_fail(e, "hipExtStreamCreateWithCUMask");
                streams.push_back(s);
                // the mask the stream reports must be the one asked for
                std::vector<uint32_t> got(mask.size(), 0u);
                e = hipExtStreamGetCUMask(s, (uint32_t)got.size(), got.data());
                if (e != hipSuccess) return hip_fail(e, "hipExtStreamGetCUMask");
                if (got != mask) {
                    set_error("stream reports a different compute-unit mask than requested");
                    return MIRIAM_ESTATE;
                }
                continue;
            } else {
                e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
                if (e != hipSuccess) return hip_fail(e, "hipStreamCreateWithFlags");
            }
            streams.push_back(s);
        }
        e = hipStreamCreateWithFlags(&prof, hipStreamNonBlocking);
        if (e != hipSuccess) return hip_fail(e, "hipStreamCreateWithFlags");
        e = hipStreamCreateWithFlags(&cap, hipStreamNonBlocking);
        if (e != hipSuccess) return hip_fail(e, "hipStreamCreateWithFlags");
        e = hipHostMalloc(reinterpret_cast<void **>(&gate_host), 64, hipHostMallocCoherent | hipHostMallocMapped);
        if (e != hipSuccess) {
            gate_host = nullptr;
            return hip_fail(e, "hipHostMalloc (gate flag)");
        }
        __atomic_store_n(gate_host, (uint64_t)0, __ATOMIC_RELEASE);
        e = hipHostGetDevicePointer(reinterpret_cast<void **>(&gate_dev), gate_host, 0);
        if (e != hipSuccess) return hip_fail(e, "hipHostGetDevicePointer (gate flag)");
        e = hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, dev);
        if (e != hipSuccess || wall_khz <= 0) return hip_fail(e, "wall clock rate");
        return MIRIAM_OK;
    }
    int gate(uint64_t seq, int64_t release_ns, int64_t limit_ns, int stream) override {
        (void)release_ns;
        const uint64_t ticks = (uint64_t)std::max<int64_t>(0, limit_ns) * (uint64_t)wall_khz / 1000000u;
        return gate_launch(gate_dev, seq, ticks, streams[stream]);
    }
    void open_gates(uint64_t seq) override {
        if (gate_host) __atomic_store_n(gate_host, seq, __ATOMIC_RELEASE);
    }
    Captured *capture(const std::vector<miriam_op *> &ops, size_t i0, size_t i1) override {
        // thread-local capture: the dispatcher thread keeps launching on its own streams meanwhile
        std::lock_guard<std::mutex> lk(cap_mu);
        HipGraphUnit *cg = new (std::nothrow) HipGraphUnit();
        if (!cg) return nullptr;
        if (hipStreamBeginCapture(cap, hipStreamCaptureModeThreadLocal) != hipSuccess) {
            delete cg;
            return nullptr;
        }
        bool ok = true;
        for (size_t i = i0; i < i1; ++i) {
            const miriam_op *op = ops[i];
            const int grid = op_full_grid(op);
            if (op_launch(op, 0, op->T, grid, 256, cap) != MIRIAM_OK) {
                ok = false;
                break;
            }
        }
        hipError_t e = hipStreamEndCapture(cap, &cg->graph);
        if (!ok || e != hipSuccess || !cg->graph ||
            hipGraphInstantiate(&cg->exec, cg->graph, nullptr, nullptr, 0) != hipSuccess) {
            delete cg;
            return nullptr;
        }
        return cg;
    }
    int warm(const WarmRange *table, int n, int grid, int *sink, int stream, const std::vector<int> &waits) override {
        for (int ev : waits) {
            hipError_t e = hipStreamWaitEvent(streams[stream], events[ev], 0);
            if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
        }
        return warm_launch(table, n, grid, sink, streams[stream]);
    }
    int launch_captured(Captured *unit, int stream) override {
        hipError_t e = hipGraphLaunch(static_cast<HipGraphUnit *>(unit)->exec, streams[stream]);
        if (e != hipSuccess) return hip_fail(e, "hipGraphLaunch");
        return MIRIAM_OK;
    }
    int launch(const miriam_op *op, int64_t b, int64_t l, int grid, int block, int stream) override {
        return op_launch(op, b, l, grid, block, streams[stream]);
    }
    int record(int stream) override {
        int id;
        if (!free_ev.empty()) {
            id = free_ev.back();
            free_ev.pop_back();
        } else {
            // completion markers only: no timing, and a device-scope release (the host polls
            // them and never reads kernel output through them; later device work, copies
            // included, sees the writes), which spares a cache writeback per recorded event
            hipEvent_t ev;
            hipError_t e = hipEventCreateWithFlags(&ev, hipEventDisableTiming | hipEventReleaseToDevice);
            if (e != hipSuccess) return hip_fail(e, "hipEventCreateWithFlags");
            events.push_back(ev);
            id = (int)events.size() - 1;
        }
        hipError_t e = hipEventRecord(events[id], streams[stream]);
        if (e != hipSuccess) {
            free_ev.push_back(id);
            return hip_fail(e, "hipEventRecord");
        }
        return id;
    }
    int wait_event(int stream, int ev) override {
        hipError_t e = hipStreamWaitEvent(streams[stream], events[ev], 0);
        return e == hipSuccess ? MIRIAM_OK : hip_fail(e, "hipStreamWaitEvent");
    }
    int query(int ev) override {
        hipError_t e = hipEventQuery(events[ev]);
        if (e == hipSuccess) return 1;
        if (e == hipErrorNotReady) return 0;
        return hip_fail(e, "hipEventQuery");
    }
    void release(int ev) override { free_ev.push_back(ev); }
    double time_us(const miriam_op *op, int64_t b, int64_t l, int grid, int block, int reps) override {
        hipEvent_t e0, e1;
        if (hipEventCreate(&e0) != hipSuccess) return -1.0;
        if (hipEventCreate(&e1) != hipSuccess) {
            (void)hipEventDestroy(e0);
            return -1.0;
        }
        double best = -1.0;
        if (op_launch(op, b, l, grid, block, prof) == MIRIAM_OK &&
            hipStreamSynchronize(prof) == hipSuccess) {
            for (int r = 0; r < reps; ++r) {
                (void)hipEventRecord(e0, prof);
                if (op_launch(op, b, l, grid, block, prof) != MIRIAM_OK) break;
                (void)hipEventRecord(e1, prof);
                if (hipEventSynchronize(e1) != hipSuccess) break;
                float ms = 0.0f;
                if (hipEventElapsedTime(&ms, e0, e1) != hipSuccess) break;
                const double us = 1000.0 * ms;
                if (best < 0.0 || us < best) best = us;
            }
        }
        (void)hipEventDestroy(e0);
        (void)hipEventDestroy(e1);
        return best;
    }
    double launch_gap_us(const miriam_op *op, int reps) override {
        // time per launch of n back-to-back empty kernels: the gap one more kernel boundary adds
        (void)op;
        const int n = 16;
        hipEvent_t e0, e1;
        if (hipEventCreate(&e0) != hipSuccess) return -1.0;
        if (hipEventCreate(&e1) != hipSuccess) {
            (void)hipEventDestroy(e0);
            return -1.0;
        }
        double best = -1.0;
        for (int r = 0; r < reps + 1; ++r) {
            (void)hipEventRecord(e0, prof);
            bool ok = true;
            for (int i = 0; i < n && ok; ++i) ok = noop_launch(prof) == MIRIAM_OK;
            (void)hipEventRecord(e1, prof);
            if (!ok || hipEventSynchronize(e1) != hipSuccess) break;
            float ms = 0.0f;
            (void)hipEventElapsedTime(&ms, e0, e1);
            const double us = 1000.0 * ms / n;
            if (r > 0 && (best < 0.0 || us < best)) best = us;
        }
        (void)hipEventDestroy(e0);
        (void)hipEventDestroy(e1);
        return best;
    }
    int reset_op(const miriam_op *op, int stream) override { return op_reset_counters(op, streams[stream]); }
    void stop() override {
        open_gates(UINT64_MAX);
        for (hipStream_t s : streams) (void)hipStreamSynchronize(s);
        for (hipEvent_t e : events) (void)hipEventDestroy(e);
        for (hipStream_t s : streams) (void)hipStreamDestroy(s);
        if (prof) {
            (void)hipStreamSynchronize(prof);
            (void)hipStreamDestroy(prof);
        }
        if (cap) (void)hipStreamDestroy(cap);
        if (gate_host) (void)hipHostFree(gate_host);
        gate_host = gate_dev = nullptr;
        events.clear();
        free_ev.clear();
        streams.clear();
        prof = nullptr;
        cap = nullptr;
    }
};

// Host-simulated device for testing the coordinator without a GPU.  Each stream
// is a FIFO; a launch of l tiles with grid G on a device of n_cu x slots
// workgroup slots takes launch_ns + ceil(l / min(G, l, n_cu*slots)) * tile_ns.
struct FakeBackend : Backend {
    int n_cu = 8, slots = 2;
    double tile_ns = 1000.0, launch_ns = 2000.0;
    int64_t fail_at = 0;   // this launch (1-based, launches and captured replays) fails; 0 = none
    int64_t n_launch = 0;
    bool injected() {
        if (++n_launch != fail_at) return false;
        set_error("injected launch failure (simulated device)");
        return true;
    }
    std::vector<int64_t> busy_until;
    std::vector<int64_t> ev_time;
    std::vector<int> free_ev;

    int start(int n, int, int, bool) override {
        busy_until.assign(n, 0);
        return MIRIAM_OK;
    }
    int64_t duration(const miriam_op *op, int64_t l, int grid) const {
        int64_t conc = std::min<int64_t>(std::min<int64_t>(grid, l), (int64_t)n_cu * slots);
        int64_t waves = (l + conc - 1) / conc;
        (void)op;
        return (int64_t)(launch_ns + waves * tile_ns);
    }
    int launch(const miriam_op *op, int64_t b, int64_t l, int grid, int block, int stream) override {
        if (!op || b < 0 || l < 1 || b + l > op->T || grid < 1 || (block != 64 && block != 128 && block != 256)) {
            set_error("fake launch: bad shard");
            return MIRIAM_ERANGE;
        }
        if (injected()) return MIRIAM_EHIP;
        const int64_t now = mono_ns();
        const int64_t st = std::max(now, busy_until[stream]);
        busy_until[stream] = st + duration(op, l, grid);
        return MIRIAM_OK;
    }
    int record(int stream) override {
        const int64_t t = std::max(mono_ns(), busy_until[stream]);
        int id;
        if (!free_ev.empty()) {
            id = free_ev.back();
            free_ev.pop_back();
            ev_time[id] = t;
        } else {
            ev_time.push_back(t);
            id = (int)ev_time.size() - 1;
        }
        return id;
    }
    int query(int ev) override { return mono_ns() >= ev_time[ev] ? 1 : 0; }
    int wait_event(int stream, int ev) override {
        busy_until[stream] = std::max(busy_until[stream], ev_time[ev]);
        return MIRIAM_OK;
    }
    void release(int ev) override { free_ev.push_back(ev); }
    double time_us(const miriam_op *op, int64_t b, int64_t l, int grid, int block, int reps) override {
        (void)b; (void)block; (void)reps;
        return duration(op, l, grid) / 1000.0;
    }
    double launch_gap_us(const miriam_op *, int) override { return launch_ns / 1000.0; }
    struct FakeUnit : Captured {
        std::vector<const miriam_op *> ops;
    };
    Captured *capture(const std::vector<miriam_op *> &ops, size_t i0, size_t i1) override {
        FakeUnit *u = new (std::nothrow) FakeUnit();
        if (u) u->ops.assign(ops.begin() + i0, ops.begin() + i1);
        return u;
    }
    int launch_captured(Captured *unit, int stream) override {
        if (injected()) return MIRIAM_EHIP;
        int64_t st = std::max(mono_ns(), busy_until[stream]);
        for (const miriam_op *op : static_cast<FakeUnit *>(unit)->ops) st += duration(op, op->T, op_full_grid(op));
        busy_until[stream] = st;
        return MIRIAM_OK;
    }
    int gate(uint64_t, int64_t release_ns, int64_t, int stream) override {
        busy_until[stream] = std::max(std::max(busy_until[stream], mono_ns()), release_ns);
        return MIRIAM_OK;
    }
    int reset_op(const miriam_op *, int) override { return MIRIAM_OK; }
    void stop() override {}
};

}  // namespace miriam

using namespace miriam;

// Per-op profile taken when a task is created (a9: occupancy and launch-overhead
// profiling that feeds Eq. (5)).
struct OpProf {
    double t_unsh_us = 0.0;     // unsharded launch (grid = T, block 256)
    double t_pers_us[3] = {0, 0, 0};  // one persistent shard over the whole GPU, per block
    double tau1_us[3] = {0, 0, 0};    // time of one tile on one workgroup, per block
    int cap[3] = {1, 1, 1};     // resident workgroups per CU, per block
    bool ok_pt[3] = {true, true, true};  // Eq. (5) persistent-thread term under its bar
    int64_t n_max = 1;          // Eq. (5) launch term: most shards the op may be cut into
};

struct miriam_task {
    std::vector<miriam_op *> ops;
    std::vector<OpProf> prof;
    int id = 0;
    std::atomic<int> pending{0};
    std::vector<Captured *> graphs;  // captured unsharded sequence (consecutive ops), or empty
    // segments: runs of consecutive short ops (profiled unsharded time within one quantum in
    // total) that a normal request issues as one captured unit while no critical kernel runs
    struct Segment {
        size_t i0, i1;
        Captured *unit;
        double est_us;
    };
    std::vector<Segment> segs;
    std::vector<int> seg_at;      // per op: the segment that starts there, or -1
    std::vector<double> end_us;   // profiled end of op i within one unsharded run
    // parameter lines touched before a release (cache warming): device table of ranges and a
    // sink word (HIP backend), their line count and estimated duration
    void *warm_dev = nullptr;
    int warm_n = 0, warm_grid = 0;
    int64_t warm_lines = 0;
    double warm_us = 0.0;
    ~miriam_task() {
        for (Captured *gph : graphs) delete gph;
        for (Segment &sg : segs) delete sg.unit;
        if (warm_dev) (void)hipFree(warm_dev);
    }
};

namespace {

// Shot::ev values other than an event id: no event recorded with this launch (it is known
// complete once a later launch of the same stream is), or known complete (failure path).
constexpr int kNoEvent = -1, kDone = -2;

struct Shot {  // one launch in flight
    int ev;
    int op;         // op index, or -1 for the task's whole captured sequence
    double est_us;  // estimated duration (task profile), counted against cfg.inflight_us
};

struct Req {
    uint64_t ticket = 0;
    miriam_task *task = nullptr;
    int crit = 0;
    int stream = 0;
    int64_t release = 0, deadline = 0, t_start = 0;
    int n_shards = 0;
    int status = MIRIAM_OK;
    size_t op = 0;       // next op to launch
    int64_t cursor = 0;  // next tile of that op
    bool launched_all = false;
    int64_t est_gpu_start = 0;  // estimated start on the GPU of a captured sequence (after the
                                // requests ahead of it on the same stream)
    int64_t est_gpu_end = 0;
    uint64_t gate = 0;  // armed: the gate its kernels wait behind (opened at the release)
    std::deque<Shot> shots;
};

struct ReleaseLater {
    bool operator()(const Req *a, const Req *b) const {
        if (a->release != b->release) return a->release > b->release;
        return a->ticket > b->ticket;
    }
};

struct Coord {
    miriam_config cfg{};
    Backend *be = nullptr;
    int n_streams = 2;
    int n_cu = 256, l_threads = 2048;
    double t_launch_us = 5.0;
    bool t_launch_measured = false;
    int next_task_id = 0;

    std::mutex mu;               // inbox, outbox, counters shared with callers
    std::condition_variable cv;  // wakes the dispatcher
    std::condition_variable cv_done;
    std::vector<Req *> inbox;
    std::deque<miriam_completion> outbox;
    int64_t outstanding = 0;
    uint64_t next_ticket = 1;
    bool stopping = false;
    std::thread th;

    // dispatcher-owned state
    std::priority_queue<Req *, std::vector<Req *>, ReleaseLater> timed;
    std::priority_queue<Req *, std::vector<Req *>, ReleaseLater> crit_timed;  // the critical ones among them
    uint64_t warmed_ticket = 0;                    // critical request whose parameters were last warmed
    Req *armed = nullptr;                          // timed critical request queued behind a gate
    uint64_t gate_seq = 0;
    std::vector<int> last_ev;                      // event of the latest launch per stream
    std::vector<double> since_ev_us;               // estimated work launched since that event
    std::vector<Req *> crit_ready;                 // released critical requests
    std::vector<std::deque<Req *>> norm_ready;     // per stream, FIFO
    std::deque<Req *> crit_active;                 // launched critical requests, stream 0
    std::vector<std::deque<Req *>> be_active;      // per stream, launched normal requests
    std::vector<int> inflight;                     // shards in flight per stream
    std::vector<double> inflight_us;               // their estimated duration per stream
    int rr_stream = 1;
    // IB: barrier events (stream, event) of the kernel groups queued on the GPU, oldest first
    std::deque<std::vector<std::pair<int, int>>> ib_groups;

    std::mutex log_mu;
    std::vector<miriam_launch_record> log;
    size_t log_read = 0;

    std::mutex stat_mu;
    miriam_stats stats{};
};

Coord *g = nullptr;
// Lifetime of g: init, shutdown and task creation hold it exclusively; submit, poll, drain,
// stats and the launch log hold it shared, so they never see g deleted under them.
std::shared_mutex g_life;

int64_t eq2_limit(int n_cu, int64_t n_rt) { return miriam_plan_eq2_grid_limit(n_cu, n_rt); }

void log_launch(Coord &c, const Req *r, int op_index, int stream, int grid, int block, bool crit_busy,
                int64_t b, int64_t l, int64_t T, int64_t limit, double est_us) {
    if (!c.cfg.log_launches) return;
    miriam_launch_record rec;
    rec.ticket = r->ticket;
    rec.op_index = op_index;
    rec.stream = stream;
    rec.criticality = r->crit;
    rec.grid = grid;
    rec.block = block;
    rec.crit_busy = crit_busy ? 1 : 0;
    rec.shard_begin = b;
    rec.shard_len = l;
    rec.num_tiles = T;
    rec.eq2_grid_limit = limit;
    rec.t_issue_ns = mono_ns();
    rec.est_us = est_us;
    std::lock_guard<std::mutex> lk(c.log_mu);
    if (c.log.size() - c.log_read < (1u << 22)) c.log.push_back(rec);
}

// Launch shard [b, b+l) of op `oi` of request r on `stream` and record its event.
int issue(Coord &c, Req *r, int oi, int64_t b, int64_t l, int grid, int block, int stream, bool crit_busy,
          int64_t limit, double est_us = 0.0, bool with_event = true) {
    const miriam_op *op = r->task->ops[oi];
    int rc = c.be->launch(op, b, l, grid, block, stream);
    if (rc != MIRIAM_OK) return rc;
    int ev = kNoEvent;
    if (with_event) {
        ev = c.be->record(stream);
        if (ev < 0) return ev;
        c.last_ev[stream] = ev;
        c.since_ev_us[stream] = 0.0;
    } else {
        c.since_ev_us[stream] += est_us;
    }
    if (r->t_start == 0) r->t_start = mono_ns();
    r->shots.push_back({ev, oi, est_us});
    r->n_shards++;
    c.inflight[stream]++;
    c.inflight_us[stream] += est_us;
    log_launch(c, r, oi, stream, grid, block, crit_busy, b, l, op->T, limit, est_us);
    std::lock_guard<std::mutex> lk(c.stat_mu);
    c.stats.launches++;
    return MIRIAM_OK;
}

void finish(Coord &c, Req *r) {
    miriam_completion cp;
    std::memset(&cp, 0, sizeof(cp));
    cp.ticket = r->ticket;
    cp.criticality = r->crit;
    cp.status = r->status;
    cp.t_release_ns = r->release;
    cp.t_start_ns = r->t_start;
    cp.t_end_ns = mono_ns();
    cp.deadline_ns = r->deadline;
    cp.deadline_met = (r->deadline == 0 || cp.t_end_ns <= r->deadline) ? 1 : 0;
    cp.n_shards = r->n_shards;
    for (miriam_op *op : r->task->ops) op->pending.fetch_sub(1);
    r->task->pending.fetch_sub(1);
    delete r;
    {
        std::lock_guard<std::mutex> lk(c.mu);
        c.outbox.push_back(cp);
        c.outstanding--;
    }
    {
        std::lock_guard<std::mutex> lk(c.stat_mu);
        c.stats.completed++;
    }
    c.cv_done.notify_all();
}

// A launch of request r failed on `stream`: the request ends with that error.  The pass over
// the op it was on may have stopped part-way, leaving split-K arrival counters non-zero, so
// the counters of every op of its task are cleared in stream order, before any later launch
// on the stream (a later request's pass then reduces the right slices).
void fail_request(Coord &c, Req *r, int status, int stream) {
    if (r->status == MIRIAM_OK) {
        std::lock_guard<std::mutex> lk(c.stat_mu);
        c.stats.failed_requests++;
    }
    r->status = status;
    int64_t n = 0;
    for (const miriam_op *op : r->task->ops)
        if (c.be->reset_op(op, stream) == MIRIAM_OK) ++n;
    std::lock_guard<std::mutex> lk(c.stat_mu);
    c.stats.failed_pass_resets += n;
}

// Launch every op of a request unsharded (grid = T, block 256) on `stream`: one replay of
// the task's captured sequence where there is one (one host call and one completion event
// instead of one launch and one event per op), else op by op.
void launch_whole(Coord &c, Req *r, int stream) {
    miriam_task *t = r->task;
    const std::deque<Req *> &ahead = stream == 0 ? c.crit_active : c.be_active[stream];
    const int64_t now = mono_ns();
    r->est_gpu_start = std::max(now, ahead.empty() ? now : ahead.back()->est_gpu_end);
    r->est_gpu_end = r->est_gpu_start + (int64_t)(1000.0 * (t->end_us.empty() ? 0.0 : t->end_us.back()));
    if (!t->graphs.empty() && c.cfg.graphs) {
        int rc = MIRIAM_OK;
        for (size_t k = 0; k < t->graphs.size() && rc == MIRIAM_OK; ++k) rc = c.be->launch_captured(t->graphs[k], stream);
        int ev = rc == MIRIAM_OK ? c.be->record(stream) : rc;
        if (ev < 0) {
            fail_request(c, r, ev, stream);
        } else {
            const double total = t->end_us.empty() ? 0.0 : t->end_us.back();
            r->t_start = now;
            r->shots.push_back({ev, -1, total});
            c.last_ev[stream] = ev;
            r->n_shards += (int)t->ops.size();
            c.inflight[stream]++;
            c.inflight_us[stream] += total;
            for (size_t i = 0; i < t->ops.size(); ++i) {
                const miriam_op *op = t->ops[i];
                log_launch(c, r, (int)i, stream, op_full_grid(op), 256, false, 0, op->T,
                           op->T, 0, t->prof[i].t_unsh_us);
            }
            std::lock_guard<std::mutex> lk(c.stat_mu);
            c.stats.launches += (int64_t)t->ops.size();
            c.stats.graph_launches++;
        }
        r->op = t->ops.size();
        r->launched_all = true;
        return;
    }
    for (size_t i = 0; i < r->task->ops.size(); ++i) {
        const miriam_op *op = r->task->ops[i];
        const int grid = op_full_grid(op);
        int rc = issue(c, r, (int)i, 0, op->T, grid, 256, stream, false, 0);
        if (rc != MIRIAM_OK) {
            fail_request(c, r, rc, stream);
            break;
        }
    }
    r->op = r->task->ops.size();
    r->launched_all = true;
}

// Retire completed launches of the requests on one stream; returns true if anything completed.
bool retire(Coord &c, std::deque<Req *> &active, int stream) {
    bool any = false;
    while (!active.empty()) {
        Req *r = active.front();
        while (!r->shots.empty()) {
            // the first launch with an event; the event-less ones before it end no later
            size_t k = 0;
            while (k < r->shots.size() && r->shots[k].ev == kNoEvent) ++k;
            if (k == r->shots.size()) break;
            const int ev = r->shots[k].ev;
            if (ev != kDone) {
                int q = c.be->query(ev);
                if (q == 0) break;
                if (q < 0) r->status = q;
                c.be->release(ev);
            }
            for (size_t i = 0; i <= k; ++i) {
                c.inflight_us[stream] -= r->shots.front().est_us;
                r->shots.pop_front();
                c.inflight[stream]--;
            }
            if (c.inflight_us[stream] < 1e-9) c.inflight_us[stream] = 0.0;
            any = true;
        }
        if (r->shots.empty() && r->launched_all) {
            active.pop_front();
            finish(c, r);
            any = true;
            continue;
        }
        break;  // later requests on this stream are behind this one (FIFO)
    }
    return any;
}

// Op index of the critical kernel running now, or -1 if no critical work is in flight.
// A captured sequence runs as one launch; its running op is inferred from the time since its
// estimated start against the task profile (the op with the most tiles, the smallest Eq. (2)
// grid limit, where the task has no profile).
int current_critical_op(Coord &c, const miriam_op **op) {
    if (c.crit_active.empty()) return -1;
    Req *r = c.crit_active.front();
    if (r->shots.empty()) return -1;
    int oi = r->shots.front().op;
    if (oi < 0) {
        const miriam_task *t = r->task;
        const int n = (int)t->ops.size();
        if (t->end_us.empty() || !(t->end_us.back() > 0.0)) {
            oi = 0;
            for (int i = 1; i < n; ++i)
                if (t->ops[i]->T > t->ops[oi]->T) oi = i;
        } else {
            const double el = 1e-3 * (double)(mono_ns() - r->est_gpu_start);
            oi = 0;
            while (oi < n - 1 && t->end_us[oi] <= el) ++oi;
        }
    }
    *op = r->task->ops[oi];
    return oi;
}

struct Decision {
    int grid, block;
    int64_t len, limit;
    double est_us;  // estimated duration of the shard
};

// §6.3 + §7: size the next shard of op `oi` of normal request r.
Decision decide(Coord &c, Req *r, const miriam_op *crit_op) {
    const miriam_op *op = r->task->ops[r->op];
    const OpProf &pf = r->task->prof[r->op];
    const int64_t T = op->T, cursor = r->cursor, remain = T - cursor;
    Decision d{0, 256, 0, 0, 0.0};
    int bi = 2;
    if (crit_op) {
        const int64_t n_rt = op_full_grid(crit_op);  // critical kernels run unsharded (whole-tile-space grid)
        const int64_t s_rt = 256;
        const int64_t gl = eq2_limit(c.n_cu, n_rt);
        const int64_t sl = miriam_plan_eq2_block_limit(c.l_threads, s_rt);
        double score[9];
        int64_t cg[9], cb[9];
        int n = 0;
        for (int64_t G : {gl, gl / 2, gl / 4}) {
            if (G < 1) continue;
            bool dup = false;
            for (int i = 0; i < n; ++i) dup |= (cg[i] == G);
            if (dup) continue;
            for (int k = 0; k < 3; ++k) {
                const int64_t B = 64 << k;
                if (B > sl) continue;
                cg[n] = G;
                cb[n] = B;
                score[n] = miriam_plan_wiscore(c.n_cu, c.l_threads, n_rt, s_rt, G, B) * (pf.ok_pt[k] ? 1.0 : 0.0);
                ++n;
            }
        }
        if (n == 0) {  // no feasible candidate: smallest footprint
            cg[0] = 1;
            cb[0] = 64;
            score[0] = 0.0;
            n = 1;
        }
        int keep[9];
        const int k = miriam_plan_top_fraction(n, score, cg, cb, c.cfg.top_frac, keep);
        (void)k;
        d.grid = (int)cg[keep[0]];
        d.block = (int)cb[keep[0]];
        if (c.cfg.busy_policy == 2) {  // ablation: smallest feasible footprint
            d.grid = (int)std::max<int64_t>(1, gl / 4);
            d.block = 64;
        }
        d.limit = gl;
        bi = d.block == 64 ? 0 : (d.block == 128 ? 1 : 2);
    } else {
        // alone on the GPU: greedy, the whole device
        bi = pf.ok_pt[2] ? 2 : (pf.ok_pt[1] ? 1 : (pf.ok_pt[0] ? 0 : 2));
        d.block = 64 << bi;
        d.grid = (int)std::min<int64_t>((int64_t)c.n_cu * std::max(1, pf.cap[bi]), INT32_MAX);
    }
    // tiles per workgroup within one time quantum
    const double tau = pf.tau1_us[bi] > 0.0 ? pf.tau1_us[bi] : 1.0;
    int64_t iters = (int64_t)std::floor(c.cfg.quantum_us / tau);
    if (iters < 1) iters = 1;
    int64_t max_len = (int64_t)d.grid * iters;
    const int64_t min_len = (T + pf.n_max - 1) / std::max<int64_t>(1, pf.n_max);
    max_len = std::max(max_len, min_len);
    max_len = std::max<int64_t>(1, std::min(max_len, remain));
    int depth = 0;
    int64_t len = miriam_plan_tree_head(T, cursor, max_len, &depth);
    if (len < 1) len = std::min<int64_t>(remain, max_len);
    d.len = len;
    d.grid = (int)std::max<int64_t>(1, std::min<int64_t>(d.grid, len));
    // estimated duration: the larger of the op's unsharded rate and the persistent rounds
    const double waves = (double)((len + d.grid - 1) / d.grid);
    d.est_us = std::max(pf.t_unsh_us * (double)len / (double)T, waves * pf.tau1_us[bi]);
    return d;
}

// Estimated normal work queued on the GPU, over all normal streams.
double queued_normal_us(const Coord &c) {
    double t = 0.0;
    for (size_t s = 1; s < c.inflight_us.size(); ++s) t += c.inflight_us[s];
    return t;
}

// Queue the cache-warming kernel over critical request nx's parameters on the normal stream
// with the most work queued, so that it runs once that work has drained.
void warm_for(Coord &c, const Req *nx) {
    c.warmed_ticket = nx->ticket;
    const miriam_task *t = nx->task;
    if (t->warm_n < 1) return;
    int s = 1;
    for (int k = 2; k < c.n_streams; ++k)
        if (c.inflight_us[k] > c.inflight_us[s]) s = k;
    char *base = static_cast<char *>(t->warm_dev);
    int rc = c.be->warm(reinterpret_cast<const WarmRange *>(base), t->warm_n, t->warm_grid,
                        base ? reinterpret_cast<int *>(base + sizeof(WarmRange) * t->warm_n) : nullptr, s, {});
    std::lock_guard<std::mutex> lk(c.stat_mu);
    if (rc == MIRIAM_OK) c.stats.warm_launches++;
}

// Release guard: true if normal work estimated at est_us, issued now behind the normal work
// already queued, would still be on the GPU at the next timed critical release (then normal
// work is held up to that release, and the request's parameters are warmed once).
bool guard_holds(Coord &c, int64_t t0, double est_us) {
    if (!c.cfg.release_guard || c.crit_timed.empty()) return false;
    const Req *nx = c.crit_timed.top();
    const double warm_us = c.cfg.warm_critical ? nx->task->warm_us : 0.0;
    if (c.warmed_ticket != nx->ticket &&
        t0 + (int64_t)(1000.0 * (queued_normal_us(c) + est_us + warm_us)) <= nx->release)
        return false;
    if (c.cfg.warm_critical && c.warmed_ticket != nx->ticket) warm_for(c, nx);
    return true;
}

// whole_when_clear: normal request r, not started, may run as one replay of its task's captured
// sequence: no critical request is pending or on the GPU, the next critical release is known
// (release guard), and the request's whole estimated time behind the normal work queued ends
// before that release.
bool whole_fits(Coord &c, const Req *r, int64_t t0) {
    if (!c.cfg.release_guard || !c.cfg.graphs || r->op != 0 || r->cursor != 0 || r->n_shards != 0) return false;
    const miriam_task *t = r->task;
    if (t->graphs.empty() || t->end_us.empty() || c.crit_timed.empty()) return false;
    if (!c.crit_ready.empty() || !c.crit_active.empty() || c.armed) return false;
    const Req *nx = c.crit_timed.top();
    const double warm_us = c.cfg.warm_critical ? nx->task->warm_us : 0.0;
    // the task profile times each op alone with warm caches; requests of several streams
    // running side by side from cold caches take longer, hence the margin
    const double margin = c.cfg.whole_margin > 0.0 ? c.cfg.whole_margin : 2.0;
    const double est = margin * (queued_normal_us(c) + t->end_us.back());
    return t0 + (int64_t)(1000.0 * (est + warm_us)) <= nx->release;
}

// Launch segment sg of normal request r on `stream` and record its event.
int issue_segment(Coord &c, Req *r, const miriam_task::Segment &sg, int stream, bool with_event) {
    int rc = c.be->launch_captured(sg.unit, stream);
    if (rc != MIRIAM_OK) return rc;
    int ev = kNoEvent;
    if (with_event) {
        ev = c.be->record(stream);
        if (ev < 0) return ev;
        c.last_ev[stream] = ev;
        c.since_ev_us[stream] = 0.0;
    } else {
        c.since_ev_us[stream] += sg.est_us;
    }
    if (r->t_start == 0) r->t_start = mono_ns();
    r->shots.push_back({ev, (int)sg.i0, sg.est_us});
    r->n_shards += (int)(sg.i1 - sg.i0);
    c.inflight[stream]++;
    c.inflight_us[stream] += sg.est_us;
    for (size_t i = sg.i0; i < sg.i1; ++i) {
        const miriam_op *op = r->task->ops[i];
        log_launch(c, r, (int)i, stream, op_full_grid(op), 256, false, 0, op->T, op->T, 0,
                   r->task->prof[i].t_unsh_us);
    }
    std::lock_guard<std::mutex> lk(c.stat_mu);
    c.stats.launches += (int64_t)(sg.i1 - sg.i0);
    c.stats.segment_launches++;
    return MIRIAM_OK;
}

// Whether a normal launch of est_us records a completion event: always on the request's
// last launch, else once event_us of estimated work has gathered since the stream's last event.
// A launch that fills the stream's in-flight depth or the shared budget also records one, so
// that the stream can always retire work and issue again.
bool want_event(const Coord &c, int stream, double est_us, bool last_of_request) {
    return last_of_request || c.cfg.event_us <= 0.0 || c.since_ev_us[stream] + est_us >= c.cfg.event_us ||
           c.inflight[stream] + 1 >= c.cfg.inflight_depth ||
           (c.cfg.inflight_us > 0.0 && queued_normal_us(c) + est_us >= c.cfg.inflight_us);
}

// Give request r's last launch an event (or, if recording fails, mark its launches complete)
// so that retiring them does not wait for a later launch: after a failure ends the request,
// and when normal work is held back.
void seal(Coord &c, Req *r, int stream) {
    if (r->shots.empty() || r->shots.back().ev != kNoEvent) return;
    const int ev = c.be->record(stream);
    r->shots.back().ev = ev >= 0 ? ev : kDone;
    c.since_ev_us[stream] = 0.0;
}

void seal_stream(Coord &c, int stream) {
    for (auto it = c.be_active[stream].rbegin(); it != c.be_active[stream].rend(); ++it)
        if (!(*it)->shots.empty()) {
            seal(c, *it, stream);
            return;
        }
}

// Issue shards for the normal requests of one stream while the in-flight budget lasts
// (every stream may keep one shard in flight; beyond that the budget is shared).
bool pump_normal(Coord &c, int s) {
    bool any = false;
    while (c.inflight[s] < c.cfg.inflight_depth &&
           (c.cfg.inflight_us <= 0.0 || c.inflight[s] == 0 || queued_normal_us(c) < c.cfg.inflight_us)) {
        Req *r = nullptr;
        for (Req *q : c.be_active[s])
            if (!q->launched_all) {
                r = q;
                break;
            }
        if (!r) {
            if (c.norm_ready[s].empty()) break;
            r = c.norm_ready[s].front();
            c.norm_ready[s].pop_front();
            c.be_active[s].push_back(r);
        }
        const int64_t t0 = mono_ns();
        const miriam_op *crit_op = nullptr;
        const bool busy = current_critical_op(c, &crit_op) >= 0;
        if (busy && c.cfg.busy_policy == 1) {  // ablation: hold normal work back
            seal_stream(c, s);
            break;
        }
        miriam_task *t = r->task;
        if (c.cfg.whole_when_clear && whole_fits(c, r, t0)) {
            launch_whole(c, r, s);
            {
                std::lock_guard<std::mutex> lk(c.stat_mu);
                c.stats.whole_clear_launches++;
            }
            any = true;
            if (r->status != MIRIAM_OK) seal(c, r, s);
            continue;
        }
        const int sid = (!busy && r->cursor == 0 && r->op < t->seg_at.size()) ? t->seg_at[r->op] : -1;
        if (sid >= 0) {  // a run of short ops as one captured unit
            const miriam_task::Segment &sg = t->segs[sid];
            if (guard_holds(c, t0, sg.est_us)) {
                seal_stream(c, s);
                break;
            }
            int rc = issue_segment(c, r, sg, s, want_event(c, s, sg.est_us, sg.i1 >= t->ops.size()));
            {
                std::lock_guard<std::mutex> lk(c.stat_mu);
                c.stats.decisions++;
                c.stats.decision_ns_total += (double)(mono_ns() - t0);
            }
            any = true;
            if (rc != MIRIAM_OK) {
                fail_request(c, r, rc, s);
                r->launched_all = true;
                seal(c, r, s);
                continue;
            }
            r->op = sg.i1;
            if (r->op >= t->ops.size()) r->launched_all = true;
            continue;
        }
        Decision d = decide(c, r, busy ? crit_op : nullptr);
        if (!busy && guard_holds(c, t0, d.est_us)) {
            seal_stream(c, s);
            break;
        }
        const int64_t t1 = mono_ns();
        const int oi = (int)r->op;
        const bool last = r->cursor + d.len >= r->task->ops[oi]->T && r->op + 1 >= r->task->ops.size();
        int rc = issue(c, r, oi, r->cursor, d.len, d.grid, d.block, s, busy, d.limit, d.est_us,
                       want_event(c, s, d.est_us, last));
        {
            std::lock_guard<std::mutex> lk(c.stat_mu);
            c.stats.decisions++;
            c.stats.decision_ns_total += (double)(t1 - t0);
            if (busy) {
                c.stats.shards_sized++;
                if (d.grid > d.limit) c.stats.eq2_violations++;
            }
        }
        any = true;
        if (rc != MIRIAM_OK) {
            fail_request(c, r, rc, s);
            r->launched_all = true;
            seal(c, r, s);
            continue;
        }
        r->cursor += d.len;
        if (r->cursor >= r->task->ops[oi]->T) {
            r->cursor = 0;
            r->op++;
            if (r->op >= r->task->ops.size()) r->launched_all = true;
        }
    }
    return any;
}

// IB baseline: one group = the next unsharded kernel of every task with work (the critical
// request in progress or next in line on the critical stream, each normal task's request on
// its stream).  Before its kernel, each stream waits on the device for the previous group's
// kernels on the other streams; after it, the stream records the group's barrier event.  At
// most two groups are queued, so a newly released critical request starts its first kernel
// behind at most two groups.  Kernels are launched op by op (a barrier follows every kernel),
// with one completion event per request, on its last kernel.
bool pump_ib(Coord &c) {
    bool any = false;
    while (!c.ib_groups.empty()) {
        bool done = true;
        for (const auto &se : c.ib_groups.front()) {
            const int q = c.be->query(se.second);
            if (q == 0) {
                done = false;
                break;
            }
        }
        if (!done) break;
        for (const auto &se : c.ib_groups.front()) c.be->release(se.second);
        c.ib_groups.pop_front();
        any = true;
    }
    if (c.ib_groups.size() >= 2) return any;
    std::vector<std::pair<Req *, int>> members;
    Req *cr = nullptr;
    if (!c.crit_active.empty() && !c.crit_active.back()->launched_all) {
        cr = c.crit_active.back();
    } else if (!c.crit_ready.empty()) {
        cr = c.crit_ready.front();
        c.crit_ready.erase(c.crit_ready.begin());
        c.crit_active.push_back(cr);
    }
    if (cr) members.push_back({cr, 0});
    for (int s = 1; s < c.n_streams; ++s) {
        Req *r = nullptr;
        if (!c.be_active[s].empty() && !c.be_active[s].back()->launched_all) {
            r = c.be_active[s].back();
        } else if (!c.norm_ready[s].empty()) {
            r = c.norm_ready[s].front();
            c.norm_ready[s].pop_front();
            c.be_active[s].push_back(r);
        }
        if (r) members.push_back({r, s});
    }
    if (members.empty()) return any;
    const std::vector<std::pair<int, int>> prev =
        c.ib_groups.empty() ? std::vector<std::pair<int, int>>() : c.ib_groups.back();
    std::vector<std::pair<int, int>> cur;
    for (const auto &m : members) {
        Req *r = m.first;
        const int s = m.second;
        int rc = MIRIAM_OK;
        for (const auto &se : prev)
            if (se.first != s && rc == MIRIAM_OK) rc = c.be->wait_event(s, se.second);
        const miriam_task *t = r->task;
        const int oi = (int)r->op;
        const bool last = r->op + 1 == t->ops.size();
        if (rc == MIRIAM_OK) {
            const miriam_op *op = t->ops[oi];
            rc = issue(c, r, oi, 0, op->T, op_full_grid(op), 256, s, false, 0, t->prof[oi].t_unsh_us, last);
        }
        if (rc != MIRIAM_OK) {
            fail_request(c, r, rc, s);
            r->op = t->ops.size();
            r->launched_all = true;
            seal(c, r, s);  // its earlier kernels carry no event: retire them with one
            continue;
        }
        r->op++;
        if (last) r->launched_all = true;
        const int ev = c.be->record(s);
        if (ev >= 0) cur.push_back({s, ev});
        else r->status = ev;
    }
    if (!cur.empty()) {
        c.ib_groups.push_back(cur);
        std::lock_guard<std::mutex> lk(c.stat_mu);
        c.stats.barrier_groups++;
    }
    return true;
}

bool all_idle(Coord &c) {
    if (!c.crit_active.empty()) return false;
    for (auto &q : c.be_active)
        if (!q.empty()) return false;
    return true;
}

// The gate of an armed request gives up this long after the release at the latest.
constexpr int64_t kGateSlackNs = 2000000;

// Queue timed critical request nx on the critical stream ahead of its release, behind a gate
// that the dispatcher opens at the release: the launch calls then cost the request nothing.
// Work released on the critical stream in the meantime waits behind the gate.
bool arm(Coord &c, Req *nx) {
    const int64_t now = mono_ns();
    const uint64_t seq = c.gate_seq + 1;
    if (c.be->gate(seq, nx->release, nx->release - now + kGateSlackNs, 0) != MIRIAM_OK) {
        c.cfg.arm_lead_us = 0.0;  // no gates on this backend: launch at the release
        return false;
    }
    c.gate_seq = seq;
    nx->gate = seq;
    launch_whole(c, nx, 0);
    nx->t_start = 0;  // set when the gate opens
    nx->est_gpu_start = std::max(nx->est_gpu_start, nx->release);
    nx->est_gpu_end = nx->est_gpu_start + (int64_t)(1000.0 * (nx->task->end_us.empty() ? 0.0 : nx->task->end_us.back()));
    c.armed = nx;
    std::lock_guard<std::mutex> lk(c.stat_mu);
    c.stats.armed_releases++;
    return true;
}

// The dispatcher sleeps only until this long before a timed release; the rest is spun.
constexpr int64_t kWakeEarlyNs = 300000;

void dispatcher(Coord *cp) {
    Coord &c = *cp;
    // timer slack of 1 us: a sleeping dispatcher must wake on time for releases
    (void)prctl(PR_SET_TIMERSLACK, 1000UL, 0UL, 0UL, 0UL);
    if (c.cfg.backend == MIRIAM_BACKEND_HIP) (void)hipSetDevice(static_cast<HipBackend *>(c.be)->dev);
    for (;;) {
        {
            std::unique_lock<std::mutex> lk(c.mu);
            for (Req *r : c.inbox) {
                c.timed.push(r);
                if (r->crit) c.crit_timed.push(r);
            }
            c.inbox.clear();
            if (c.stopping && c.outstanding == 0) break;
        }
        const int64_t now = mono_ns();
        while (!c.timed.empty() && c.timed.top()->release <= now) {
            Req *r = c.timed.top();
            c.timed.pop();
            if (r == c.armed) {  // its kernels are queued: open the gate
                c.be->open_gates(r->gate);
                r->t_start = mono_ns();
                c.crit_active.push_back(r);
                c.armed = nullptr;
            } else if (r->crit) {
                c.crit_ready.push_back(r);
            } else {
                c.norm_ready[r->stream].push_back(r);
            }
        }
        while (!c.crit_timed.empty() && c.crit_timed.top()->release <= now) c.crit_timed.pop();
        bool progress = false;
        if (c.cfg.arm_lead_us > 0.0 && c.cfg.policy == MIRIAM_POLICY_ELASTIC && !c.armed && !c.crit_timed.empty()) {
            Req *nx = c.crit_timed.top();
            if (nx->release > now && nx->release - now <= (int64_t)(1000.0 * c.cfg.arm_lead_us)) progress |= arm(c, nx);
        }
        // retire finished work
        progress |= retire(c, c.crit_active, 0);
        for (int s = 1; s < c.n_streams; ++s) progress |= retire(c, c.be_active[s], s);

        // order pending critical requests: earliest deadline, then release, then ticket
        if (c.crit_ready.size() > 1)
            std::stable_sort(c.crit_ready.begin(), c.crit_ready.end(), [](const Req *a, const Req *b) {
                const int64_t da = a->deadline ? a->deadline : INT64_MAX, db = b->deadline ? b->deadline : INT64_MAX;
                if (da != db) return da < db;
                if (a->release != b->release) return a->release < b->release;
                return a->ticket < b->ticket;
            });

        if (c.cfg.policy == MIRIAM_POLICY_SEQUENTIAL) {
            if (all_idle(c)) {
                if (!c.crit_ready.empty()) {
                    Req *r = c.crit_ready.front();
                    c.crit_ready.erase(c.crit_ready.begin());
                    launch_whole(c, r, 0);
                    c.crit_active.push_back(r);
                    progress = true;
                } else {
                    for (int k = 0; k < c.n_streams - 1; ++k) {
                        const int s = 1 + (c.rr_stream - 1 + k) % (c.n_streams - 1);
                        if (c.norm_ready[s].empty()) continue;
                        Req *r = c.norm_ready[s].front();
                        c.norm_ready[s].pop_front();
                        launch_whole(c, r, 0);
                        c.crit_active.push_back(r);  // one stream carries everything
                        c.rr_stream = 1 + s % (c.n_streams - 1);
                        progress = true;
                        break;
                    }
                }
            }
        } else if (c.cfg.policy == MIRIAM_POLICY_IB) {
            progress |= pump_ib(c);
        } else {
            // critical requests: unsharded, in order, on the critical stream
            while (!c.crit_ready.empty()) {
                Req *r = c.crit_ready.front();
                c.crit_ready.erase(c.crit_ready.begin());
                launch_whole(c, r, 0);
                c.crit_active.push_back(r);
                progress = true;
            }
            for (int s = 1; s < c.n_streams; ++s) {
                if (c.cfg.policy == MIRIAM_POLICY_MULTISTREAM) {
                    if (c.be_active[s].empty() && !c.norm_ready[s].empty()) {
                        Req *r = c.norm_ready[s].front();
                        c.norm_ready[s].pop_front();
                        launch_whole(c, r, s);
                        c.be_active[s].push_back(r);
                        progress = true;
                    }
                } else {
                    progress |= pump_normal(c, s);
                }
            }
        }

        if (!progress) {
            bool idle = all_idle(c);
            for (int s = 1; s < c.n_streams && idle; ++s) idle = c.norm_ready[s].empty();
            idle = idle && c.crit_ready.empty();
            if (idle) {
                // nothing on the GPU: sleep until a submission or the next timed release
                std::unique_lock<std::mutex> lk(c.mu);
                if (c.inbox.empty() && !(c.stopping && c.outstanding == 0)) {
                    // sleep until shortly before the next timed release, then spin to it
                    int64_t wait_ns = 2000000;
                    if (!c.timed.empty()) wait_ns = std::min<int64_t>(wait_ns, c.timed.top()->release - mono_ns());
                    const int64_t early = std::max<int64_t>(kWakeEarlyNs, (int64_t)(1000.0 * c.cfg.arm_lead_us) + 100000);
                    if (wait_ns > early) c.cv.wait_for(lk, std::chrono::nanoseconds(wait_ns - early));
                }
            } else {
                std::this_thread::yield();
            }
        }
    }
}

int estate(const char *m) {
    set_error(m);
    return MIRIAM_ESTATE;
}

// a9 + Eq. (5) inputs: time each op unsharded and as one persistent shard per block.
void profile_task(Coord &c, miriam_task *t) {
    const int reps = c.cfg.profile_reps > 0 ? c.cfg.profile_reps : 0;
    if (!c.t_launch_measured && !t->ops.empty() && (reps > 0 || c.cfg.backend == MIRIAM_BACKEND_FAKE)) {
        const double g = c.be->launch_gap_us(t->ops[0], std::max(1, reps));
        if (g > 0.0) c.t_launch_us = g;
        c.t_launch_measured = true;
    }
    for (size_t i = 0; i < t->ops.size(); ++i) {
        const miriam_op *op = t->ops[i];
        OpProf &p = t->prof[i];
        for (int k = 0; k < 3; ++k) {
            p.cap[k] = op->max_wg_per_cu[k] > 0 ? op->max_wg_per_cu[k] : 1;
            if (c.cfg.backend == MIRIAM_BACKEND_FAKE) p.cap[k] = static_cast<FakeBackend *>(c.be)->slots;
        }
        if (reps == 0 && c.cfg.backend == MIRIAM_BACKEND_HIP) {
            p.n_max = 1;
            continue;
        }
        const int greps = std::max(1, reps);
        p.t_unsh_us = c.be->time_us(op, 0, op->T, op_full_grid(op), 256, greps);
        for (int k = 0; k < 3; ++k) {
            const int64_t gp = std::min<int64_t>(op->T, (int64_t)c.n_cu * p.cap[k]);
            p.t_pers_us[k] = c.be->time_us(op, 0, op->T, (int)gp, 64 << k, greps);
            const int64_t iters = (op->T + gp - 1) / gp;
            p.tau1_us[k] = p.t_pers_us[k] > 0.0 ? p.t_pers_us[k] / (double)iters : 0.0;
            p.ok_pt[k] = p.t_unsh_us > 0.0 && (p.t_pers_us[k] - p.t_unsh_us) < c.cfg.max_pt_frac * p.t_unsh_us;
        }
        if (!p.ok_pt[0] && !p.ok_pt[1] && !p.ok_pt[2]) p.ok_pt[2] = true;  // keep the full block usable
        // (n - 1) * t_launch < MAX_blk = max_blk_frac * t_unsharded
        const double budget = c.cfg.max_blk_frac * std::max(0.0, p.t_unsh_us);
        p.n_max = 1 + (int64_t)std::floor(budget / std::max(1e-3, c.t_launch_us));
        p.n_max = std::max<int64_t>(1, std::min<int64_t>(p.n_max, op->T));
    }
    t->end_us.assign(t->ops.size(), 0.0);
    double acc = 0.0;
    for (size_t i = 0; i < t->ops.size(); ++i) t->end_us[i] = (acc += std::max(0.0, t->prof[i].t_unsh_us));
}

// Group runs of consecutive ops whose profiled unsharded times sum to at most one quantum
// into segments of two or more ops, each captured as one unit.
void build_segments(Coord &c, miriam_task *t) {
    const size_t n = t->ops.size();
    t->seg_at.assign(n, -1);
    const double q = c.cfg.quantum_us;
    size_t i = 0;
    while (i < n) {
        size_t j = i;
        double sum = 0.0;
        while (j < n && t->prof[j].t_unsh_us > 0.0 && sum + t->prof[j].t_unsh_us <= q) sum += t->prof[j++].t_unsh_us;
        if (j - i >= 2) {
            Captured *u = c.be->capture(t->ops, i, j);
            if (!u) return;  // no capture on this backend: ops launched one by one
            t->seg_at[i] = (int)t->segs.size();
            t->segs.push_back({i, j, u, sum});
            i = j;
        } else {
            i = std::max(j, i + 1);
        }
    }
}

// Line table of the task's parameters (each distinct range once) for cache warming; its
// duration is estimated at 2 TB/s (whole 64-byte lines) plus a launch.
int build_warm(Coord &c, miriam_task *t) {
    std::vector<WarmRange> tab;
    std::vector<const void *> seen;
    for (const miriam_op *op : t->ops) {
        const void *p[3];
        int64_t b[3];
        const int n = op_param_ranges(op, p, b);
        for (int i = 0; i < n; ++i) {
            if (std::find(seen.begin(), seen.end(), p[i]) != seen.end()) continue;
            seen.push_back(p[i]);
            const uintptr_t a0 = reinterpret_cast<uintptr_t>(p[i]) & ~(uintptr_t)63;
            const uintptr_t a1 = reinterpret_cast<uintptr_t>(p[i]) + (uintptr_t)b[i];
            tab.push_back({reinterpret_cast<const char *>(a0), (int64_t)((a1 - a0 + 63) / 64)});
            t->warm_lines += tab.back().lines;
        }
    }
    t->warm_n = (int)tab.size();
    t->warm_us = 4.0 + 64.0 * (double)t->warm_lines / 2.0e6;
    t->warm_grid = (int)std::max<int64_t>(1, std::min<int64_t>(16 * c.n_cu, (t->warm_lines + 1023) / 1024));
    if (c.cfg.backend != MIRIAM_BACKEND_HIP || tab.empty()) return MIRIAM_OK;
    const size_t bytes = sizeof(WarmRange) * tab.size() + 64;
    hipError_t e = hipMalloc(&t->warm_dev, bytes);
    if (e != hipSuccess) {
        t->warm_dev = nullptr;
        return hip_fail(e, "hipMalloc (warm table)");
    }
    e = hipMemcpy(t->warm_dev, tab.data(), sizeof(WarmRange) * tab.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy (warm table)");
    return MIRIAM_OK;
}

}  // namespace

extern "C" {

int64_t miriam_now_ns(void) { return mono_ns(); }

int miriam_gate_check(void *stream, int64_t limit_us, int64_t open_after_us, double *held_us) {
    if (!held_us || limit_us < 1 || limit_us > 100000) {
        set_error("gate check: limit_us in [1, 100000] and held_us required");
        return MIRIAM_EINVAL;
    }
    hipStream_t st = static_cast<hipStream_t>(stream);
    int dev = 0, khz = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev);
    if (e != hipSuccess || khz <= 0) return hip_fail(e, "wall clock rate");
    uint64_t *host = nullptr, *devp = nullptr;
    e = hipHostMalloc(reinterpret_cast<void **>(&host), 64, hipHostMallocCoherent | hipHostMallocMapped);
    if (e != hipSuccess) return hip_fail(e, "hipHostMalloc (gate flag)");
    __atomic_store_n(host, (uint64_t)0, __ATOMIC_RELEASE);
    hipEvent_t e0 = nullptr, e1 = nullptr;
    int rc = MIRIAM_OK;
    if ((e = hipHostGetDevicePointer(reinterpret_cast<void **>(&devp), host, 0)) != hipSuccess ||
        (e = hipEventCreate(&e0)) != hipSuccess || (e = hipEventCreate(&e1)) != hipSuccess ||
        (e = hipEventRecord(e0, st)) != hipSuccess) {
        rc = hip_fail(e, "gate check set-up");
    } else {
        rc = gate_launch(devp, 1, (uint64_t)limit_us * (uint64_t)khz / 1000u, st);
        if (rc == MIRIAM_OK && (e = hipEventRecord(e1, st)) != hipSuccess) rc = hip_fail(e, "hipEventRecord");
        if (rc == MIRIAM_OK && open_after_us >= 0) {
            std::this_thread::sleep_for(std::chrono::microseconds(open_after_us));
            __atomic_store_n(host, (uint64_t)1, __ATOMIC_RELEASE);
        }
        // the gate has a bounded wait, so this returns
        if (rc == MIRIAM_OK && (e = hipEventSynchronize(e1)) != hipSuccess) rc = hip_fail(e, "hipEventSynchronize");
        float ms = 0.0f;
        if (rc == MIRIAM_OK && (e = hipEventElapsedTime(&ms, e0, e1)) != hipSuccess) rc = hip_fail(e, "hipEventElapsedTime");
        *held_us = 1000.0 * ms;
    }
    if (rc != MIRIAM_OK) (void)hipStreamSynchronize(st);
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    (void)hipHostFree(host);
    return rc;
}

int miriam_init(const miriam_config *cfg) {
    std::unique_lock<std::shared_mutex> life(g_life);
    if (g) return estate("already initialised");
    if (!cfg) {
        set_error("null config");
        return MIRIAM_EINVAL;
    }
    if (cfg->policy < 0 || cfg->policy > 3 || cfg->backend < 0 || cfg->backend > 1 || cfg->n_be_streams < 1 ||
        cfg->n_be_streams > 7 || cfg->inflight_depth < 1 || !(cfg->top_frac > 0.0 && cfg->top_frac <= 1.0) ||
        !(cfg->quantum_us > 0.0) || cfg->max_blk_frac < 0.0 || cfg->max_pt_frac < 0.0 || cfg->profile_reps < 0 ||
        cfg->inflight_us < 0.0 || cfg->busy_policy < 0 || cfg->busy_policy > 2 || cfg->graphs < 0 ||
        cfg->graphs > 1 || cfg->release_guard < 0 || cfg->release_guard > 1 ||
        cfg->warm_critical < 0 || cfg->warm_critical > 1 || cfg->graph_chunk < 0 || !(cfg->arm_lead_us >= 0.0) ||
        cfg->segments < 0 || cfg->segments > 1 || !(cfg->event_us >= 0.0) || cfg->be_cu_reserve < 0 ||
        cfg->whole_when_clear < 0 || cfg->whole_when_clear > 1 || !(cfg->whole_margin >= 0.0) ||
        cfg->fake_fail_launch < 0 || cfg->crit_cu_exclusive < 0 || cfg->crit_cu_exclusive > 1) {
        set_error("invalid coordinator configuration");
        return MIRIAM_EINVAL;
    }
    Coord *c = new (std::nothrow) Coord();
    if (!c) {
        set_error("out of host memory");
        return MIRIAM_ENOMEM;
    }
    c->cfg = *cfg;
    c->n_streams = 1 + cfg->n_be_streams;
    if (cfg->backend == MIRIAM_BACKEND_HIP) {
        miriam_device_desc dd;
        int rc = miriam_device_query(&dd);
        if (rc != MIRIAM_OK) {
            delete c;
            return rc;
        }
        if (cfg->be_cu_reserve >= dd.n_cu) {
            delete c;
            set_error("be_cu_reserve must be below the device's compute-unit count");
            return MIRIAM_EINVAL;
        }
        c->n_cu = dd.n_cu;
        c->l_threads = dd.max_threads_per_cu;
        c->be = new HipBackend();
    } else {
        FakeBackend *f = new FakeBackend();
        f->n_cu = cfg->fake_n_cu > 0 ? cfg->fake_n_cu : 8;
        f->slots = cfg->fake_slots_per_cu > 0 ? cfg->fake_slots_per_cu : 2;
        f->tile_ns = cfg->fake_tile_ns > 0 ? cfg->fake_tile_ns : 1000.0;
        f->launch_ns = cfg->fake_launch_ns >= 0 ? cfg->fake_launch_ns : 2000.0;
        f->fail_at = cfg->fake_fail_launch;
        c->n_cu = f->n_cu;
        c->l_threads = 2048;
        c->be = f;
    }
    int rc = c->be->start(c->n_streams, c->n_cu, cfg->backend == MIRIAM_BACKEND_HIP ? cfg->be_cu_reserve : 0,
                          cfg->crit_cu_exclusive != 0);
    if (rc != MIRIAM_OK) {
        c->be->stop();
        delete c->be;
        delete c;
        return rc;
    }
    c->norm_ready.resize(c->n_streams);
    c->be_active.resize(c->n_streams);
    c->inflight.assign(c->n_streams, 0);
    c->inflight_us.assign(c->n_streams, 0.0);
    c->last_ev.assign(c->n_streams, -1);
    c->since_ev_us.assign(c->n_streams, 0.0);
    g = c;
    c->th = std::thread(dispatcher, c);
    return MIRIAM_OK;
}

int miriam_task_create(miriam_op *const *ops, int n_ops, miriam_task **out) {
    if (!ops || n_ops < 1 || !out) {
        set_error("task needs at least one op");
        return MIRIAM_EINVAL;
    }
    for (int i = 0; i < n_ops; ++i)
        if (!ops[i]) {
            set_error("null op in task");
            return MIRIAM_EINVAL;
        }
    std::unique_lock<std::shared_mutex> life(g_life);
    if (!g) return estate("coordinator not initialised");
    miriam_task *t = new (std::nothrow) miriam_task();
    if (!t) {
        set_error("out of host memory");
        return MIRIAM_ENOMEM;
    }
    t->ops.assign(ops, ops + n_ops);
    t->prof.resize(n_ops);
    t->id = g->next_task_id++;
    profile_task(*g, t);
    if (g->cfg.graphs) {  // no graph: launched op by op
        const size_t n = t->ops.size(), chunk = g->cfg.graph_chunk > 0 ? (size_t)g->cfg.graph_chunk : n;
        for (size_t i0 = 0; i0 < n; i0 += chunk) {
            Captured *gph = g->be->capture(t->ops, i0, std::min(n, i0 + chunk));
            if (!gph) {
                for (Captured *q : t->graphs) delete q;
                t->graphs.clear();
                break;
            }
            t->graphs.push_back(gph);
        }
    }
    if (g->cfg.segments) build_segments(*g, t);
    if (g->cfg.warm_critical) {
        int rc = build_warm(*g, t);
        if (rc != MIRIAM_OK) {
            delete t;
            return rc;
        }
    }
    *out = t;
    return MIRIAM_OK;
}

int miriam_submit(miriam_task *task, int criticality, int64_t release_ns, int64_t deadline_ns,
                  uint64_t *ticket_out) {
    if (!task || (criticality != 0 && criticality != 1) || release_ns < 0 || deadline_ns < 0) {
        set_error("bad submit arguments");
        return MIRIAM_EINVAL;
    }
    std::shared_lock<std::shared_mutex> life(g_life);
    if (!g) return estate("coordinator not initialised");
    Req *r = new (std::nothrow) Req();
    if (!r) {
        set_error("out of host memory");
        return MIRIAM_ENOMEM;
    }
    r->task = task;
    r->crit = criticality;
    r->release = release_ns > 0 ? release_ns : mono_ns();
    r->deadline = deadline_ns;
    r->stream = criticality ? 0 : 1 + task->id % (g->n_streams - 1);
    task->pending.fetch_add(1);
    for (miriam_op *op : task->ops) op->pending.fetch_add(1);
    uint64_t ticket;
    {
        std::lock_guard<std::mutex> lk(g->mu);
        if (g->stopping) {
            task->pending.fetch_sub(1);
            for (miriam_op *op : task->ops) op->pending.fetch_sub(1);
            delete r;
            return estate("coordinator is shutting down");
        }
        // the dispatcher owns r once it is queued (it may finish and free it at any time)
        ticket = r->ticket = g->next_ticket++;
        g->inbox.push_back(r);
        g->outstanding++;
    }
    g->cv.notify_one();
    if (ticket_out) *ticket_out = ticket;
    return MIRIAM_OK;
}

int miriam_poll(miriam_completion *out, int max_out) {
    if (!out || max_out < 0) {
        set_error("bad poll arguments");
        return MIRIAM_EINVAL;
    }
    std::shared_lock<std::shared_mutex> life(g_life);
    Coord *c = g;
    if (!c) return estate("coordinator not initialised");
    std::lock_guard<std::mutex> lk(c->mu);
    int n = 0;
    while (n < max_out && !c->outbox.empty()) {
        out[n++] = c->outbox.front();
        c->outbox.pop_front();
    }
    return n;
}

int miriam_drain(int64_t timeout_ms) {
    std::shared_lock<std::shared_mutex> life(g_life);
    Coord *c = g;
    if (!c) return estate("coordinator not initialised");
    std::unique_lock<std::mutex> lk(c->mu);
    const bool ok = c->cv_done.wait_for(lk, std::chrono::milliseconds(timeout_ms < 0 ? 0 : timeout_ms),
                                        [c] { return c->outstanding == 0; });
    if (!ok) {
        set_error("requests still in flight");
        return MIRIAM_EBUSY;
    }
    return MIRIAM_OK;
}

int miriam_stats_get(miriam_stats *out) {
    if (!out) {
        set_error("null output");
        return MIRIAM_EINVAL;
    }
    std::shared_lock<std::shared_mutex> life(g_life);
    Coord *c = g;
    if (!c) return estate("coordinator not initialised");
    std::lock_guard<std::mutex> lk(c->stat_mu);
    *out = c->stats;
    return MIRIAM_OK;
}

int miriam_launch_log(miriam_launch_record *out, int max_out) {
    if (!out || max_out < 0) {
        set_error("bad arguments");
        return MIRIAM_EINVAL;
    }
    std::shared_lock<std::shared_mutex> life(g_life);
    Coord *c = g;
    if (!c) return estate("coordinator not initialised");
    std::lock_guard<std::mutex> lk(c->log_mu);
    int n = 0;
    while (n < max_out && c->log_read < c->log.size()) out[n++] = c->log[c->log_read++];
    if (c->log_read == c->log.size()) {
        c->log.clear();
        c->log_read = 0;
    }
    return n;
}

int miriam_task_destroy(miriam_task *t) {
    if (!t) {
        set_error("null task");
        return MIRIAM_EINVAL;
    }
    if (t->pending.load() > 0) {
        set_error("task has pending requests");
        return MIRIAM_EBUSY;
    }
    delete t;
    return MIRIAM_OK;
}

int miriam_shutdown(void) {
    std::unique_lock<std::shared_mutex> life(g_life);
    Coord *c = g;
    if (!c) return estate("coordinator not initialised");
    {
        std::lock_guard<std::mutex> lk(c->mu);
        c->stopping = true;
    }
    c->cv.notify_one();
    c->th.join();
    c->be->stop();
    delete c->be;
    g = nullptr;
    delete c;
    return MIRIAM_OK;
}

}  // extern "C"
