/*
 * miriam.h — C ABI of the Miriam elastic-kernel library for AMD Instinct MI355X (gfx950).
 *
 * Paper: "Miriam: Exploiting Elastic Kernels for Real-time Multi-DNN Inference on
 * Edge GPU" (Zhao, Ling, Guan, Xing; arXiv 2307.04339).
 *
 * Three groups of entry points:
 *   1. Elastic operators (§6.1 elastic block, §6.2 elastic grid, §6.4 index functions):
 *      create an operator over caller-owned device buffers, query its logical tile
 *      space, and launch any contiguous shard [shard_begin, shard_begin+shard_len) of
 *      that tile space with any grid and any block of 64, 128 or 256 threads.  The
 *      output is bitwise identical for every shard plan, shard order, grid and block.
 *   2. Design-space shrinking and shard planning (§6.2 Eq. (1), §6.3 Eq. (2), (4), (5),
 *      §7 shaded binary tree): host-only functions, usable without a GPU.
 *   3. The runtime coordinator (§5.2, §7): two task queues (critical and normal),
 *      critical tasks run unsharded, normal tasks are cut into elastic shards sized to
 *      the resources the critical kernels leave free.
 *
 * Conventions (all entry points):
 *   - Every function returns an int: MIRIAM_OK (0) or a negative miriam_err.  No C++
 *     exception and no abort crosses this boundary.  miriam_last_error() returns a
 *     thread-local text for the last failure on the calling thread.
 *   - Pointers named "device" are HIP device addresses owned by the caller; the
 *     library never frees them.  Streams are hipStream_t values passed as void*
 *     (NULL = the legacy default stream).
 *   - Element types: activations/weights/outputs use the operator's dtype; per-channel
 *     parameters (bias, batch-norm, layer-norm gamma/beta) are always float32.
 *   - Layouts: activations NHWC; convolution weights [Cout][KH][KW][Cin/groups];
 *     depthwise weights [KH][KW][C]; GEMM computes Y[m][n] = sum_k A[m][k] * B[n][k]
 *     (B "K-major") or sum_k A[m][k] * B[k][n] (B "N-major").
 */
#ifndef MIRIAM_H
#define MIRIAM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MIRIAM_OK = 0,
    MIRIAM_EINVAL = -1,    /* malformed argument (null pointer, bad enum, bad shape) */
    MIRIAM_ERANGE = -2,    /* shard outside [0, T), grid < 1 or unsupported block size */
    MIRIAM_EHIP = -3,      /* the HIP runtime reported an error (text in miriam_last_error) */
    MIRIAM_ENOMEM = -4,    /* host or device allocation failed */
    MIRIAM_EBUSY = -5,     /* object still referenced by work in flight */
    MIRIAM_ESTATE = -6,    /* call not valid in the current state (e.g. not initialised) */
    MIRIAM_ENOTFOUND = -7  /* unknown ticket or handle */
} miriam_err;

typedef enum {
    MIRIAM_OP_CONV2D = 0,    /* implicit-GEMM convolution (+ fused epilogue) */
    MIRIAM_OP_GEMM = 1,      /* fully connected / matrix product (+ fused epilogue) */
    MIRIAM_OP_BGEMM = 2,     /* strided batched matrix product (attention scores, context) */
    MIRIAM_OP_DWCONV = 3,    /* depthwise convolution (+ fused epilogue) */
    MIRIAM_OP_POOL_MAX = 4,  /* max pooling, ignored padding */
    MIRIAM_OP_POOL_AVG = 5,  /* average pooling, divisor = window size */
    MIRIAM_OP_SOFTMAX = 6,   /* row softmax of scale * x */
    MIRIAM_OP_LAYERNORM = 7, /* row layer normalisation (+ residual added first) */
    MIRIAM_OP_BN_ACT = 8     /* elementwise epilogue: act(BN(x + bias) + residual) */
} miriam_op_kind;

typedef enum { MIRIAM_F32 = 0, MIRIAM_F16 = 1, MIRIAM_BF16 = 2 } miriam_dtype;

typedef enum { MIRIAM_ACT_NONE = 0, MIRIAM_ACT_RELU = 1, MIRIAM_ACT_RELU6 = 2, MIRIAM_ACT_GELU = 3 } miriam_act;

/* Epilogue flags for CONV2D, GEMM, BGEMM, DWCONV and BN_ACT, applied in this order:
 * v = acc (+ bias[c]); v = BN(v); v = v (+ residual); y = act(v). */
enum {
    MIRIAM_EPI_BIAS = 1,      /* bias: float32[Cout] */
    MIRIAM_EPI_BN = 2,        /* bn: float32[4*Cout] = gamma, beta, running mean, running var */
    MIRIAM_EPI_RESIDUAL = 4,  /* residual: same dtype/layout/strides as y */
    /* Not an epilogue step: index-function option (§6.4) for CONV2D / GEMM / BGEMM.  With it the
     * host computes, at creation, every output row's (image, first input row, first input
     * column) into a device table owned by the op, and each tile stages its rows of the table in
     * LDS instead of dividing the row index in the kernel (memory-based index function; the
     * default is computation-based).  Results are bitwise the same.  Served by the pipelined
     * contraction kernel only: the op is created on it (16-byte aligned K-major operands; an
     * explicit tile must be 1..4), else creation fails with MIRIAM_EINVAL. */
    MIRIAM_INDEX_MEMORY = 8
};

/*
 * Operator descriptor.  Fields not used by a kind are ignored.
 *   CONV2D / DWCONV / POOL_*: x is N x H x W x C (NHWC, pixel stride C unless ldx > 0),
 *       y is N x Ho x Wo x K (pixel stride K unless ldy > 0), Ho = (H + 2 pad - kh)/stride + 1.
 *       CONV2D: wt is [K][kh][kw][C/groups] (groups must be 1).  DWCONV: wt is [kh][kw][C],
 *       K = C.  POOL: K = C, kh x kw window.
 *   GEMM:  A = x is m x kk (row stride ldx, default kk), B = wt is nn x kk (row stride ldw,
 *       default kk), y is m x nn (row stride ldy, default nn).
 *   BGEMM: batch matrices; batch index bi splits as (bi / batch_div, bi % batch_div) and
 *       operand X's offset is (bi / batch_div) * sX0 + (bi % batch_div) * sX1 elements.
 *       b_nmajor = 0: B[n][k] (row stride ldw); 1: B[k][n] (row stride ldw).
 *   SOFTMAX: x, y are m rows of nn values (row strides ldx, ldy); y = softmax(scale * x).
 *   LAYERNORM: y = LN(x (+ residual)) * gamma + beta over rows of nn; gamma = wt, beta = bias
 *       (float32[nn]).
 *   BN_ACT: x, y are m rows of nn channels; epilogue flags as above.
 */
typedef struct miriam_op_desc {
    int32_t kind;       /* miriam_op_kind */
    int32_t dtype;      /* miriam_dtype */
    int32_t act;        /* miriam_act */
    int32_t flags;      /* MIRIAM_EPI_* */
    int64_t n, h, w, c; /* input geometry (NHWC) */
    int64_t k;          /* output channels (CONV2D) */
    int64_t kh, kw, stride, pad, groups;
    int64_t m, nn, kk;  /* GEMM-style sizes */
    int64_t batch, batch_div;
    int64_t ldx, ldw, ldy;               /* row strides in elements, 0 = dense */
    int64_t sx0, sx1, sw0, sw1, sy0, sy1; /* BGEMM batch strides in elements */
    int32_t b_nmajor;
    int32_t ksplit;     /* contractions: 0 = library choice, 1 = no split, n = split K over n workgroups
                           per output tile (partials reduced in fixed order; the op then owns a device
                           workspace and arrival counters, every pass over the op must cover its whole
                           tile space, and passes over one op must not overlap in time).  The library
                           choice splits small-batch FC layers (tile 5) into the fewest slices that
                           give every CU a tile (twice as many for slices of 8192 K values or more;
                           slices of about 1024 K values or more), and implicit-GEMM ops into the
                           most slices, up to 4, whose workgroups are all resident at once (two per
                           CU) with 8 or more K chunks each (32 or more when the op fills more than
                           half of the CUs); the workspace is allocated here, at creation */
    int32_t tile;       /* contractions: 0 = library choice, 1 = 32x32, 2 = 64x64, 3 = 128x128, 4 = 128x64,
                           5 = 16-column split-K (GEMM, fp16/bf16, m <= 16), 6 = 256x128,
                           7 = direct 3x3 stride-1 conv: 4x32 output pixels x 64 channels, the tile's
                           input patch held in LDS (C a multiple of 64 fp16/bf16 or 32 fp32 channels),
                           8 = direct 3x3 stride-1 conv with the weights resident in registers: same
                           tile, fp16/bf16, C in {8, 16, 32, 64}, at most 64 output channels */
    float eps;          /* BN / LN epsilon */
    float scale;        /* SOFTMAX scale */
    const void *x, *wt, *bias, *bn, *residual; /* device pointers (wt = weights) */
    void *y;                                 /* device pointer */
} miriam_op_desc;

typedef struct miriam_op miriam_op;     /* opaque; created by miriam_op_create */
typedef struct miriam_task miriam_task; /* opaque; an ordered list of ops = one request */

typedef struct miriam_op_info {
    int64_t num_tiles;        /* T: size of the logical tile space */
    int32_t logical_block;    /* threads of the logical block (256 = 4 logical waves) */
    int32_t lds_bytes;        /* LDS per workgroup; independent of the physical block */
    int32_t tile_m, tile_n;   /* contraction tile shape (0 for other kinds) */
    int32_t max_wg_per_cu[3]; /* resident workgroups per CU for blocks 64, 128, 256 (0 if unknown) */
    double flops;             /* algorithmic floating-point operations of the whole op */
    double bytes;             /* algorithmic HBM bytes: inputs and weights read once, outputs written once */
    int32_t path;             /* miriam_kernel_path: which kernel family serves the op */
    int32_t ksplit;           /* K slices per output tile (1 = no split); num_tiles counts slices */
    int32_t full_grid;        /* grid of the op's whole-tile-space (unsharded) launch: num_tiles (one
                                 workgroup per tile); for kernels that keep operands resident
                                 across tiles the workgroups that fit the device at once; for the
                                 global->LDS pipelined contraction (paths 2 and 3) with one to two
                                 rounds of resident workgroups' worth of tiles, half the tiles (two
                                 per workgroup) */
} miriam_op_info;

/* Kernel family behind an op (diagnostic; results do not depend on it beyond rounding
 * order, which is fixed per op). */
typedef enum miriam_kernel_path {
    MIRIAM_PATH_OTHER = 0,       /* memory-bound operator kernels */
    MIRIAM_PATH_STAGED = 1,      /* contraction, operands staged through registers */
    MIRIAM_PATH_DMA = 2,         /* contraction, global->LDS pipeline, per-lane K decode */
    MIRIAM_PATH_DMA_UNIFORM = 3, /* contraction, global->LDS pipeline, chunk-uniform filter taps */
    MIRIAM_PATH_SKINNY = 4,      /* small-batch fully connected, K split over logical waves */
    MIRIAM_PATH_HALO = 5,        /* direct 3x3 stride-1 convolution, input patch of the tile in LDS */
    MIRIAM_PATH_RESIDENT = 6     /* direct 3x3 stride-1 convolution, weights resident in registers
                                    across the tiles of a workgroup, input patch streamed through LDS */
} miriam_kernel_path;

/* ------------------------------------------------------------------ device */
typedef struct miriam_device_desc {
    int32_t n_cu;              /* compute units (N_SM of Table 1) */
    int32_t max_threads_per_cu; /* L_threads of Table 1 */
    int32_t lds_per_cu;        /* bytes */
    int32_t n_xcd;             /* dies that workgroups are dealt round-robin to */
    int32_t wave_size;
    int32_t clock_khz;
    char arch[64];
} miriam_device_desc;

/* Query the current HIP device.  Returns MIRIAM_EHIP if no device is present. */
int miriam_device_query(miriam_device_desc *out);

/* ---------------------------------------------------------- elastic operators */

/* Validate *d and create an operator that borrows the device pointers in *d until
 * miriam_op_destroy.  Allocates host memory only.  §6.4: the operator's index
 * function is computation-based (logical ids computed in-kernel). */
int miriam_op_create(const miriam_op_desc *d, miriam_op **out);

/* Device scratch of ops created by miriam_op_create_noalloc, per GPU: 1 MiB of split-K arrival
 * counters followed by the fp32 partials. */
#define MIRIAM_NOALLOC_SCRATCH_BYTES (32u << 20)

/*
 * For callers that cannot allocate device memory (code under stream capture, serving loops,
 * harnesses that forbid hipMalloc): miriam_op_create without any device allocation.  An op
 * whose kernels need a workspace (split K, miriam_op_info.ksplit > 1) takes it from a static
 * device array of MIRIAM_NOALLOC_SCRATCH_BYTES that the library holds on each GPU until the
 * process ends, shared by every op created this way on that GPU; the arrival counters it uses
 * are cleared here (a synchronous clear on the null stream).  Launches, queries and
 * miriam_op_destroy work as for any op.  Passes over two ops created this way on one GPU must
 * not overlap in time: they race on the shared array.  Errors: as miriam_op_create;
 * MIRIAM_EINVAL for MIRIAM_INDEX_MEMORY (its table is device memory); MIRIAM_ERANGE when the
 * caller asks for split K (ksplit > 1) and the workspace exceeds the array (more than 1 MiB of
 * counters or the rest of the array in partials); a split the library would choose is then
 * left out instead.  Host memory for the op object is still allocated.
 */
int miriam_op_create_noalloc(const miriam_op_desc *d, miriam_op **out);

/* Fill *out with the operator's tile space and resource figures. */
int miriam_op_query(const miriam_op *op, miriam_op_info *out);

/*
 * §6.1-6.2: launch shard [shard_begin, shard_begin + shard_len) of the operator's
 * tile space on `stream` with `grid` workgroups of `block` threads (64, 128 or 256).
 * Workgroup g runs tiles shard_begin + r(g) + i*grid (i = 0, 1, ...) below the shard's
 * end, where r(g) ranks workgroups so that those on one die take consecutive tiles.
 * A grid larger than shard_len is legal (the surplus workgroups exit at once).
 * Asynchronous: no synchronisation and no allocation.  Returns MIRIAM_ERANGE without
 * launching anything if 0 <= shard_begin, 1 <= shard_len, shard_begin + shard_len <= T,
 * grid >= 1 or block in {64,128,256} does not hold.
 */
int miriam_elastic_launch(const miriam_op *op, int64_t shard_begin, int64_t shard_len,
                          int grid, int block, void *stream);

/*
 * Same launch, additionally recording for every tile t of the shard, in caller-owned
 * device arrays of T int32 entries: owner_wg[t] = physical workgroup, owner_iter[t] =
 * persistent-loop iteration, and count[t] += 1 (atomic).  Used to check the tile map
 * (§6.2 elastic grid).  When wave_phys and wave_slot (caller-owned device arrays of 4 T
 * int32 entries) are non-null, entry 4 t + lambda receives, from the physical wave that ran
 * logical wave lambda (0..3) of tile t, that wave's index in the workgroup and the place of
 * lambda among the logical waves it runs (§6.1 N:1 logical-to-physical map: expected
 * lambda mod (block / 64) and lambda div (block / 64)).  Entries of tiles outside the shard
 * are left untouched.  MIRIAM_EINVAL if owner_wg, owner_iter or count is null, or if only
 * one of wave_phys and wave_slot is.
 */
int miriam_elastic_launch_traced(const miriam_op *op, int64_t shard_begin, int64_t shard_len,
                                 int grid, int block, void *stream,
                                 int32_t *owner_wg, int32_t *owner_iter, int32_t *count,
                                 int32_t *wave_phys, int32_t *wave_slot);

/* Split-K ops (miriam_op_info.ksplit > 1) count the slices that have arrived at each output
 * tile, and the last one to arrive reduces them and resets the count; a pass that covers the
 * whole tile space leaves every count at zero.  After a pass that did not (abandoned, or ended
 * by a failed launch), queue this on the stream of that pass before the next pass over the op:
 * it clears the counts in stream order (asynchronous).  MIRIAM_OK and nothing queued for ops
 * without split K; MIRIAM_EHIP if the clear cannot be queued.  The coordinator does this itself
 * for the ops of a request that a failed launch ends. */
int miriam_op_reset_counters(const miriam_op *op, void *stream);

/* Release the operator.  MIRIAM_EBUSY if a submitted task that uses it is pending. */
int miriam_op_destroy(miriam_op *op);

/* ------------------------------------------------------ planning (host only) */

/* Eq. (1): dichotomy slice widths of a kernel with M blocks, smallest first.
 * Returns the number of widths written (n+1), or MIRIAM_EINVAL / MIRIAM_ERANGE (cap). */
int miriam_plan_dichotomy(int64_t M, int64_t *widths, int cap);

/* Balanced slicing plan of T tiles into n shards: shard j = [floor(jT/n), floor((j+1)T/n)). */
int miriam_plan_split(int64_t T, int64_t n, int64_t *begin, int64_t *len);

/* Logical rank of physical workgroup g in a launch of G workgroups over n_xcd dies. */
int64_t miriam_plan_wg_rank(int64_t g, int64_t G, int64_t n_xcd);

/* Eq. (2): largest elastic grid and block next to a critical kernel of n_blk_rt
 * workgroups of s_blk_rt threads. */
int64_t miriam_plan_eq2_grid_limit(int64_t n_sm, int64_t n_blk_rt);
int64_t miriam_plan_eq2_block_limit(int64_t l_threads, int64_t s_blk_rt);

/* Eq. (4) WIScore, second factor read as (S_blk_rt + S_blk_be) / L_threads. */
double miriam_plan_wiscore(int64_t n_sm, int64_t l_threads, int64_t n_blk_rt, int64_t s_blk_rt,
                           int64_t n_blk_be, int64_t s_blk_be);

/* Eq. (5) OScore over n shards' launch-overhead terms. */
int miriam_plan_oscore(int64_t n, const double *lo_blk, const double *lo_pt,
                       double max_blk, double max_pt);

/* §6.3: keep the best ceil(frac*n) (>= 1) candidates by (score, grid, block), best first.
 * Returns the number kept. */
int miriam_plan_top_fraction(int n, const double *score, const int64_t *grid,
                             const int64_t *block, double frac, int *keep);

/* §7 shaded binary tree: length of the shallowest node that starts at `cursor` and
 * holds at most max_len tiles; *depth receives its depth.  Negative on bad input. */
int64_t miriam_plan_tree_head(int64_t T, int64_t cursor, int64_t max_len, int *depth);

/* ------------------------------------------------------------- coordinator */

typedef enum {
    MIRIAM_POLICY_ELASTIC = 0,     /* Miriam: critical unsharded, normal as elastic shards */
    MIRIAM_POLICY_SEQUENTIAL = 1,  /* one request at a time, critical first (baseline) */
    MIRIAM_POLICY_MULTISTREAM = 2, /* every task on its own stream, full kernels (baseline) */
    MIRIAM_POLICY_IB = 3           /* inter-stream barrier (baseline, §8.1.3): the tasks' full kernels
                                      advance in groups of one kernel per task, each stream waiting
                                      on the device for the previous group's kernels */
} miriam_policy;

typedef enum { MIRIAM_BACKEND_HIP = 0, MIRIAM_BACKEND_FAKE = 1 } miriam_backend;

typedef struct miriam_config {
    int32_t policy;          /* miriam_policy */
    int32_t backend;         /* miriam_backend; FAKE simulates a device on the host (tests) */
    int32_t n_be_streams;    /* streams for normal tasks (1..3) */
    int32_t inflight_depth;  /* max shards in flight per normal stream (>= 1) */
    double top_frac;         /* §6.3 kept fraction (0.2) */
    double max_blk_frac;     /* Eq. (5) MAX_blk as a fraction of the unsharded time (0.1) */
    double max_pt_frac;      /* Eq. (5) MAX_pt as a fraction of the unsharded time (0.1) */
    double quantum_us;       /* target duration of one normal shard */
    double inflight_us;      /* normal work (estimated from the task profile) kept queued on the GPU,
                                summed over the normal streams (each stream may always keep one
                                shard in flight); 0 = bounded by inflight_depth only */
    int32_t busy_policy;     /* normal shards while a critical kernel runs: 0 = Eq. (2) + WIScore x OScore
                                top fraction (the paper's rule), 1 = issue none until it completes,
                                2 = smallest feasible footprint (grid = Eq. (2) limit / 4, block 64) */
    int32_t log_launches;    /* keep miriam_launch_record entries (diagnostics, tests) */
    int32_t profile_reps;    /* timed repetitions per op when a task is created (HIP backend) */
    /* FAKE backend only: simulated compute units, WG slots per CU, ns per tile, launch ns */
    int32_t fake_n_cu, fake_slots_per_cu;
    double fake_tile_ns, fake_launch_ns;
    int32_t graphs;          /* 1 = capture each task's unsharded kernel sequence (grid = T, block 256
                                per op) into a HIP graph when the task is created, and run every
                                whole-request launch (critical requests; all requests under
                                SEQUENTIAL and MULTISTREAM) as one replay of it with one completion
                                event; 0 = launch op by op.  Normal elastic shards are launched
                                individually either way.  FAKE backend: ignored. */
    int32_t release_guard;   /* 1 = while no critical work runs, issue a normal shard only if the
                                normal work queued on the GPU plus that shard (estimated from the
                                task profiles) ends before the next timed critical release already
                                submitted; 0 = ignore future releases */
    int32_t warm_critical;   /* with release_guard: when normal work is first held for a critical
                                release, queue a kernel that reads the critical task's parameters
                                (weights, bias, normalisation vectors) behind the normal work in
                                flight (on the normal stream with the most), so the request finds
                                them in the caches;
                                the guard reserves its estimated time.  The task then owns a small
                                device table of its parameter ranges. */
    int32_t graph_chunk;     /* with graphs: most kernels per captured graph (a task's sequence is
                                captured as consecutive graphs launched back to back); 0 = one
                                graph per task */
    double arm_lead_us;      /* ELASTIC: this long before a timed critical release, queue the request's
                                kernels on the critical stream behind a one-wave gate kernel that
                                waits for a flag the dispatcher raises at the release (the gate gives
                                up 2 ms after the release at the latest); 0 = launch at the release.
                                Critical work released in between waits behind the gate. */
    int32_t segments;        /* ELASTIC: runs of consecutive ops of a task whose profiled unsharded
                                times sum to at most quantum_us are captured (at task creation) as
                                units; a normal request issues such a run as one launch with one
                                event while no critical kernel runs (ops launched unsharded).
                                Longer ops are sharded as usual. */
    double event_us;         /* ELASTIC: a normal launch records a completion event only once this
                                much estimated work has gathered on its stream since the last event,
                                and on each request's last launch (an event costs GPU time between
                                kernels); 0 = an event per launch */
    int32_t be_cu_reserve;   /* HIP backend, spatial isolation (any policy): the normal-task streams
                                are created with a compute-unit mask that leaves out this many CUs
                                (mask bits n_cu - be_cu_reserve .. n_cu - 1), so only the critical
                                stream, which keeps every CU, runs there; shard sizing still counts
                                every CU.  0 = no mask; must be below the device's CU count.
                                FAKE backend: ignored. */
    int32_t whole_when_clear; /* ELASTIC with release_guard and graphs: a normal request not yet
                                started, whose whole unsharded sequence (task profile) ends,
                                behind the normal work queued, before the next timed critical
                                release while no critical work is pending or running, is launched
                                as one replay of its captured graph (the greedy whole-GPU rule
                                taken to the whole request) instead of as shards; 0 = shards
                                only. */
    double whole_margin;     /* whole_when_clear: factor on the estimated time of the queued normal
                                work plus the request (profiled alone, warm caches); 0 = 2.0 */
    int32_t fake_fail_launch; /* FAKE backend only: the n-th launch (1-based, counting kernel launches
                                and captured replays since miriam_init) fails with MIRIAM_EHIP, ending
                                its request with that status; 0 = none (tests of the failure path) */
    int32_t crit_cu_exclusive; /* HIP backend, with be_cu_reserve > 0: the critical stream is created
                                with the complementary mask (the top be_cu_reserve CUs only), so
                                the two classes never share a CU; 0 = the critical stream keeps
                                every CU.  FAKE backend: ignored. */
} miriam_config;

typedef struct miriam_completion {
    uint64_t ticket;
    int32_t criticality;     /* 1 critical, 0 normal */
    int32_t status;          /* MIRIAM_OK or the error that failed the task */
    int64_t t_release_ns;    /* scheduled release (CLOCK_MONOTONIC) */
    int64_t t_start_ns;      /* first launch of the task */
    int64_t t_end_ns;        /* completion observed */
    int64_t deadline_ns;     /* absolute; 0 = none */
    int32_t deadline_met;    /* 1 if no deadline or t_end <= deadline */
    int32_t n_shards;        /* launches issued for this request */
} miriam_completion;

typedef struct miriam_stats {
    int64_t launches;         /* kernel launches issued */
    int64_t shards_sized;     /* normal shards sized next to a critical kernel */
    int64_t eq2_violations;   /* normal shards launched above the Eq. (2) limit (must stay 0) */
    int64_t decisions;        /* shard decisions taken */
    double decision_ns_total; /* host time spent deciding */
    int64_t completed;        /* requests completed */
    int64_t graph_launches;   /* whole requests run as one replay of their task's captured graph
                                 (each also counts its ops in `launches`) */
    int64_t warm_launches;    /* cache-warming kernels queued ahead of critical releases */
    int64_t armed_releases;   /* critical requests queued behind a gate ahead of their release */
    int64_t segment_launches; /* runs of short normal ops issued as one captured unit */
    int64_t barrier_groups;   /* IB: kernel groups issued behind an inter-stream barrier */
    int64_t whole_clear_launches; /* normal requests launched whole before a known release
                                     (whole_when_clear) */
    int64_t failed_requests;  /* requests ended by a failed launch (completion status < 0) */
    int64_t failed_pass_resets; /* ops of those requests whose split-K arrival counters were cleared
                                   in stream order after the failure (every op of the request's task) */
} miriam_stats;

/* Start the coordinator (creates its streams and its dispatcher thread). */
int miriam_init(const miriam_config *cfg);

/* Group ops (run in order) into one inference request template.  The task borrows the ops. */
int miriam_task_create(miriam_op *const *ops, int n_ops, miriam_task **out);

/* Submit one request of `task`.  criticality 1 = critical queue, 0 = normal queue.
 * release_ns: absolute CLOCK_MONOTONIC time before which it is held back (0 = now).
 * deadline_ns: absolute, 0 = none (recorded; ties among pending critical requests are
 * broken by earliest deadline).  Thread-safe. */
int miriam_submit(miriam_task *task, int criticality, int64_t release_ns, int64_t deadline_ns,
                  uint64_t *ticket_out);

/* Diagnostic of the release gate used by armed critical requests (arm_lead_us): queue one
 * gate kernel on `stream` (a hipStream_t; NULL = the null stream) behind a start event, with a
 * fresh flag that the host raises open_after_us microseconds after the launch (open_after_us
 * < 0: never) and a wall-clock limit of limit_us (1 .. 100000); wait for the stream and
 * return in *held_us the time between the events around the gate.  The gate always ends:
 * held_us is about min(open_after_us, limit_us).  Blocks the calling thread. */
int miriam_gate_check(void *stream, int64_t limit_us, int64_t open_after_us, double *held_us);

/* Non-blocking: move up to max_out completion records into out; returns the count. */
int miriam_poll(miriam_completion *out, int max_out);

/* Block until every submitted request has completed or timeout_ms passes
 * (MIRIAM_EBUSY on timeout). */
int miriam_drain(int64_t timeout_ms);

/* Counters since miriam_init. */
int miriam_stats_get(miriam_stats *out);

/* One launch issued by the coordinator (kept when cfg.log_launches is set). */
typedef struct miriam_launch_record {
    uint64_t ticket;       /* request the launch belongs to */
    int32_t op_index;      /* position of the op in its task */
    int32_t stream;        /* 0 = critical stream, 1.. = normal streams */
    int32_t criticality;
    int32_t grid, block;
    int32_t crit_busy;     /* a critical request was in flight when the shard was sized */
    int64_t shard_begin, shard_len, num_tiles;
    int64_t eq2_grid_limit; /* Eq. (2) grid limit in force (0 if none) */
    int64_t t_issue_ns;
    double est_us;         /* the coordinator's estimate of the launch's duration (task profile) */
} miriam_launch_record;

/* Copy up to max_out of the oldest unread launch records; returns the count. */
int miriam_launch_log(miriam_launch_record *out, int max_out);

/* MIRIAM_EBUSY if a submitted request of this task is pending. */
int miriam_task_destroy(miriam_task *t);

/* Drain, stop the dispatcher, destroy internal streams and events. */
int miriam_shutdown(void);

/* CLOCK_MONOTONIC in ns (the clock of release, start and end stamps). */
int64_t miriam_now_ns(void);

/* Text of the last error on the calling thread ("" if none). */
const char *miriam_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* MIRIAM_H */
