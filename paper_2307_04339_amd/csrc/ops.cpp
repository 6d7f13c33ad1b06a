// Operator registry of the elastic-kernel library: validation of operator
// descriptors, tile-space construction, kernel selection, and the elastic launch
// entry points (§6.1 elastic block, §6.2 elastic grid, §6.4 computation-based
// index functions).
#include <algorithm>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include <hip/hip_runtime.h>

#include "internal.h"

namespace miriam {

static thread_local std::string g_last_error;

void set_error(const std::string &msg) { g_last_error = msg; }

int hip_fail(hipError_t e, const char *what) {
    set_error(std::string(what) + ": " + hipGetErrorString(e));
    return MIRIAM_EHIP;
}

static int einval(const char *msg) {
    set_error(msg);
    return MIRIAM_EINVAL;
}

static int esize(int dtype) { return dtype == MIRIAM_F32 ? 4 : 2; }
static int vec_elems(int dtype) { return 16 / esize(dtype); }
static bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

static int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

static int get_igemm_table(int dtype, int cfg, int lay, const void *out[3], int *lds) {
    switch (dtype) {
    case MIRIAM_F32: return igemm_kernels_f32(cfg, lay, out, lds);
    case MIRIAM_F16: return igemm_kernels_f16(cfg, lay, out, lds);
    case MIRIAM_BF16: return igemm_kernels_bf16(cfg, lay, out, lds);
    default: return -1;
    }
}

static int get_igemm_mi_table(int dtype, int cfg, bool uni, const void *out[3], int *lds) {
    switch (dtype) {
    case MIRIAM_F32: return igemm_mi_kernels_f32(cfg, uni, out, lds);
    case MIRIAM_F16: return igemm_mi_kernels_f16(cfg, uni, out, lds);
    case MIRIAM_BF16: return igemm_mi_kernels_bf16(cfg, uni, out, lds);
    default: return -1;
    }
}

static int tile_m_of(int cfg) { return cfg == CFG_32 ? 32 : (cfg == CFG_64 ? 64 : (cfg == CFG_256x128 ? 256 : 128)); }  // halo: 4 x 32 pixels
static int tile_n_of(int cfg) { return cfg == CFG_32 ? 32 : (cfg == CFG_64 || cfg == CFG_128x64 ? 64 : 128); }
constexpr int TILE_SKINNY = 5;  // descriptor tile code of the split-K skinny kernel

static int device_cus();

// Column groups of 16 per skinny tile: two (one activation load per two weight loads) when
// the op still has about four tiles per CU at 32 columns with slices of 1024 K values or more
// (VGG-16 fc6, 8 x 4096 x 25088: 51.1 -> 48.7 us); one otherwise, where wider tiles left too
// few tiles (fc7 15.0 / 15.1 us, fc8 10.5 / 11.1, ResNet-18 fc 6.6 / 8.0).
static int skinny_cols(int64_t M, int64_t Nc, int64_t K) {
    (void)M;
    return cdiv(Nc, 32) * std::max<int64_t>(2, K / 1024) >= 4 * (int64_t)device_cus() ? 2 : 1;
}

// Fill the per-physical-block residency of the op's kernels.  Without a device
// the figures stay 0 ("unknown"); the error state of the runtime is cleared.
static void query_occupancy(miriam_op *op) {
    op->full_grid = op->T;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return;
    }
    for (int i = 0; i < 3; ++i) {
        int n = 0;
        const int block = 64 << i;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, op->kern[i], block, 0) == hipSuccess)
            op->max_wg_per_cu[i] = n;
        else
            (void)hipGetLastError();
    }
    // kernels that keep operands resident across tiles run persistently: as many workgroups
    // as fit the device at once (one per tile when that is fewer)
    if (op->family == FAM_IGEMM && op->lay == LAY_RW && op->max_wg_per_cu[2] > 0)
        op->full_grid = std::min<int64_t>(op->T, (int64_t)device_cus() * op->max_wg_per_cu[2]);
    // the pipelined contraction with more tiles than resident workgroups, but at most twice as
    // many: half as many workgroups, two tiles each, none waiting for a second dispatch (VGG-16
    // b8 fp16, 128x128 tiles on 512 resident slots, cold caches: conv2_2's 784 tiles 50.8 ->
    // 49.1 us, conv2_1 34.3 -> 33.1 us, same bits; a grid of the 512 slots, 54.5 us, gives the
    // second tiles to whole dies, since consecutive ranks share a die)
    if (op->family == FAM_IGEMM && (op->lay == LAY_VEC || op->lay == LAY_VEC_UNI) && op->max_wg_per_cu[2] > 0) {
        const int64_t slots = (int64_t)device_cus() * op->max_wg_per_cu[2];
        if (op->T > slots && op->T <= 2 * slots) op->full_grid = cdiv(op->T, 2);
    }
}

static Epilogue make_epi(const miriam_op_desc &d, int64_t C) {
    Epilogue e;
    e.bias = static_cast<const float *>(d.bias);
    e.bn = static_cast<const float *>(d.bn);
    e.eps = d.eps;
    e.act = d.act;
    e.flags = d.flags & (MIRIAM_EPI_BIAS | MIRIAM_EPI_BN | MIRIAM_EPI_RESIDUAL);
    e.C = C;
    return e;
}

static int check_epi(const miriam_op_desc &d, int extra_flags = 0) {
    if (d.act < MIRIAM_ACT_NONE || d.act > MIRIAM_ACT_GELU) return einval("unknown activation");
    if (d.flags & ~(MIRIAM_EPI_BIAS | MIRIAM_EPI_BN | MIRIAM_EPI_RESIDUAL | extra_flags)) return einval("unknown epilogue flag");
    if ((d.flags & MIRIAM_EPI_BIAS) && !d.bias) return einval("bias flag without bias pointer");
    if ((d.flags & MIRIAM_EPI_BN) && !d.bn) return einval("bn flag without bn pointer");
    if ((d.flags & MIRIAM_EPI_RESIDUAL) && !d.residual) return einval("residual flag without residual pointer");
    if ((d.flags & MIRIAM_EPI_BN) && !(d.eps >= 0.0f)) return einval("negative eps");
    return MIRIAM_OK;
}

// Compute units of the current device (256 when no device is visible).
static int device_cus() {
    static int n = 0;
    if (n == 0) {
        int dev = 0;
        hipDeviceProp_t p;
        if (hipGetDevice(&dev) == hipSuccess && hipGetDeviceProperties(&p, dev) == hipSuccess)
            n = p.multiProcessorCount;
        else {
            (void)hipGetLastError();
            n = 256;
        }
    }
    return n;
}

// Contraction tile choice, from per-layer sweeps of the pipelined kernel on the CNN
// workloads: 128x128 when N > 64 and it still gives 1.5 tiles per compute unit (its
// operands cost the fewest bytes per flop); otherwise the largest of 128x64, 64x64,
// 32x32 that gives three quarters of a tile per compute unit (a smaller tile beats a
// larger one once the larger leaves CUs idle), or 1.1 tiles per compute unit when K is at
// most four 128-byte chunks: such a tile is mostly its epilogue, and more tiles in flight
// hide it (MobileNetV2 b16 / b32 1x1 projections and expansions, bf16, with 0.77-0.88 larger
// tiles per CU: 9.0 -> 8.2, 10.6 -> 9.7, 10.9 -> 9.9, 11.3 -> 10.2 us; with 1.15 per CU the
// larger tile still wins, 8.5 against 10.7 us; the encoder's K = 768 products keep 64x64 at
// three quarters of a tile per CU).  256x128 never won: too few tiles.
static int choose_cfg(int64_t batch, int64_t M, int64_t N, int64_t k_chunks) {
    const int64_t cus = device_cus();
    const int64_t fill = k_chunks <= 4 ? cus * 11 / 10 : cus * 3 / 4;
    if (N > 64 && batch * cdiv(M, 128) * cdiv(N, 128) >= cus * 3 / 2) return CFG_128;
    if (batch * cdiv(M, 128) * cdiv(N, 64) >= fill) return CFG_128x64;
    if (batch * cdiv(M, 64) * cdiv(N, 64) >= fill) return CFG_64;
    return CFG_32;
}

// ---------------------------------------------------------- device scratch
// Split-K workspace of ops created by miriam_op_create_noalloc: a static device array per GPU
// (held until the process ends), shared by every such op on that GPU.  Host code never uses
// the array's name as an address: its device address is looked up once per device with
// hipGetSymbolAddress (with that device current) and kept in g_scratch_ptr.  Layout: the
// arrival counters of every such op start at offset 0 (a whole pass leaves each count it
// used at zero, so the region is all zeros between passes whichever op ran last), the fp32
// partials at kScratchCounters; passes over two such ops must not overlap in time.
constexpr size_t kScratchBytes = (size_t)MIRIAM_NOALLOC_SCRATCH_BYTES;
constexpr size_t kScratchCounters = (size_t)1 << 20;
static __device__ __align__(256) char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void *g_scratch_ptr[kMaxDevices];

static int scratch_ptr(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) {
        set_error("device index beyond the scratch table");
        return MIRIAM_ERANGE;
    }
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) return hip_fail(e, "hipGetSymbolAddress (scratch)");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return MIRIAM_OK;
}

// Split-K workspace: wbytes of fp32 partials and cbytes of arrival counters, the counters zeroed.
// Regular ops allocate it; no-alloc ops (op->noalloc) take it from the device scratch.  Returns
// 1 when placed, 0 when the op runs without split K instead (allocation failed and the split was
// the library's choice), < 0 on error (the caller asked for the split, `required`).
static int alloc_workspace(miriam_op *op, size_t wbytes, size_t cbytes, bool required) {
    if (op->noalloc) {
        if (cbytes > kScratchCounters || wbytes > kScratchBytes - kScratchCounters) {
            if (!required) return 0;
            set_error("split-K workspace exceeds the no-alloc device scratch (" +
                      std::to_string((kScratchBytes - kScratchCounters) >> 20) + " MiB of partials, " +
                      std::to_string(kScratchCounters / 4) + " counters)");
            return MIRIAM_ERANGE;
        }
        void *base = nullptr;
        int rc = scratch_ptr(&base);
        if (rc != MIRIAM_OK) return rc;
        char *b = static_cast<char *>(base);
        hipError_t e = hipMemsetAsync(b, 0, cbytes, nullptr);
        if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
        if (e != hipSuccess) return hip_fail(e, "clearing the split-K counters in the device scratch");
        op->counters = b;
        op->work = b + kScratchCounters;
        op->counters_bytes = cbytes;
        return 1;
    }
    if (hipMalloc(&op->work, wbytes) == hipSuccess && hipMalloc(&op->counters, cbytes) == hipSuccess &&
        hipMemset(op->counters, 0, cbytes) == hipSuccess && hipDeviceSynchronize() == hipSuccess) {
        op->counters_bytes = cbytes;
        return 1;
    }
    (void)hipGetLastError();
    if (op->work) (void)hipFree(op->work);
    if (op->counters) (void)hipFree(op->counters);
    (void)hipGetLastError();
    op->work = op->counters = nullptr;
    if (!required) return 0;
    set_error("split-K workspace allocation failed");
    return MIRIAM_ENOMEM;
}

// Release an op's device memory (none for no-alloc ops: their workspace is the scratch).
static void free_device(miriam_op *op) {
    if (op->noalloc) return;
    if (op->work) (void)hipFree(op->work);
    if (op->counters) (void)hipFree(op->counters);
    if (op->rowtab) (void)hipFree(op->rowtab);
}

static int create_igemm(miriam_op *op) {
    const miriam_op_desc &d = op->d;
    IgemmArgs &a = op->ig;
    std::memset(&a, 0, sizeof(a));
    const int es = esize(d.dtype), V = vec_elems(d.dtype);
    int64_t batch = 1;
    bool a_vec = true, b_vec = true;
    const bool nmaj = d.kind == MIRIAM_OP_BGEMM && d.b_nmajor;
    if (d.kind == MIRIAM_OP_CONV2D) {
        if (d.n < 1 || d.h < 1 || d.w < 1 || d.c < 1 || d.k < 1 || d.kh < 1 || d.kw < 1)
            return einval("conv2d: sizes must be >= 1");
        if (d.stride < 1 || d.pad < 0) return einval("conv2d: stride >= 1 and pad >= 0 required");
        if (d.groups != 0 && d.groups != 1) return einval("conv2d: groups must be 1 (use DWCONV for depthwise)");
        a.H = d.h; a.W = d.w; a.C = d.c;
        a.ldx = d.ldx > 0 ? d.ldx : d.c;
        if (a.ldx < d.c) return einval("conv2d: ldx < c");
        a.KH = (int32_t)d.kh; a.KW = (int32_t)d.kw; a.stride = (int32_t)d.stride; a.pad = (int32_t)d.pad;
        a.Ho = (d.h + 2 * d.pad - d.kh) / d.stride + 1;
        a.Wo = (d.w + 2 * d.pad - d.kw) / d.stride + 1;
        if (d.h + 2 * d.pad < d.kh || d.w + 2 * d.pad < d.kw || a.Ho < 1 || a.Wo < 1)
            return einval("conv2d: kernel larger than padded input");
        a.M = d.n * a.Ho * a.Wo;
        a.Nc = d.k;
        a.K = d.kh * d.kw * d.c;
        a.ldw = d.ldw > 0 ? d.ldw : a.K;
        a.ldy = d.ldy > 0 ? d.ldy : d.k;
        if (a.ldw < a.K || a.ldy < d.k) return einval("conv2d: row stride too small");
        a.img_x = d.h * d.w * a.ldx;
        a.bdiv = 1;
        a_vec = (d.c % V == 0) && (a.ldx % V == 0) && aligned16(d.x);
    } else {
        if (d.m < 1 || d.nn < 1 || d.kk < 1) return einval("gemm: m, nn, kk must be >= 1");
        a.H = 1; a.W = 1; a.C = d.kk; a.Ho = 1; a.Wo = 1;
        a.KH = 1; a.KW = 1; a.stride = 1; a.pad = 0;
        a.M = d.m; a.Nc = d.nn; a.K = d.kk;
        a.ldx = d.ldx > 0 ? d.ldx : d.kk;
        a.ldw = d.ldw > 0 ? d.ldw : (nmaj ? d.nn : d.kk);
        a.ldy = d.ldy > 0 ? d.ldy : d.nn;
        if (a.ldx < d.kk || a.ldy < d.nn || a.ldw < (nmaj ? d.nn : d.kk)) return einval("gemm: row stride too small");
        a.img_x = a.ldx;
        a.bdiv = 1;
        if (d.kind == MIRIAM_OP_BGEMM) {
            if (d.batch < 1 || d.batch_div < 1) return einval("bgemm: batch and batch_div must be >= 1");
            batch = d.batch;
            a.bdiv = d.batch_div;
            a.sx0 = d.sx0; a.sx1 = d.sx1; a.sw0 = d.sw0; a.sw1 = d.sw1; a.sy0 = d.sy0; a.sy1 = d.sy1;
            if (a.sx0 < 0 || a.sx1 < 0 || a.sw0 < 0 || a.sw1 < 0 || a.sy0 < 0 || a.sy1 < 0)
                return einval("bgemm: negative batch stride");
        }
        a_vec = (d.kk % V == 0) && (a.ldx % V == 0) && (a.sx0 % V == 0) && (a.sx1 % V == 0) && aligned16(d.x);
    }
    if (nmaj)
        b_vec = (d.nn % V == 0) && (a.ldw % V == 0) && (a.sw0 % V == 0) && (a.sw1 % V == 0) && aligned16(d.wt);
    else
        b_vec = (a.K % V == 0) && (a.ldw % V == 0) && (a.sw0 % V == 0) && (a.sw1 % V == 0) && aligned16(d.wt);
    if (nmaj && d.dtype == MIRIAM_F32) return einval("bgemm: [k][n] right operand needs fp16/bf16");
    if (d.kind == MIRIAM_OP_CONV2D && d.b_nmajor) return einval("conv2d: weights must be [Cout][KH][KW][Cin]");
    int rc = check_epi(d, MIRIAM_INDEX_MEMORY);
    if (rc) return rc;
    const bool memidx = (d.flags & MIRIAM_INDEX_MEMORY) != 0;
    if (memidx && op->noalloc) return einval("memory-based index function: needs a device table (not with no-alloc ops)");
    a.x = d.x; a.w = d.wt; a.y = d.y; a.res = d.residual;
    a.epi = make_epi(d, a.Nc);
    if (a.Ho * a.Wo >= (int64_t)INT32_MAX) return einval("contraction: output image too large for 32-bit pixel indexing");
    a.fd_howo = make_fastdiv((uint32_t)(a.Ho * a.Wo));
    a.fd_wo = make_fastdiv((uint32_t)a.Wo);

    a.vec_store = (a.ldy % V == 0) && (a.sy0 % V == 0) && (a.sy1 % V == 0) && aligned16(d.y) &&
                  (!(d.flags & MIRIAM_EPI_RESIDUAL) || aligned16(d.residual));
    // fully connected layers at small batch: split-K skinny kernel
    // (its operands are read with 32-bit byte offsets: the M activation rows and a tile's
    // weight rows must span less than 2^31 bytes)
    const int skinny_cg = skinny_cols(a.M, a.Nc, a.K);
    const bool skinny_ok = d.kind == MIRIAM_OP_GEMM && d.dtype != MIRIAM_F32 && a.M <= 16 && a_vec && b_vec &&
                           ((a.M - 1) * a.ldx + a.K) * es < ((int64_t)1 << 31) &&
                           ((16 * skinny_cg - 1) * a.ldw + a.K) * es < ((int64_t)1 << 31);
    // direct 3x3 / stride-1 convolution with the input patch in LDS: C a whole number of
    // 128-byte chunks, aligned rows.  The library picks it for layers with at most 64 output
    // channels (one n tile) when it gives 1.5 tiles per CU and the 32-pixel tile columns waste
    // at most a quarter of the output width; on wider layers the 128x128 / 128x64 implicit
    // GEMM measured as fast or faster (VGG-16 b8: conv1_2 84 us vs 95 us at 128x64; conv3_2
    // 64 us vs 54 us at 128x128)
    const int64_t kt = 128 / es;
    const bool halo_ok = d.kind == MIRIAM_OP_CONV2D && d.kh == 3 && d.kw == 3 && d.stride == 1 && a_vec && b_vec &&
                         d.c % kt == 0 && d.ksplit <= 1;
    const int64_t halo_tx = cdiv(a.Wo, 32), halo_ty = cdiv(a.Ho, 4);
    const int64_t halo_T = d.n * halo_ty * halo_tx * cdiv(a.Nc, 64);
    // 4x32-pixel x 64-channel tiles with the weights resident in registers (fp16/bf16, a
    // workgroup's filter slice fits its registers): 3x3 stride 1 with C in {8, 16, 32, 64} and
    // at most 64 output channels, 3x3 stride 2 on 8-channel images, 1x1 stride 1 with C in
    // {16, 24, 32, 64} and any number of output channels.  Chosen over the LDS-patch kernel
    // and the implicit GEMM wherever it applies with 1.5 tiles per CU.
    const bool rw_shape = (d.kh == 3 && d.kw == 3 && d.stride == 1 && (d.c == 8 || d.c == 16 || d.c == 32 || d.c == 64) &&
                           a.Nc <= 64) ||
                          (d.kh == 3 && d.kw == 3 && d.stride == 2 && d.c == 8 && a.Nc <= 64) ||
                          (d.kh == 1 && d.kw == 1 && d.stride == 1 && d.pad == 0 &&
                           (d.c == 16 || d.c == 24 || d.c == 32 || d.c == 64));
    const bool rw_ok = d.kind == MIRIAM_OP_CONV2D && d.dtype != MIRIAM_F32 && rw_shape && a_vec && b_vec &&
                       d.ksplit <= 1 && a.img_x * esize(d.dtype) < ((int64_t)1 << 31);
    const int64_t rw_T = d.n * halo_ty * halo_tx * cdiv(a.Nc, 64);
    int cfg = d.tile;
    // the memory-based index function is served by the pipelined kernel only
    if (cfg == 0 && !memidx && rw_ok && rw_T >= (int64_t)device_cus() * 3 / 2 && halo_tx * 32 * 4 <= a.Wo * 5)
        cfg = CFG_RW;
    if (cfg == 0 && !memidx && halo_ok && a.Nc <= 64 && halo_T >= (int64_t)device_cus() * 3 / 2 &&
        halo_tx * 32 * 4 <= a.Wo * 5)
        cfg = CFG_HALO;
    if (cfg == 0) cfg = (skinny_ok && !memidx) ? TILE_SKINNY : choose_cfg(batch, a.M, a.Nc, cdiv(a.K * es, 128));
    if (memidx && (cfg == CFG_RW || cfg == CFG_HALO || cfg == TILE_SKINNY))
        return einval("memory-based index function: tiles 1..4 only (pipelined contraction kernel)");
    if (cfg == CFG_RW) {
        if (!rw_ok) return einval("tile 8 (resident-weight direct conv) needs an fp16/bf16 conv that is 3x3 stride 1 with C in {8,16,32,64} and at most 64 output channels, 3x3 stride 2 with C = 8 and at most 64 output channels, or 1x1 stride 1 pad 0 with C in {16,24,32,64}; 16-byte rows; images under 2 GiB; no split K");
        a.tX = halo_tx;
        a.tY = halo_ty;
        a.mT = halo_ty * halo_tx;
        a.nT = cdiv(a.Nc, 64);
        a.ksplit = 1;
        a.cps = 1;
        {
            // whole 16-byte output pieces within 2^31 bytes: the kernel's buffer-store epilogue
            const int64_t y_span = d.n * a.Ho * a.Wo * a.ldy * (int64_t)esize(d.dtype);
            a.y_bytes = (a.vec_store && a.Nc % vec_elems(d.dtype) == 0 && y_span < ((int64_t)1 << 31)) ? (uint32_t)y_span : 0u;
        }
        op->T = d.n * a.mT * a.nT;
        op->cfg = cfg;
        op->tile_m = 128;
        op->tile_n = 64;
        op->lay = LAY_RW;
        if (rw_kernels(d.dtype, d.kh, d.stride, d.c, op->kern, &op->lds_bytes) != 0)
            return einval("no resident-weight kernel for this dtype / shape");
    } else if (cfg == CFG_HALO) {
        if (!halo_ok) return einval("tile 7 (direct 3x3) needs a 3x3 stride-1 conv with C a multiple of the 128-byte chunk, 16-byte rows and no split K");
        a.tX = halo_tx;
        a.tY = halo_ty;
        a.mT = halo_ty * halo_tx;
        a.nT = cdiv(a.Nc, 64);
        a.ksplit = 1;
        a.cps = (int32_t)cdiv(a.K, kt);
        op->T = d.n * a.mT * a.nT;
        op->cfg = cfg;
        op->tile_m = 128;
        op->tile_n = 64;
        op->lay = LAY_HALO;
        if (get_igemm_table(d.dtype, cfg, op->lay, op->kern, &op->lds_bytes) != 0)
            return einval("no direct 3x3 kernel for this dtype");
    } else if (cfg == TILE_SKINNY) {
        if (!skinny_ok) return einval("skinny tile needs an fp16/bf16 GEMM with m <= 16 and 16-byte rows");
        op->family = FAM_SKINNY;
        const int cg = skinny_cg;
        const int64_t group = skinny_group(cg);
        a.mT = 1;
        a.nT = cdiv(a.Nc, 16 * cg);
        // K slices: each slice keeps at least one group per logical wave.  The library choice
        // takes the fewest slices that give every CU a tile, twice as many when those slices
        // would still hold 8192 K values or more (two tiles per CU, each streaming a long
        // slice), and keeps slices of about 1024 K values or more.  Measured unsharded (cold
        // caches, VGG-16 b8 fp16): fc6 (25088 -> 4096, 128 32-column tiles) 46.9 / 50.4 / 42.9 /
        // 51.0 / 46.8 / 48.0 us at 2 / 3 / 4 / 5 / 6 / 8 slices; fc7 (4096 -> 4096, 256 tiles)
        // 13.1 / 14.0 / 15.1 us at 1 / 2 / 4; fc8 (4096 -> 1000, 63 tiles) 10.8 / 10.3 / 10.4 /
        // 12.3 us at 2 / 3 / 4 / 8; the MobileNetV2 b16 classifier (1280 -> 1000) 8.8 / 9.4 us
        // at 1 / 2.
        const int64_t max_ks = std::max<int64_t>(1, cdiv(a.K, group) / 4);
        int64_t lib_ks = cdiv((int64_t)device_cus(), a.nT);
        if (a.K / lib_ks >= 8192) lib_ks *= 2;
        lib_ks = std::min<int64_t>(std::min<int64_t>(lib_ks, max_ks), std::max<int64_t>(1, a.K / 1024));
        int64_t ks = d.ksplit > 1 ? std::min<int64_t>(d.ksplit, max_ks) : d.ksplit == 1 ? 1 : lib_ks;
        ks = std::max<int64_t>(1, ks);
        // slice length as the kernel derives it (whole numbers of 4 groups); count only the
        // slices that hold K values
        ks = cdiv(a.K, cdiv(a.K, ks * 4 * group) * 4 * group);
        a.ksplit = 1;
        if (ks > 1) {
            const size_t wbytes = (size_t)a.nT * (size_t)ks * 16 * 16 * cg * sizeof(float);
            const size_t cbytes = (size_t)a.nT * sizeof(int32_t);
            const int wr = alloc_workspace(op, wbytes, cbytes, d.ksplit > 1);
            if (wr < 0) return wr;
            if (wr > 0) {
                a.ksplit = (int32_t)ks;
                a.work = static_cast<float *>(op->work);
                a.counters = static_cast<int32_t *>(op->counters);
            }
        }
        op->T = a.nT * a.ksplit;
        op->cfg = cfg;
        op->tile_m = 16;
        op->tile_n = 16 * cg;
        op->lay = LAY_VEC;
        op->lds_bytes = 4 * 16 * (16 * cg + 1) * 4;
        if (skinny_kernels(d.dtype, cg, op->kern) != 0) return einval("no skinny kernel for this dtype");
    } else {
        if (cfg < CFG_32 || cfg > CFG_256x128 || cfg == TILE_SKINNY) return einval("unknown tile configuration");
        a.mT = cdiv(a.M, tile_m_of(cfg));
        a.nT = cdiv(a.Nc, tile_n_of(cfg));
        op->T = batch * a.mT * a.nT;
        a.ksplit = 1;
        a.cps = (int32_t)cdiv(a.K, d.dtype == MIRIAM_F32 ? 32 : 64);  // K chunks of one 128-byte row
        // split K over workgroups with a fixed-order reduction (pipelined kernel only) when
        // the caller asks for it, or by the library's choice: the most slices, up to 4, that
        // keep every slice of every tile resident at once (two workgroups per CU), with 8 or
        // more K chunks per slice when the op fills at most half the CUs and 32 or more when
        // it fills up to all of them.  A slice's latency-bound chunk loop is that much shorter;
        // the partial tiles cost one device-coherent write and read each (1 KB per store
        // instruction).  Measured (unsplit -> split): ResNet-18 b1 layer 3 14.5 -> 11.2 us and
        // layer 4 21.6 -> 12.5 us at 4 slices; encoder b1 FFN2 (96 32x32 tiles) 16.9 -> 12.7 us
        // at 4; VGG-16 b8 conv5_x (200 64x64 tiles, 72 chunks) 27.8 -> 24.0 us at 2.  Lost:
        // encoder b4 FFN2 (192 64x64 tiles, 48 chunks) 22.2 -> 24.0 us at 2; ops whose slices
        // would not all be resident (conv4_2, 392 tiles: 49.7 -> 62.5 us at 2).
        const int64_t nch = a.cps;
        const bool vec_layout = (a_vec && b_vec && !nmaj);
        int64_t want_ks = d.ksplit;
        if (d.ksplit == 0 && vec_layout) {
            const int64_t slots = 2 * (int64_t)device_cus();
            const int64_t min_chunks = op->T * 2 <= (int64_t)device_cus() ? 8 : 32;
            want_ks = 1;
            for (int64_t k = 2; k <= 4; ++k)
                if (op->T * k <= slots && nch / k >= min_chunks) want_ks = k;
        }
        if (want_ks > 1 && vec_layout) {
            int64_t ks = std::min<int64_t>(want_ks, nch);
            if (ks > 1) {
                const int64_t cps = cdiv(nch, ks);
                ks = cdiv(nch, cps);  // no empty slices
                const size_t wbytes = (size_t)op->T * (size_t)ks * tile_m_of(cfg) * tile_n_of(cfg) * sizeof(float);
                const size_t cbytes = (size_t)op->T * sizeof(int32_t);
                const int wr = alloc_workspace(op, wbytes, cbytes, d.ksplit > 1);
                if (wr < 0) return wr;
                if (wr > 0) {
                    a.ksplit = (int32_t)ks;
                    a.cps = (int32_t)cps;
                    a.work = static_cast<float *>(op->work);
                    a.counters = static_cast<int32_t *>(op->counters);
                    op->T *= ks;
                }
            }
        }
        op->cfg = cfg;
        op->tile_m = tile_m_of(cfg);
        op->tile_n = tile_n_of(cfg);
        if (nmaj) op->lay = (a_vec && b_vec) ? LAY_VEC_NB : LAY_SCALAR_NB;
        else op->lay = (a_vec && b_vec) ? LAY_VEC : LAY_SCALAR;
        // every 128-byte K chunk inside one filter tap: per-lane pointers advance per chunk
        // the chunk-uniform decode reads its operands as buffers with 32-bit offsets: spans in
        // bytes from a batch entry's base, below 2^31 (zeros past the end come from the range check)
        {
            const int64_t x_span = (d.kind == MIRIAM_OP_CONV2D ? d.n * a.img_x : (a.M - 1) * a.ldx + a.K) * es;
            const int64_t w_span = ((a.Nc - 1) * a.ldw + a.K) * es;
            if (op->lay == LAY_VEC && a.C % (128 / es) == 0 && x_span < ((int64_t)1 << 31) &&
                w_span < ((int64_t)1 << 31)) {
                op->lay = LAY_VEC_UNI;
                a.x_bytes = (uint32_t)x_span;
                a.w_bytes = (uint32_t)w_span;
            }
            // the epilogue stores whole 16-byte pieces as buffer stores with 32-bit offsets
            // when there is one batch entry and the output spans less than 2^31 bytes
            const int64_t y_span = a.M * a.ldy * es;
            if (batch == 1 && a.vec_store && a.Nc % (16 / es) == 0 && y_span < ((int64_t)1 << 31))
                a.y_bytes = (uint32_t)y_span;
        }
        if (!memidx && get_igemm_table(d.dtype, cfg, op->lay, op->kern, &op->lds_bytes) != 0)
            return einval("no kernel for this dtype / layout");
        if (memidx) {
            if (op->lay != LAY_VEC && op->lay != LAY_VEC_UNI)
                return einval("memory-based index function needs 16-byte aligned K-major operands");
            if (get_igemm_mi_table(d.dtype, cfg, op->lay == LAY_VEC_UNI, op->kern, &op->lds_bytes) != 0)
                return einval("memory-based index function: tiles 1..4 only");
            // host-computed index table: one (image, h0, w0, valid) row per tile row
            const int64_t rows = a.mT * tile_m_of(cfg);
            std::vector<int32_t> tab((size_t)rows * 4, 0);
            const int64_t howo = a.Ho * a.Wo;
            for (int64_t m = 0; m < rows; ++m) {
                const int64_t mm = m < a.M ? m : 0;
                const int64_t img = mm / howo, pq = mm % howo, p = pq / a.Wo, q = pq % a.Wo;
                int32_t *e = &tab[(size_t)m * 4];
                e[0] = (int32_t)img;
                e[1] = (int32_t)(p * a.stride - a.pad);
                e[2] = (int32_t)(q * a.stride - a.pad);
                e[3] = m < a.M ? 1 : 0;
            }
            const size_t tb = tab.size() * sizeof(int32_t);
            if (hipMalloc(&op->rowtab, tb) != hipSuccess) {
                (void)hipGetLastError();
                op->rowtab = nullptr;
                set_error("memory-based index table allocation failed");
                return MIRIAM_ENOMEM;
            }
            if (hipMemcpy(op->rowtab, tab.data(), tb, hipMemcpyHostToDevice) != hipSuccess) {
                (void)hipGetLastError();
                set_error("memory-based index table upload failed");
                return MIRIAM_ENOMEM;
            }
            a.rowtab = static_cast<const int32_t *>(op->rowtab);
        }
    }
    // kernels index tiles, rows and batch entries with 32-bit arithmetic
    if (op->T >= (int64_t)INT32_MAX || a.M >= (int64_t)INT32_MAX || batch >= (int64_t)INT32_MAX)
        return einval("contraction too large for 32-bit tile indexing");
    op->flops = 2.0 * (double)batch * (double)a.M * (double)a.Nc * (double)a.K;
    const double xin = d.kind == MIRIAM_OP_CONV2D ? (double)d.n * d.h * d.w * d.c : (double)batch * a.M * a.K;
    const double win = (d.kind == MIRIAM_OP_BGEMM ? (double)batch : 1.0) * (double)a.Nc * a.K;
    const double yout = (double)batch * a.M * a.Nc;
    op->bytes = es * (xin + win + yout * ((d.flags & MIRIAM_EPI_RESIDUAL) ? 2.0 : 1.0));
    return MIRIAM_OK;
}

static int create_pix(miriam_op *op) {
    const miriam_op_desc &d = op->d;
    PixArgs &a = op->px;
    std::memset(&a, 0, sizeof(a));
    const int es = esize(d.dtype), V = vec_elems(d.dtype);
    int kind;
    if (d.kind == MIRIAM_OP_BN_ACT) {
        if (d.m < 1 || d.nn < 1) return einval("bn_act: m, nn must be >= 1");
        kind = PIX_EW;
        a.N = d.m; a.H = 1; a.W = 1; a.C = d.nn; a.Ho = 1; a.Wo = 1;
        a.KH = 1; a.KW = 1; a.stride = 1; a.pad = 0;
    } else {
        if (d.n < 1 || d.h < 1 || d.w < 1 || d.c < 1 || d.kh < 1 || d.kw < 1)
            return einval("pixel op: sizes must be >= 1");
        if (d.stride < 1 || d.pad < 0) return einval("pixel op: stride >= 1 and pad >= 0 required");
        if (d.h + 2 * d.pad < d.kh || d.w + 2 * d.pad < d.kw) return einval("pixel op: window larger than padded input");
        if (d.pad >= d.kh || d.pad >= d.kw) return einval("pixel op: pad must be smaller than the window");
        kind = d.kind == MIRIAM_OP_DWCONV ? PIX_DW : (d.kind == MIRIAM_OP_POOL_MAX ? PIX_MAX : PIX_AVG);
        if (kind == PIX_DW && d.k != 0 && d.k != d.c) return einval("dwconv: k must equal c");
        if (kind == PIX_DW && d.groups != 0 && d.groups != d.c) return einval("dwconv: groups must equal c");
        a.N = d.n; a.H = d.h; a.W = d.w; a.C = d.c;
        a.KH = (int32_t)d.kh; a.KW = (int32_t)d.kw; a.stride = (int32_t)d.stride; a.pad = (int32_t)d.pad;
        a.Ho = (d.h + 2 * d.pad - d.kh) / d.stride + 1;
        a.Wo = (d.w + 2 * d.pad - d.kw) / d.stride + 1;
        if (kind != PIX_DW && (d.flags != 0 || d.act != 0)) return einval("pooling has no epilogue");
    }
    if (d.ldx != 0 || d.ldy != 0) return einval("pixel op: dense layouts only");
    int rc = check_epi(d);
    if (rc) return rc;
    const bool vec = (a.C % V == 0) && aligned16(d.x) && aligned16(d.y) &&
                     (kind != PIX_DW || aligned16(d.wt)) &&
                     (!(d.flags & MIRIAM_EPI_RESIDUAL) || aligned16(d.residual)) &&
                     (!(d.flags & MIRIAM_EPI_BIAS) || aligned16(d.bias)) && (!(d.flags & MIRIAM_EPI_BN) || aligned16(d.bn));
    const int v = vec ? V : 1;
    a.x = d.x; a.w = d.wt; a.y = d.y; a.res = d.residual;
    a.epi = make_epi(d, a.C);
    // 3x3 depthwise with 16-byte channel vectors: strips of kDwStrip output pixels per item
    // (a third of the input loads per output), where the strips still give three quarters of a
    // tile per CU; measured on MobileNetV2 (bf16, cold caches): b16 56x56x144 22.2 -> 19.2 us,
    // 112x112x32 21.8 -> 18.9 us, 28x28x192 12.8 -> 11.2 us; b32 14x14x576 15.1 -> 11.8 us,
    // 14x14x384 12.8 -> 11.1 us; with fewer tiles (b16 14x14x384 at 0.66 per CU, 7x7x960 at
    // 0.4) the per-pixel kernel stays faster (9.0 against 9.4, 7.9 against 8.9 us), as does
    // stride 2 (112 -> 56, C = 96: 21.4 against 22.2 us)
    // (16-bit types only: fp32 keeps the per-pixel kernel)
    if (kind == PIX_DW && vec && d.dtype != MIRIAM_F32 && a.KH == 3 && a.KW == 3 && a.stride == 1 &&
        cdiv(a.N * a.Ho * cdiv(a.Wo, kDwStrip) * (a.C / v), 256) >= 3 * (int64_t)device_cus() / 4)
        kind = PIX_DW3;
    a.Ws = kind == PIX_DW3 ? cdiv(a.Wo, kDwStrip) : a.Wo;
    a.items = a.N * a.Ho * a.Ws * (a.C / v);
    if (a.items >= (int64_t)INT32_MAX || a.N * a.Ho * a.Wo * (a.C / v) >= (int64_t)INT32_MAX)
        return einval("pixel op too large for 32-bit item indexing");
    a.fd_cv = make_fastdiv((uint32_t)(a.C / v));
    a.fd_howo = make_fastdiv((uint32_t)(a.Ho * a.Ws));
    a.fd_wo = make_fastdiv((uint32_t)a.Ws);
    op->T = cdiv(a.items, 256);
    op->lds_bytes = 0;
    if (pix_kernels(d.dtype, kind, vec, op->kern) != 0) return einval("no kernel for this dtype");
    const double outs = (double)a.N * a.Ho * a.Wo * a.C;
    const double ins = kind == PIX_EW ? outs : (double)a.N * a.H * a.W * a.C;
    const bool dw = kind == PIX_DW || kind == PIX_DW3;
    op->flops = kind == PIX_EW ? 4.0 * outs : (dw ? 2.0 : 1.0) * outs * a.KH * a.KW;
    op->bytes = es * (ins + outs + (dw ? (double)a.KH * a.KW * a.C : 0.0) +
                      ((d.flags & MIRIAM_EPI_RESIDUAL) ? outs : 0.0));
    return MIRIAM_OK;
}

static int create_row(miriam_op *op) {
    const miriam_op_desc &d = op->d;
    RowArgs &a = op->rw;
    std::memset(&a, 0, sizeof(a));
    const int es = esize(d.dtype), V = vec_elems(d.dtype);
    if (d.m < 1 || d.nn < 1) return einval("row op: m, nn must be >= 1");
    a.rows = d.m; a.n = d.nn;
    a.ldx = d.ldx > 0 ? d.ldx : d.nn;
    a.ldy = d.ldy > 0 ? d.ldy : d.nn;
    if (a.ldx < d.nn || a.ldy < d.nn) return einval("row op: row stride too small");
    const int kind = d.kind == MIRIAM_OP_SOFTMAX ? ROW_SOFTMAX : ROW_LAYERNORM;
    if (kind == ROW_LAYERNORM) {
        if (!d.wt || !d.bias) return einval("layernorm: gamma (w) and beta (bias) required");
        if (!(d.eps >= 0.0f)) return einval("layernorm: negative eps");
        a.has_res = (d.flags & MIRIAM_EPI_RESIDUAL) ? 1 : 0;
        if (a.has_res && !d.residual) return einval("layernorm: residual flag without pointer");
        if (d.flags & ~MIRIAM_EPI_RESIDUAL) return einval("layernorm: only the residual flag applies");
    } else if (d.flags != 0) {
        return einval("softmax has no epilogue");
    }
    if (d.act != 0) return einval("row ops take no activation");
    a.x = d.x; a.res = d.residual; a.y = d.y;
    a.gamma = static_cast<const float *>(d.wt);
    a.beta = static_cast<const float *>(d.bias);
    a.scale = kind == ROW_SOFTMAX ? (d.scale == 0.0f ? 1.0f : d.scale) : 1.0f;
    a.eps = d.eps;
    const bool vec = (d.nn % V == 0) && (a.ldx % V == 0) && (a.ldy % V == 0) && aligned16(d.x) &&
                     aligned16(d.y) && (!a.has_res || aligned16(d.residual));
    op->T = cdiv(a.rows, 4);
    op->lds_bytes = 0;
    if (row_kernels(d.dtype, kind, vec, op->kern) != 0) return einval("no kernel for this dtype");
    const double n = (double)a.rows * a.n;
    op->flops = 5.0 * n;
    op->bytes = es * (n * 2.0 + (a.has_res ? n : 0.0)) + (kind == ROW_LAYERNORM ? 8.0 * a.n : 0.0);
    return MIRIAM_OK;
}

int op_launch(const miriam_op *op, int64_t b, int64_t l, int grid, int block, hipStream_t st,
              int32_t *owner_wg, int32_t *owner_iter, int32_t *count, int32_t *wave_phys, int32_t *wave_slot) {
    if (!op) return einval("null op");
    if (b < 0 || l < 1 || b + l > op->T || b + l < b) {
        set_error("shard outside the tile space");
        return MIRIAM_ERANGE;
    }
    if (grid < 1) {
        set_error("grid must be >= 1");
        return MIRIAM_ERANGE;
    }
    int pi;
    switch (block) {
    case 64: pi = 0; break;
    case 128: pi = 1; break;
    case 256: pi = 2; break;
    default: set_error("block must be 64, 128 or 256"); return MIRIAM_ERANGE;
    }
    Shard sh{b, l, owner_wg, owner_iter, count, wave_phys, wave_slot};
    void *args[2];
    switch (op->family) {
    case FAM_IGEMM:
    case FAM_SKINNY: args[0] = const_cast<IgemmArgs *>(&op->ig); break;
    case FAM_PIX: args[0] = const_cast<PixArgs *>(&op->px); break;
    default: args[0] = const_cast<RowArgs *>(&op->rw); break;
    }
    args[1] = &sh;
    hipError_t e = hipLaunchKernel(op->kern[pi], dim3(grid), dim3(block), args, 0, st);
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    return MIRIAM_OK;
}

int op_reset_counters(const miriam_op *op, hipStream_t st) {
    if (!op->counters || op->counters_bytes == 0) return MIRIAM_OK;
    hipError_t e = hipMemsetAsync(op->counters, 0, op->counters_bytes, st);
    return e == hipSuccess ? MIRIAM_OK : hip_fail(e, "hipMemsetAsync (split-K counters)");
}

int op_param_ranges(const miriam_op *op, const void *ptr[3], int64_t bytes[3]) {
    const miriam_op_desc &d = op->d;
    const int64_t es = esize(d.dtype);
    int n = 0;
    auto add = [&](const void *p, int64_t b) {
        if (p && b > 0 && n < 3) {
            ptr[n] = p;
            bytes[n] = b;
            ++n;
        }
    };
    int64_t ch = 0;  // channels of the per-channel epilogue vectors
    if (op->family == FAM_IGEMM || op->family == FAM_SKINNY) {
        const IgemmArgs &a = op->ig;
        const bool nmaj = d.kind == MIRIAM_OP_BGEMM && d.b_nmajor;
        if (d.kind != MIRIAM_OP_BGEMM || (a.sw0 == 0 && a.sw1 == 0))  // weights shared by the batch
            add(d.wt, es * (nmaj ? (a.K - 1) * a.ldw + a.Nc : (a.Nc - 1) * a.ldw + a.K));
        ch = a.Nc;
    } else if (op->family == FAM_PIX) {
        if (d.kind == MIRIAM_OP_DWCONV) add(d.wt, es * d.kh * d.kw * d.c);
        ch = d.c;
    } else if (d.kind == MIRIAM_OP_LAYERNORM) {
        add(d.wt, 4 * d.nn);
        add(d.bias, 4 * d.nn);
        return n;
    }
    if (d.flags & MIRIAM_EPI_BIAS) add(d.bias, 4 * ch);
    if (d.flags & MIRIAM_EPI_BN) add(d.bn, 16 * ch);
    return n;
}

}  // namespace miriam

using namespace miriam;

extern "C" {

const char *miriam_last_error(void) { return g_last_error.c_str(); }

int miriam_device_query(miriam_device_desc *out) {
    if (!out) return einval("null output");
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    hipDeviceProp_t p;
    e = hipGetDeviceProperties(&p, dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
    std::memset(out, 0, sizeof(*out));
    out->n_cu = p.multiProcessorCount;
    out->max_threads_per_cu = p.maxThreadsPerMultiProcessor;
    out->lds_per_cu = (int32_t)p.maxSharedMemoryPerMultiProcessor;
    out->n_xcd = kDies;
    out->wave_size = p.warpSize;
    out->clock_khz = p.clockRate;
    std::snprintf(out->arch, sizeof(out->arch), "%s", p.gcnArchName);
    return MIRIAM_OK;
}

static int op_create(const miriam_op_desc *d, miriam_op **out, bool noalloc) {
    if (!d || !out) return einval("null argument");
    *out = nullptr;
    if (d->dtype < MIRIAM_F32 || d->dtype > MIRIAM_BF16) return einval("unknown dtype");
    if (!d->x || !d->y) return einval("x and y are required");
    miriam_op *op = new (std::nothrow) miriam_op();
    if (!op) {
        set_error("out of host memory");
        return MIRIAM_ENOMEM;
    }
    op->d = *d;
    op->noalloc = noalloc;
    int rc;
    switch (d->kind) {
    case MIRIAM_OP_CONV2D:
    case MIRIAM_OP_GEMM:
    case MIRIAM_OP_BGEMM:
        if (!d->wt) { rc = einval("weights required"); break; }
        op->family = FAM_IGEMM;
        rc = create_igemm(op);
        break;
    case MIRIAM_OP_DWCONV:
        if (!d->wt) { rc = einval("weights required"); break; }
        op->family = FAM_PIX;
        rc = create_pix(op);
        break;
    case MIRIAM_OP_POOL_MAX:
    case MIRIAM_OP_POOL_AVG:
    case MIRIAM_OP_BN_ACT:
        op->family = FAM_PIX;
        rc = create_pix(op);
        break;
    case MIRIAM_OP_SOFTMAX:
    case MIRIAM_OP_LAYERNORM:
        op->family = FAM_ROW;
        rc = create_row(op);
        break;
    default:
        rc = einval("unknown op kind");
    }
    if (rc != MIRIAM_OK) {
        free_device(op);
        delete op;
        return rc;
    }
    query_occupancy(op);
    *out = op;
    return MIRIAM_OK;
}

int miriam_op_create(const miriam_op_desc *d, miriam_op **out) { return op_create(d, out, false); }

int miriam_op_create_noalloc(const miriam_op_desc *d, miriam_op **out) { return op_create(d, out, true); }

int miriam_op_query(const miriam_op *op, miriam_op_info *out) {
    if (!op || !out) return einval("null argument");
    std::memset(out, 0, sizeof(*out));
    out->num_tiles = op->T;
    out->logical_block = kLogicalBlock;
    out->lds_bytes = op->lds_bytes;
    const bool contraction = op->family == FAM_IGEMM || op->family == FAM_SKINNY;
    out->tile_m = contraction ? op->tile_m : 0;
    out->tile_n = contraction ? op->tile_n : 0;
    for (int i = 0; i < 3; ++i) out->max_wg_per_cu[i] = op->max_wg_per_cu[i];
    out->flops = op->flops;
    out->bytes = op->bytes;
    if (op->family == FAM_SKINNY) out->path = MIRIAM_PATH_SKINNY;
    else if (op->family == FAM_IGEMM)
        out->path = op->lay == LAY_RW        ? MIRIAM_PATH_RESIDENT
                    : op->lay == LAY_HALO    ? MIRIAM_PATH_HALO
                    : op->lay == LAY_VEC_UNI ? MIRIAM_PATH_DMA_UNIFORM
                    : op->lay == LAY_VEC     ? MIRIAM_PATH_DMA
                                             : MIRIAM_PATH_STAGED;
    else out->path = MIRIAM_PATH_OTHER;
    out->ksplit = (op->family == FAM_IGEMM || op->family == FAM_SKINNY) ? op->ig.ksplit : 1;
    out->full_grid = op_full_grid(op);
    return MIRIAM_OK;
}

int miriam_elastic_launch(const miriam_op *op, int64_t shard_begin, int64_t shard_len, int grid, int block,
                          void *stream) {
    return op_launch(op, shard_begin, shard_len, grid, block, static_cast<hipStream_t>(stream), nullptr,
                     nullptr, nullptr, nullptr, nullptr);
}

int miriam_elastic_launch_traced(const miriam_op *op, int64_t shard_begin, int64_t shard_len, int grid,
                                 int block, void *stream, int32_t *owner_wg, int32_t *owner_iter,
                                 int32_t *count, int32_t *wave_phys, int32_t *wave_slot) {
    if (!owner_wg || !owner_iter || !count) return einval("trace arrays required");
    if ((wave_phys == nullptr) != (wave_slot == nullptr)) return einval("wave_phys and wave_slot go together");
    return op_launch(op, shard_begin, shard_len, grid, block, static_cast<hipStream_t>(stream), owner_wg,
                     owner_iter, count, wave_phys, wave_slot);
}

int miriam_op_reset_counters(const miriam_op *op, void *stream) {
    if (!op) return einval("null op");
    return op_reset_counters(op, static_cast<hipStream_t>(stream));
}

int miriam_op_destroy(miriam_op *op) {
    if (!op) return einval("null op");
    if (op->pending.load() > 0) {
        set_error("op referenced by a pending request");
        return MIRIAM_EBUSY;
    }
    free_device(op);
    delete op;
    return MIRIAM_OK;
}

}  // extern "C"
