// Load-path microbenchmark for the contraction kernels' operand stream on gfx950.
//
// Part 1, raw rates: every wave of a 4-wave workgroup streams 1 KB per instruction
// (global_load_lds_dwordx4 into LDS, or global_load_dwordx4 into registers) from an L2-resident
// 64 KB block or from a large buffer; bytes per clock per CU at one and two workgroups per CU.
// Part 2, the pipelined implicit GEMM's operand stream without arithmetic: per 128 x 128 tile
// and 64-element K chunk, 128 input rows of 128 B (pixel stride 256 B, the nine 3x3 tap
// shifts: VGG-16 b8 conv2_2) and 128 weight rows of 128 B (row stride 2304 B), by LDS DMA into
// a 3-stage A ring and a 2-stage B ring, with the kernel's vmcnt wait and barrier per chunk or
// free-running; the same byte count from contiguous 1 KB blocks for comparison.
// Part 3, streaming reads of a 3 GiB buffer (the practical HBM read rate).  Part 4, a small-batch
// FC layer's weight stream in the skinny kernel's load pattern and row-contiguous.  Part 5, the
// MFMA peak from registers (fp16, bf16, fp32).
//
// Every address is inside its buffer by construction (see the bounds noted at each index).
// Build and run:  hipcc --offload-arch=gfx950 -O3 -o /tmp/loadpath tests/perf/loadpath_bench.hip && /tmp/loadpath
#include <hip/hip_runtime.h>
#include <cstdint>
#include <cstdio>

#define CHECK(x)                                                                         \
    do {                                                                                 \
        hipError_t e_ = (x);                                                             \
        if (e_ != hipSuccess) {                                                          \
            printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);        \
            return 1;                                                                    \
        }                                                                                \
    } while (0)

__device__ __forceinline__ void dma16(const void *g, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds) : "memory", "m0");
}
template <int N>
__device__ __forceinline__ void wait_vm() {
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
__device__ __forceinline__ uint32_t lds_addr(char *p) {
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)p;
}

// ---- part 1: raw rates.  Wave w of the workgroup, instruction j of iteration i reads the 1 KB
// block ((i * 8 + j) * 4 + w) masked to the span (a power of two >= 64 KB), offset by 64 KB per
// workgroup when per_wg; LDS target: 8 KB per wave (32 KB per workgroup).
template <bool DMA>
__global__ __launch_bounds__(256) void raw_kernel(const char *src, uint64_t span_mask, int iters, int per_wg, int *sink) {
    __shared__ __attribute__((aligned(1024))) char lds[32768];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64), lane = threadIdx.x % 64;
    const uint32_t base = lds_addr(lds);
    const uint64_t off = per_wg ? (uint64_t)blockIdx.x * 65536 : 0;
    uint32_t acc = 0;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint64_t o = (off + (uint64_t)((i * 8 + j) * 4 + wave) * 1024) & span_mask;  // o + 1 KB <= span
            const char *p = src + o + lane * 16;
            if constexpr (DMA) {
                dma16(p, base + wave * 8192 + j * 1024);
            } else {
                const uint4 v = *reinterpret_cast<const uint4 *>(p);
                acc ^= v.x ^ v.y ^ v.z ^ v.w;
            }
        }
        if constexpr (DMA) wait_vm<8>();  // one batch of 8 instructions in flight behind the newest
    }
    wait_vm<0>();
    __syncthreads();
    if constexpr (DMA) acc ^= *reinterpret_cast<const uint32_t *>(lds + threadIdx.x * 4);
    if (acc == 0x12345678u) sink[0] = (int)acc;
}

// ---- part 2: the operand stream of a 128 x 128 implicit-GEMM tile
constexpr int kPix = 8 * 112 * 112;  // input pixels, 256 B each
constexpr int kK = 1152;             // weight row length (elements): 2304 B rows, 128 rows

// PAT 0: the convolution's rows; 1: contiguous 1 KB per instruction
template <int PAT, bool BAR>
__global__ __launch_bounds__(256) void conv_kernel(const char *X, const char *W, int tiles, int *sink) {
    __shared__ __attribute__((aligned(1024))) char lds[81920];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64), lane = threadIdx.x % 64;
    const int lrow = lane >> 3, slot = lane & 7;
    const uint32_t base = lds_addr(lds);
    for (int t = blockIdx.x; t < tiles; t += gridDim.x) {
        const int m0 = (t * 128) % (kPix - 128 - 2 * 112 - 2);  // m0 + 127 + 226 < kPix
        for (int c = 0; c < 18; ++c) {
            const int tap = c >> 1, half = c & 1;
            const int shift = (tap / 3) * 112 + (tap % 3);  // <= 226
            const uint32_t sa = base + (c % 3) * 16384, sb = base + 49152 + (c % 2) * 16384;  // < 80 KB
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int row = 8 * (j * 4 + wave) + lrow;  // < 128
                const char *pb = PAT == 0 ? W + (int64_t)row * (kK * 2) + c * 128 + slot * 16  // <= 294912 B
                                          : W + (int64_t)((c * 16 + j * 4 + wave) % 256) * 1024 + lane * 16;  // < 256 KB
                dma16(pb, sb + (8 * (j * 4 + wave)) * 128);
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int row = 8 * (j * 4 + wave) + lrow;
                const char *pa = PAT == 0 ? X + (int64_t)(m0 + row + shift) * 256 + half * 128 + slot * 16
                                          : X + (int64_t)(m0 * 2 + (c * 16 + j * 4 + wave) * 64) * 16 + lane * 16;
                dma16(pa, sa + (8 * (j * 4 + wave)) * 128);
            }
            if (BAR) {
                wait_vm<4>();
                __syncthreads();
            } else {
                wait_vm<16>();
            }
        }
    }
    wait_vm<0>();
    __syncthreads();
    if (lds[threadIdx.x] == 123 && lds[threadIdx.x + 1] == 45) sink[0] = 1;
}

// ---- part 3: streaming reads from HBM.  Workgroup g reads the contiguous region
// [g * per_wg, (g + 1) * per_wg) of a buffer larger than every cache, 16 B per lane per load,
// U loads in flight per lane; per_wg is a multiple of 256 * 16 * U bytes.
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
template <int U>
__global__ __launch_bounds__(256) void stream_kernel(const u32x4 *src, long long per_wg_vec, int *sink) {
    const u32x4 *p = src + (long long)blockIdx.x * per_wg_vec + threadIdx.x;
    uint32_t acc = 0;
    for (long long i = 0; i < per_wg_vec; i += 256 * U) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(p + i + u * 256);
#pragma unroll
        for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    if (acc == 0x12345678u) sink[0] = (int)acc;
}

// ---- part 4: the weight stream of a small-batch FC layer (VGG-16 fc6: 4096 rows of 25088
// fp16 values, 50176 B apart).  1024 workgroups of 4 waves; workgroup g covers rows
// 16 (g % 256) .. +15 and K slice g / 256 (of 4), wave w the slice's quarter w (1568 values).
// ROWPAT 1 (the skinny kernel's MFMA-operand pattern): a load instruction reads 64 B of each of
// the 16 rows (lane l: row l % 16, 16 B at 8 (l / 16) values into a 32-value step), 4 steps per
// group, one group loaded and consumed at a time.  ROWPAT 0: an instruction reads 1 KB of one
// row (512 values), cycling over the 16 rows, 16 instructions in flight.  Offsets stay inside
// the buffer: the last 1 KB instruction of a quarter may run past it into the next quarter of
// the same row, and the last quarter of a row stops at the row's end (clamped).
constexpr long long kFcRow = 25088, kFcQ = 1568;
template <int ROWPAT>
__global__ __launch_bounds__(256) void fc_stream_kernel(const unsigned short *W, int *sink) {
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    const long long n0 = (long long)(blockIdx.x % 256) * 16, slice = blockIdx.x / 256;
    const long long kb = slice * (kFcRow / 4) + wave * kFcQ;
    uint32_t acc = 0;
    if constexpr (ROWPAT == 1) {
        const int row = lane % 16, grp = lane / 16;
        const unsigned short *wr = W + (n0 + row) * kFcRow;
        for (long long k0 = kb; k0 < kb + kFcQ; k0 += 128) {
            u32x4 v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const long long k = k0 + j * 32 + grp * 8;  // k + 8 <= kb + kFcQ + 96 <= kFcRow
                v[j] = k + 8 <= kFcRow ? *reinterpret_cast<const u32x4 *>(wr + k) : u32x4{0, 0, 0, 0};
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) acc ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
        }
    } else {
        for (long long c = 0; c < kFcQ; c += 512) {
            u32x4 v[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                long long k = kb + c + lane * 8;
                if (k + 8 > kFcRow) k = kFcRow - 8;
                v[r] = *reinterpret_cast<const u32x4 *>(W + (n0 + r) * kFcRow + k);
            }
#pragma unroll
            for (int r = 0; r < 16; ++r) acc ^= v[r].x ^ v[r].y ^ v[r].z ^ v[r].w;
        }
    }
    if (acc == 0x12345678u) sink[0] = (int)acc;
}

// ---- part 5: the MFMA peak from registers: each wave runs 8 independent accumulator chains of
// v_mfma_f32_32x32x16_{f16,bf16} (32768 FLOP each) or v_mfma_f32_32x32x2f32 (4096 FLOP), no memory.
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
template <int KIND>
__global__ __launch_bounds__(256) void mfma_kernel(int iters, float *sink) {
    f32x16_t acc[8];
#pragma unroll
    for (int c = 0; c < 8; ++c)
        for (int e = 0; e < 16; ++e) acc[c][e] = 0.0f;
    const float x = (float)(threadIdx.x & 7) * 0.001f;
    f16x8_t a16, b16;
    bf16x8_t a16b, b16b;
    for (int e = 0; e < 8; ++e) {
        a16[e] = (_Float16)x;
        b16[e] = (_Float16)(x + 0.5f);
        a16b[e] = (__bf16)x;
        b16b[e] = (__bf16)(x + 0.5f);
    }
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            if constexpr (KIND == 0) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a16, b16, acc[c], 0, 0, 0);
            else if constexpr (KIND == 1) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a16b, b16b, acc[c], 0, 0, 0);
            else acc[c] = __builtin_amdgcn_mfma_f32_32x32x2f32(x, x + 0.5f, acc[c], 0, 0, 0);
        }
    }
    float s = 0.0f;
#pragma unroll
    for (int c = 0; c < 8; ++c) s += acc[c][0] + acc[c][15];
    if (s == 1234.5f) sink[0] = s;
}

static int cus = 0;

template <class F>
static int best_ms(F launch, float *out) {
    hipEvent_t a, b;
    CHECK(hipEventCreate(&a));
    CHECK(hipEventCreate(&b));
    launch();
    CHECK(hipDeviceSynchronize());
    float best = 1e30f;
    for (int r = 0; r < 5; ++r) {
        CHECK(hipEventRecord(a));
        launch();
        CHECK(hipEventRecord(b));
        CHECK(hipEventSynchronize(b));
        float ms = 0;
        CHECK(hipEventElapsedTime(&ms, a, b));
        if (ms < best) best = ms;
    }
    CHECK(hipEventDestroy(a));
    CHECK(hipEventDestroy(b));
    *out = best;
    return 0;
}

// Median over 9 launches of one launch's event time, each launch preceded by `evict` (events
// bracket the timed launch only).
template <class F, class E>
static int cold_ms(F launch, E evict, float *out) {
    hipEvent_t a, b;
    CHECK(hipEventCreate(&a));
    CHECK(hipEventCreate(&b));
    float t[9];
    for (int r = 0; r < 9; ++r) {
        evict();
        CHECK(hipEventRecord(a));
        launch();
        CHECK(hipEventRecord(b));
        CHECK(hipEventSynchronize(b));
        CHECK(hipEventElapsedTime(&t[r], a, b));
    }
    for (int i = 1; i < 9; ++i)
        for (int j = i; j > 0 && t[j] < t[j - 1]; --j) {
            const float x = t[j];
            t[j] = t[j - 1];
            t[j - 1] = x;
        }
    CHECK(hipEventDestroy(a));
    CHECK(hipEventDestroy(b));
    *out = t[4];
    return 0;
}

static void report(const char *name, int grid, double bytes, float ms) {
    printf("%-44s grid %5d  %9.1f us  %8.1f GB/s  %5.1f B/clk/CU\n", name, grid, ms * 1e3, bytes / (ms * 1e-3) / 1e9,
           bytes / (ms * 1e-3) / 2.4e9 / cus);
}

int main() {
    CHECK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0));
    const uint64_t big = 1ull << 30;
    char *src, *X, *W;
    int *sink;
    CHECK(hipMalloc(&src, big));
    CHECK(hipMemset(src, 1, big));
    CHECK(hipMalloc(&X, (size_t)kPix * 256));
    CHECK(hipMemset(X, 1, (size_t)kPix * 256));
    CHECK(hipMalloc(&W, (size_t)1 << 20));
    CHECK(hipMemset(W, 1, (size_t)1 << 20));
    CHECK(hipMalloc(&sink, 64));
    printf("CUs %d; rates at 2.4 GHz\n", cus);
    float ms;
    for (int k = 1; k <= 2; ++k) {
        const int grid = cus * k, it = 2000;
        printf("-- part 1: %d workgroup(s) of 4 waves per CU\n", k);
        const double b_hot = (double)grid * 256 * 16 * 8 * it, b_big = b_hot / 4;
        if (best_ms([&] { hipLaunchKernelGGL(raw_kernel<true>, dim3(grid), dim3(256), 0, 0, src, 65535ull, it, 0, sink); }, &ms)) return 1;
        report("LDS DMA, L2-resident 64 KB", grid, b_hot, ms);
        if (best_ms([&] { hipLaunchKernelGGL(raw_kernel<false>, dim3(grid), dim3(256), 0, 0, src, 65535ull, it, 0, sink); }, &ms)) return 1;
        report("load to VGPR, L2-resident 64 KB", grid, b_hot, ms);
        if (best_ms([&] { hipLaunchKernelGGL(raw_kernel<true>, dim3(grid), dim3(256), 0, 0, src, big - 1, it / 4, 1, sink); }, &ms)) return 1;
        report("LDS DMA, 16 MB per workgroup of 1 GB", grid, b_big, ms);
        if (best_ms([&] { hipLaunchKernelGGL(raw_kernel<false>, dim3(grid), dim3(256), 0, 0, src, big - 1, it / 4, 1, sink); }, &ms)) return 1;
        report("load to VGPR, 16 MB per workgroup of 1 GB", grid, b_big, ms);
    }
    for (int k = 1; k <= 2; ++k) {
        const int grid = cus * k;
        printf("-- part 2: %d workgroup(s) per CU, 128x128 tiles of 18 K chunks (32 KB each)\n", k);
        for (int tiles : {grid, 784}) {
            const double bytes = (double)tiles * 18 * 32768;
            char name[64];
            snprintf(name, sizeof(name), "conv rows, barrier per chunk, %d tiles", tiles);
            if (best_ms([&] { hipLaunchKernelGGL((conv_kernel<0, true>), dim3(grid), dim3(256), 0, 0, X, W, tiles, sink); }, &ms)) return 1;
            report(name, grid, bytes, ms);
            snprintf(name, sizeof(name), "conv rows, free running, %d tiles", tiles);
            if (best_ms([&] { hipLaunchKernelGGL((conv_kernel<0, false>), dim3(grid), dim3(256), 0, 0, X, W, tiles, sink); }, &ms)) return 1;
            report(name, grid, bytes, ms);
            snprintf(name, sizeof(name), "contiguous 1 KB, barrier per chunk, %d tiles", tiles);
            if (best_ms([&] { hipLaunchKernelGGL((conv_kernel<1, true>), dim3(grid), dim3(256), 0, 0, X, W, tiles, sink); }, &ms)) return 1;
            report(name, grid, bytes, ms);
        }
    }
    {
        const size_t bytes = (size_t)3 << 30;  // 3 GiB: beyond the L2s and the 256 MB Infinity Cache
        char *big3;
        CHECK(hipMalloc(&big3, bytes));
        CHECK(hipMemset(big3, 1, bytes));
        printf("-- part 3: streaming reads of 3 GiB (nontemporal 16-byte loads)\n");
        for (int k : {1, 2, 4, 8}) {
            const int grid = cus * k;
            const long long per_vec = (long long)(bytes / 16 / grid) / (256 * 8) * (256 * 8);
            const double rb = (double)per_vec * 16 * grid;
            if (best_ms([&] { hipLaunchKernelGGL(stream_kernel<8>, dim3(grid), dim3(256), 0, 0,
                                                 reinterpret_cast<const u32x4 *>(big3), per_vec, sink); }, &ms)) return 1;
            char name[64];
            snprintf(name, sizeof(name), "stream, %d workgroups per CU, 8 loads in flight", k);
            printf("%-44s grid %5d  %9.1f us  %8.1f GB/s\n", name, grid, ms * 1e3, rb / (ms * 1e-3) / 1e9);
        }
        CHECK(hipFree(big3));
    }
    {
        const size_t wbytes = (size_t)4096 * kFcRow * 2;
        unsigned short *Wf;
        CHECK(hipMalloc(&Wf, wbytes));
        CHECK(hipMemset(Wf, 1, wbytes));
        // cold: a 512 MiB read between the timed launches evicts the L2s and the 256 MB
        // Infinity Cache (back to back, most of the 205 MB stays in the Infinity Cache)
        const size_t ebytes = (size_t)512 << 20;
        char *ev;
        CHECK(hipMalloc(&ev, ebytes));
        CHECK(hipMemset(ev, 1, ebytes));
        const int egrid = cus * 4;
        const long long evec = (long long)(ebytes / 16 / egrid) / (256 * 8) * (256 * 8);
        auto evict = [&] { hipLaunchKernelGGL(stream_kernel<8>, dim3(egrid), dim3(256), 0, 0, reinterpret_cast<const u32x4 *>(ev), evec, sink); };
        const long long wvec = (long long)(wbytes / 16 / 1024) / (256 * 8) * (256 * 8);  // contiguous: 1024 x 192 KB
        const double wst = (double)wvec * 16 * 1024;
        printf("-- part 4: VGG-16 fc6 weight stream (205 MB), 1024 workgroups (warm: back to back; cold: after a 512 MiB read)\n");
        for (int cold = 0; cold < 2; ++cold) {
            auto timed = [&](auto launch, float *out) { return cold ? cold_ms(launch, evict, out) : best_ms(launch, out); };
            if (timed([&] { hipLaunchKernelGGL(fc_stream_kernel<1>, dim3(1024), dim3(256), 0, 0, Wf, sink); }, &ms)) return 1;
            printf("%-5s %-44s  %9.1f us  %8.1f GB/s\n", cold ? "cold" : "warm", "16 rows x 64 B per instruction", ms * 1e3,
                   wbytes / (ms * 1e-3) / 1e9);
            if (timed([&] { hipLaunchKernelGGL(fc_stream_kernel<0>, dim3(1024), dim3(256), 0, 0, Wf, sink); }, &ms)) return 1;
            printf("%-5s %-44s  %9.1f us  %8.1f GB/s\n", cold ? "cold" : "warm", "1 row x 1 KB per instruction", ms * 1e3,
                   wbytes / (ms * 1e-3) / 1e9);
            if (timed([&] { hipLaunchKernelGGL(stream_kernel<8>, dim3(1024), dim3(256), 0, 0, reinterpret_cast<const u32x4 *>(Wf), wvec, sink); }, &ms)) return 1;
            printf("%-5s %-44s  %9.1f us  %8.1f GB/s\n", cold ? "cold" : "warm", "contiguous stream of 201 MB of the buffer", ms * 1e3,
                   wst / (ms * 1e-3) / 1e9);
        }
        CHECK(hipFree(ev));
        CHECK(hipFree(Wf));
    }
    {
        float *fs;
        CHECK(hipMalloc(&fs, 64));
        printf("-- part 5: MFMA from registers, 8 chains per wave, 2 workgroups of 4 waves per CU\n");
        const int grid = cus * 2, it = 4000;
        const char *names[3] = {"v_mfma_f32_32x32x16_f16", "v_mfma_f32_32x32x16_bf16", "v_mfma_f32_32x32x2f32"};
        const double flop_per[3] = {32768.0, 32768.0, 4096.0};
        const double peak[3] = {2500.0, 2500.0, 157.3};
        for (int kind = 0; kind < 3; ++kind) {
            int rc = 0;
            if (kind == 0) rc = best_ms([&] { hipLaunchKernelGGL(mfma_kernel<0>, dim3(grid), dim3(256), 0, 0, it, fs); }, &ms);
            if (kind == 1) rc = best_ms([&] { hipLaunchKernelGGL(mfma_kernel<1>, dim3(grid), dim3(256), 0, 0, it, fs); }, &ms);
            if (kind == 2) rc = best_ms([&] { hipLaunchKernelGGL(mfma_kernel<2>, dim3(grid), dim3(256), 0, 0, it, fs); }, &ms);
            if (rc) return 1;
            const double tf = (double)grid * 4 * it * 8 * flop_per[kind] / (ms * 1e-3) / 1e12;
            printf("%-44s  %9.1f us  %8.1f TFLOP/s  %5.1f %% of %.1f\n", names[kind], ms * 1e3, tf, 100.0 * tf / peak[kind],
                   peak[kind]);
        }
        CHECK(hipFree(fs));
    }
    return 0;
}
