// Host-side internals shared by the library's C++ translation units.
#pragma once

#include <atomic>
#include <cstdint>
#include <string>

#include <hip/hip_runtime_api.h>

#include "../../include/miriam.h"
#include "kargs.h"

namespace miriam {

void set_error(const std::string &msg);
int hip_fail(hipError_t e, const char *what);  // records the HIP error text, returns MIRIAM_EHIP

enum Family { FAM_IGEMM = 0, FAM_PIX = 1, FAM_ROW = 2, FAM_SKINNY = 3 };

// Kernel tables (one entry per physical block of 64, 128, 256 threads).
int igemm_kernels_f32(int cfg, int lay, const void *out[3], int *lds);
int igemm_kernels_f16(int cfg, int lay, const void *out[3], int *lds);
int igemm_kernels_bf16(int cfg, int lay, const void *out[3], int *lds);
// pipelined kernel with the memory-based index function (tiles 1..4); uni: chunk-uniform decode
int igemm_mi_kernels_f32(int cfg, bool uni, const void *out[3], int *lds);
int igemm_mi_kernels_f16(int cfg, bool uni, const void *out[3], int *lds);
int igemm_mi_kernels_bf16(int cfg, bool uni, const void *out[3], int *lds);
int pix_kernels(int dtype, int kind, bool vec, const void *out[3]);
int row_kernels(int dtype, int kind, bool vec, const void *out[3]);
int skinny_kernels(int dtype, int cg, const void *out[3]);  // cg: 16-column groups per tile (1 or 2)
int skinny_group(int cg);                                   // K per wave group of that kernel
// resident-weight direct convolution: (3x3, stride 1, C in {8,16,32,64}), (3x3, stride 2, C = 8),
// (1x1, stride 1, C in {16,24,32,64})
int rw_kernels(int dtype, int64_t ks, int64_t stride, int64_t c, const void *out[3], int *lds);

}  // namespace miriam

struct miriam_op {
    miriam_op_desc d;
    int family;
    int64_t T;              // logical tiles
    int cfg, lay;           // contraction tile config and load layout
    int tile_m, tile_n;
    int lds_bytes;
    const void *kern[3];    // kernels for physical blocks 64, 128, 256
    int max_wg_per_cu[3];
    int64_t full_grid;      // grid of a whole-tile-space launch (T, or the resident capacity)
    double flops, bytes;
    miriam::IgemmArgs ig;
    miriam::PixArgs px;
    miriam::RowArgs rw;
    std::atomic<int> pending{0};  // submitted requests that still reference the op
    void *work = nullptr;         // split-K partial tiles (device memory owned by the op)
    void *counters = nullptr;     // split-K arrival counters (device memory owned by the op)
    size_t counters_bytes = 0;
    bool noalloc = false;         // created by miriam_op_create_noalloc: workspace in the device scratch
    void *rowtab = nullptr;       // memory-based index table (device memory owned by the op)
};

namespace miriam {
// Grid of the op's whole-tile-space (unsharded) launch.
inline int op_full_grid(const miriam_op *op) {
    return (int)(op->full_grid < INT32_MAX ? op->full_grid : INT32_MAX);
}

// Launch helper used by the public entry points and by the coordinator.
int op_launch(const miriam_op *op, int64_t b, int64_t l, int grid, int block, hipStream_t st,
              int32_t *owner_wg = nullptr, int32_t *owner_iter = nullptr, int32_t *count = nullptr,
              int32_t *wave_phys = nullptr, int32_t *wave_slot = nullptr);

// Clear the op's split-K arrival counters on `st` (stream-ordered); MIRIAM_OK without split K.
int op_reset_counters(const miriam_op *op, hipStream_t st);

// Read-only parameter ranges of an op (weights, bias, batch-norm and layer-norm vectors)
// that every request reads again: up to 3 (pointer, bytes) pairs; returns the count.
// Operands that change per request (activations, batched right operands) are not listed.
int op_param_ranges(const miriam_op *op, const void *ptr[3], int64_t bytes[3]);

// One range of whole 64-byte lines for the cache-warming kernel.
struct WarmRange {
    const char *line0;  // first line (address rounded down to 64 bytes)
    int64_t lines;      // lines to touch
};

// Touch one word of every line of the `n` ranges of the device table `table` (grid x 256
// threads) on stream `st`; `sink` is a device word the kernel may write (never read back).
int warm_launch(const WarmRange *table, int n, int grid, int *sink, hipStream_t st);

// An empty one-wave kernel on `st` (launch-gap measurement).
int noop_launch(hipStream_t st);

// One-wave kernel on `st` that returns once *flag (coherent host memory, device address)
// reaches `seq` or `limit_ticks` ticks of the device wall clock have passed.
int gate_launch(const uint64_t *flag, uint64_t seq, uint64_t limit_ticks, hipStream_t st);
}  // namespace miriam
