// Kernel argument blocks, passed by value to the elastic kernels.  Plain structs
// so the host runtime can fill them without device headers.
#pragma once

#include <stdint.h>

namespace miriam {

constexpr int kLogicalWaves = 4;   // logical block = 4 waves
constexpr int kLogicalBlock = 256;  // threads of the logical block
constexpr int kWave = 64;           // wavefront size of CDNA
constexpr int kDies = 8;            // XCDs of an MI355X; workgroups are dealt to them round-robin

// Division of n < 2^31 by a divisor d >= 1 fixed per operator, as a multiply-high, an add and
// a shift (unsigned division by invariant integers, Granlund and Montgomery 1994):
//   l = ceil(log2 d),  m = floor(2^32 (2^l - d) / d) + 1,  n / d = (mulhi(n, m) + n) >> l.
struct FastDiv {
    uint32_t m;
    uint32_t s;
};

inline FastDiv make_fastdiv(uint32_t d) {
    uint32_t l = 0;
    while (l < 32 && (1ull << l) < (uint64_t)d) ++l;
    FastDiv f;
    f.m = (uint32_t)((((1ull << l) - (uint64_t)d) << 32) / (uint64_t)d + 1ull);
    f.s = l;
    return f;
}

// Host evaluation of the same formula (used to check the constants).
inline uint32_t fastdiv_host(uint32_t n, FastDiv f) {
    const uint32_t hi = (uint32_t)(((uint64_t)n * (uint64_t)f.m) >> 32);
    return (uint32_t)(((uint64_t)hi + (uint64_t)n) >> f.s);
}

// Shard description passed to every kernel.  The trace arrays are null except
// in traced launches, where they record the tile -> (workgroup, iteration) map and,
// when wave_phys is set, the logical wave -> (physical wave, slot) map of every tile:
// entry 4 t + lambda of wave_phys / wave_slot is written by the physical wave that ran
// logical wave lambda of tile t (slot = its place among the logical waves that wave runs).
struct Shard {
    int64_t begin;
    int64_t len;
    int32_t *owner_wg;
    int32_t *owner_iter;
    int32_t *count;
    int32_t *wave_phys;
    int32_t *wave_slot;
};

// Fused epilogue: v = act(BN(acc + bias[c]) + residual).
struct Epilogue {
    const float *bias;   // [C]
    const float *bn;     // [4*C]: gamma, beta, mean, var
    float eps;
    int act;
    int flags;
    int64_t C;           // channels (bn stride)
};

// Contraction (convolution / GEMM / batched GEMM).
struct IgemmArgs {
    const void *x;
    const void *w;
    void *y;
    const void *res;
    int64_t H, W, C, ldx;  // input image and its pixel (row) stride in elements
    int64_t Ho, Wo;        // output image
    int32_t KH, KW, stride, pad;
    int64_t M, Nc, K;      // GEMM sizes per batch entry
    int64_t ldw, ldy;      // B row stride, output row stride
    int64_t mT, nT;        // tiles along m and n
    int64_t bdiv, sx0, sx1, sw0, sw1, sy0, sy1;  // batch offsets
    int64_t img_x;         // elements between images of x
    int64_t tY, tX;        // direct 3x3 kernel: tile rows and tile columns per output image
    FastDiv fd_howo, fd_wo; // division by Ho * Wo and by Wo (output pixel -> image, row, column)
    int32_t vec_store;     // 1: output / residual rows allow 16-byte vector access
    int32_t ksplit;        // K slices per output tile (1 = none); tile id = output tile * ksplit + slice
    int32_t cps;           // K chunks per slice
    float *work;           // ksplit fp32 partial tiles per output tile (ksplit > 1)
    int32_t *counters;     // arrivals per output tile; back to 0 once a pass over the op completes
    // memory-based index function: per output row m < mT * TM, (image, p * stride - pad,
    // q * stride - pad, m < M) as 4 int32; null = computed in the kernel
    const int32_t *rowtab;
    // bytes addressable from one batch entry's x / w base (chunk-uniform decode only: the
    // operands are read as buffers of this size, below 2^31 bytes)
    uint32_t x_bytes, w_bytes;
    uint32_t y_bytes;  // resident-weight kernel: output span in bytes when below 2^31 and 16-byte stores apply, else 0
    Epilogue epi;
};

// Channel-vector kernels (depthwise, pooling, standalone epilogue).
struct PixArgs {
    const void *x;
    const void *w;     // depthwise weights [KH][KW][C]
    void *y;
    const void *res;   // same layout as y
    int64_t N, H, W, C, Ho, Wo;
    int32_t KH, KW, stride, pad;
    int64_t items;     // lane items: N*Ho*Wo*(C/V); PIX_DW3: N*Ho*Ws*(C/V)
    int64_t Ws;        // PIX_DW3: strips of kDwStrip output pixels per output row
    FastDiv fd_cv, fd_howo, fd_wo;  // division by C/V, Ho*Wo and Wo (PIX_DW3: Ho*Ws and Ws)
    Epilogue epi;
};

// Row kernels (softmax, layer normalisation).
struct RowArgs {
    const void *x;
    const void *res;    // LAYERNORM residual (added before normalising)
    const float *gamma; // LAYERNORM
    const float *beta;
    void *y;
    int64_t rows, n, ldx, ldy;
    float scale;        // SOFTMAX
    float eps;          // LAYERNORM
    int has_res;
};

enum PixKind { PIX_DW = 0, PIX_MAX = 1, PIX_AVG = 2, PIX_EW = 3, PIX_DW3 = 4 };
constexpr int kDwStrip = 4;  // PIX_DW3: output pixels along a row per lane item
enum RowKind { ROW_SOFTMAX = 0, ROW_LAYERNORM = 1 };
enum IgemmLayout { LAY_VEC = 0, LAY_SCALAR = 1, LAY_VEC_NB = 2, LAY_SCALAR_NB = 3, LAY_VEC_UNI = 4, LAY_HALO = 5, LAY_RW = 6 };
enum IgemmCfg { CFG_32 = 1, CFG_64 = 2, CFG_128 = 3, CFG_128x64 = 4, CFG_256x128 = 6, CFG_HALO = 7, CFG_RW = 8 };

}  // namespace miriam
