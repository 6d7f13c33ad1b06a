// Kernel tables of the bandwidth-bound elastic kernels (depthwise convolution,
// pooling, standalone epilogue, softmax, layer normalisation).
#include "memops.h"

namespace miriam {

template <class T, int V, int KIND>
static void pix_table(const void *out[3]) {
    out[0] = reinterpret_cast<const void *>(&pix_kernel<T, V, KIND, 1>);
    out[1] = reinterpret_cast<const void *>(&pix_kernel<T, V, KIND, 2>);
    out[2] = reinterpret_cast<const void *>(&pix_kernel<T, V, KIND, 4>);
}

template <class T, int KIND>
static void pix_table_v(bool vec, const void *out[3]) {
    if (vec) pix_table<T, 16 / sizeof(T), KIND>(out);
    else pix_table<T, 1, KIND>(out);
}

template <class T>
static int pix_table_k(int kind, bool vec, const void *out[3]) {
    switch (kind) {
    case PIX_DW: pix_table_v<T, PIX_DW>(vec, out); return 0;
    case PIX_MAX: pix_table_v<T, PIX_MAX>(vec, out); return 0;
    case PIX_AVG: pix_table_v<T, PIX_AVG>(vec, out); return 0;
    case PIX_EW: pix_table_v<T, PIX_EW>(vec, out); return 0;
    case PIX_DW3:
        // 16-bit types only
        if constexpr (sizeof(T) != 2) {
            return -1;
        } else {
            if (!vec) return -1;
            pix_table<T, 16 / sizeof(T), PIX_DW3>(out);
            return 0;
        }
    default: return -1;
    }
}

int pix_kernels(int dtype, int kind, bool vec, const void *out[3]) {
    switch (dtype) {
    case 0: return pix_table_k<float>(kind, vec, out);
    case 1: return pix_table_k<half_t>(kind, vec, out);
    case 2: return pix_table_k<bf16_t>(kind, vec, out);
    default: return -1;
    }
}

template <class T, int V, int KIND>
static void row_table(const void *out[3]) {
    out[0] = reinterpret_cast<const void *>(&row_kernel<T, V, KIND, 1>);
    out[1] = reinterpret_cast<const void *>(&row_kernel<T, V, KIND, 2>);
    out[2] = reinterpret_cast<const void *>(&row_kernel<T, V, KIND, 4>);
}

template <class T>
static int row_table_k(int kind, bool vec, const void *out[3]) {
    constexpr int V = 16 / sizeof(T);
    switch (kind * 2 + (vec ? 1 : 0)) {
    case 0: row_table<T, 1, ROW_SOFTMAX>(out); return 0;
    case 1: row_table<T, V, ROW_SOFTMAX>(out); return 0;
    case 2: row_table<T, 1, ROW_LAYERNORM>(out); return 0;
    case 3: row_table<T, V, ROW_LAYERNORM>(out); return 0;
    default: return -1;
    }
}

int row_kernels(int dtype, int kind, bool vec, const void *out[3]) {
    switch (dtype) {
    case 0: return row_table_k<float>(kind, vec, out);
    case 1: return row_table_k<half_t>(kind, vec, out);
    case 2: return row_table_k<bf16_t>(kind, vec, out);
    default: return -1;
    }
}

}  // namespace miriam
