// Kernel tables of the resident-weight direct convolution (fp16 and bf16).
#include "conv_rw.h"

namespace miriam {
int rw_kernels(int dtype, int64_t ks, int64_t stride, int64_t c, const void *out[3], int *lds) {
    // dtype codes follow miriam_dtype: 1 = fp16, 2 = bf16
    if (dtype == 1) return rw_table_c<half_t>(ks, stride, c, out, lds);
    if (dtype == 2) return rw_table_c<bf16_t>(ks, stride, c, out, lds);
    return -1;
}
}  // namespace miriam
