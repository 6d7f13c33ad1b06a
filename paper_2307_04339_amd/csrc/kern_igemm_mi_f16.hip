// Kernel table of the pipelined contraction kernel with the memory-based index function
// (output-row indices from a host-computed table) for f16 operands; a translation unit of its
// own so the build stays parallel.
#include "igemm_dma.h"

namespace miriam {
int igemm_mi_kernels_f16(int cfg, bool uni, const void *out[3], int *lds) {
    return igemm_dma_mi_table_cfg<half_t>(cfg, uni, out, lds);
}
}  // namespace miriam
