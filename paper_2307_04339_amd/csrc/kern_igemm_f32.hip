// Kernel table of the elastic contraction kernel for f32 operands (one translation unit
// per element type keeps the build parallel).
#include "conv_halo.h"

namespace miriam {
int igemm_kernels_f32(int cfg, int lay, const void *out[3], int *lds) {
    switch (lay) {
    case LAY_VEC: return igemm_dma_table_cfg<float, false>(cfg, out, lds);
    case LAY_VEC_UNI: return igemm_dma_table_cfg<float, true>(cfg, out, lds);
    case LAY_HALO: return halo_table<float>(out, lds);
    case LAY_SCALAR: return igemm_table_cfg<float, LAY_SCALAR>(cfg, out, lds);
    default: return -1;
    }
}
}  // namespace miriam
