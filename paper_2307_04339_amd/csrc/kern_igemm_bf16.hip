// Kernel table of the elastic contraction kernel for bf16 operands (one translation unit
// per element type keeps the build parallel).
#include "conv_halo.h"

namespace miriam {
int igemm_kernels_bf16(int cfg, int lay, const void *out[3], int *lds) {
    switch (lay) {
    case LAY_VEC: return igemm_dma_table_cfg<bf16_t, false>(cfg, out, lds);
    case LAY_VEC_UNI: return igemm_dma_table_cfg<bf16_t, true>(cfg, out, lds);
    case LAY_HALO: return halo_table<bf16_t>(out, lds);
    case LAY_SCALAR: return igemm_table_cfg<bf16_t, LAY_SCALAR>(cfg, out, lds);
    case LAY_VEC_NB: return igemm_table_cfg<bf16_t, LAY_VEC_NB>(cfg, out, lds);
    case LAY_SCALAR_NB: return igemm_table_cfg<bf16_t, LAY_SCALAR_NB>(cfg, out, lds);
    default: return -1;
    }
}
}  // namespace miriam
