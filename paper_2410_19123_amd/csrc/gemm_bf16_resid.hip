// bf16 instantiations of the grouped GEMM: fp32 residual add.
#include "gemm_kernels.hpp"

namespace readme {

hipError_t launch_tile_bf16_resid(int tile, GemmArgs g, hipStream_t s) {
    return launch_tile<false, EPI_RESID_ADD>(tile, g, s);
}

}  // namespace readme
