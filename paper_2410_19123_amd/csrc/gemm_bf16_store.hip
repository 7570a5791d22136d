// bf16 instantiations of the grouped GEMM: plain store.
#include "gemm_kernels.hpp"

namespace readme {

hipError_t launch_tile_bf16_store(int tile, GemmArgs g, hipStream_t s) {
    return launch_tile<false, EPI_STORE>(tile, g, s);
}

}  // namespace readme
