// bf16 instantiations of the grouped GEMM: gate/up + SiLU*mul.
#include "gemm_kernels.hpp"

namespace readme {

hipError_t launch_tile_bf16_gate_up(int tile, GemmArgs g, hipStream_t s) {
    return launch_tile<false, EPI_GATE_UP_SILU>(tile, g, s);
}

}  // namespace readme
