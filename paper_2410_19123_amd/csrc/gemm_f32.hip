// fp32 instantiations of the grouped GEMM (gate/up + SiLU*mul, plain store).
#include "gemm_kernels.hpp"

namespace readme {

hipError_t launch_tile_f32_gate_up(int tile, GemmArgs g, hipStream_t s) {
    return launch_tile<true, EPI_GATE_UP_SILU>(tile, g, s);
}

hipError_t launch_tile_f32_store(int tile, GemmArgs g, hipStream_t s) {
    return launch_tile<true, EPI_STORE>(tile, g, s);
}

}  // namespace readme
