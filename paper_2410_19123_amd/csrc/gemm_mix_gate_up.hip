// bf16 grouped GEMM with tiles of several heights in one launch: gate/up + SiLU*mul.
#include "gemm_mix.hpp"

namespace readme {

hipError_t launch_mix_bf16_gate_up(int tile, GemmArgs g, hipStream_t s) {
    return launch_mix_tile<EPI_GATE_UP_SILU>(tile, g, s);
}

}  // namespace readme
