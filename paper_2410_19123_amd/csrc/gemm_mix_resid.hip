// bf16 grouped GEMM with tiles of several heights in one launch: fp32 residual add (stacked layers).
#include "gemm_mix.hpp"

namespace readme {

hipError_t launch_mix_bf16_resid(int tile, GemmArgs g, hipStream_t s) {
    return launch_mix_tile<EPI_RESID_ADD>(tile, g, s);
}

}  // namespace readme
