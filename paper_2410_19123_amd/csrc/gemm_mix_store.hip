// bf16 grouped GEMM with tiles of several heights in one launch: plain store (down projection).
#include "gemm_mix.hpp"

namespace readme {

hipError_t launch_mix_bf16_store(int tile, GemmArgs g, hipStream_t s) {
    return launch_mix_tile<EPI_STORE>(tile, g, s);
}

}  // namespace readme
