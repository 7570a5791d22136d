// One-time repack of expert weights into the layout the FFN kernels stream.
//
// gate/up block [E][2*Ip][d]: 32-row groups alternate gate (even group g)
//   and up (odd group g) for intermediate neurons 32*(g/2) .. +31, so a
//   32-column MFMA tile of gate outputs and the next one of up outputs hold
//   the same neurons and SiLU(g)*u can be formed in registers.
// down block [E][d][Ip]: W_down rows with the intermediate axis padded.
// Neurons i >= I are zero (exact: silu(0) * 0 = 0 and zero columns add 0).
#include "common.hpp"
#include "internal.hpp"

namespace readme {

template <typename T>
__global__ __launch_bounds__(256) void k_pack_gate_up(int64_t E, int64_t d, int64_t I,
                                                      int64_t Ip, const T* __restrict__ wg,
                                                      const T* __restrict__ wu,
                                                      T* __restrict__ out) {
    const int64_t total = E * 2 * Ip * d;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total;
         o += (int64_t)gridDim.x * blockDim.x) {
        const int64_t k = o % d;
        const int64_t p = (o / d) % (2 * Ip);
        const int64_t e = o / (d * 2 * Ip);
        const int64_t g = p / 32;
        const int64_t i = (g / 2) * 32 + (p % 32);
        T v = T(0);
        if (i < I) v = ((g & 1) ? wu : wg)[(e * I + i) * d + k];
        out[o] = v;
    }
}

template <typename T>
__global__ __launch_bounds__(256) void k_pack_down(int64_t E, int64_t d, int64_t I, int64_t Ip,
                                                   const T* __restrict__ wd,
                                                   T* __restrict__ out) {
    const int64_t total = E * d * Ip;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total;
         o += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = o % Ip;
        const int64_t row = o / Ip;  // e * d + c
        out[o] = i < I ? wd[row * I + i] : T(0);
    }
}

template <typename T>
static hipError_t pack_t(int64_t E, int64_t d, int64_t I, const void* wg, const void* wu,
                         const void* wd, void* packed, hipStream_t s) {
    const int64_t Ip = padded_I(I);
    T* gu = reinterpret_cast<T*>(packed);
    T* dn = gu + E * 2 * Ip * d;
    const unsigned blocks = 4096;
    k_pack_gate_up<T><<<blocks, 256, 0, s>>>(E, d, I, Ip, reinterpret_cast<const T*>(wg),
                                              reinterpret_cast<const T*>(wu), gu);
    k_pack_down<T><<<blocks, 256, 0, s>>>(E, d, I, Ip, reinterpret_cast<const T*>(wd), dn);
    return hipGetLastError();
}

hipError_t launch_pack(readme_dtype dt, int64_t E, int64_t d, int64_t I, const void* wg,
                       const void* wu, const void* wd, void* packed, hipStream_t s) {
    if (dt == README_F32) return pack_t<uint32_t>(E, d, I, wg, wu, wd, packed, s);
    return pack_t<uint16_t>(E, d, I, wg, wu, wd, packed, s);
}

}  // namespace readme
