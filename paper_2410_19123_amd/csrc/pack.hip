// One-time repack of expert weights into the layout the FFN kernels stream.
//
// Logical packed matrices (K-contiguous weight rows, as the GEMM consumes):
//   gate/up  [E][2*Ip][d]: 32-row groups alternate gate (even group g) and up
//            (odd group g) for intermediate neurons 32*(g/2) .. +31, so a
//            32-column MFMA tile of gate outputs and the next one of up
//            outputs hold the same neurons and SiLU(g)*u forms in registers;
//   down     [E][d][Ip]: W_down rows, the intermediate axis padded.
// Neurons i >= I are zero (exact: silu(0) * 0 = 0 and zero columns add 0).
//
// Physical layout of each logical [N][K] matrix (N a multiple of 32, K*elt a
// multiple of 128 bytes): blocks of 32 rows x 128 bytes of K, ordered
// (K block, row group) -- all row groups of one K block side by side --
// each block stored as the four matrix-core operand fragments it holds:
// 16-byte chunk c of row r goes to fragment c/2, lane (c%2)*32 + r, i.e.
// byte (c/2)*1024 + ((c%2)*32 + r)*16 of the block.  A fragment is then one
// contiguous KB that a wave loads with one fully coalesced instruction (lane
// l takes bytes 16*l .. 16*l+15), whether it goes to registers directly or
// through LDS.  Workgroups that stream neighbouring row groups at about the
// same K block then read neighbouring 4 KB blocks: a probe of the decode
// weight streams (616 row groups, four per workgroup) moved 5.95 TB/s in
// this order against 5.53 TB/s with each row group's K blocks consecutive.
#include "common.hpp"
#include "internal.hpp"

namespace readme {

// Byte offset of element (n, k) of a blocked [N][K] matrix with `groups`
// 32-row groups (N / 32), elements of `esz` bytes.
__device__ __forceinline__ int64_t blocked_offset(int64_t n, int64_t k, int64_t groups,
                                                  int esz) {
    const int64_t kb = k * esz;               // byte column
    const int64_t grp = n >> 5, r = n & 31;
    const int64_t s = kb >> 7, c = (kb >> 4) & 7, inner = kb & 15;
    const int64_t slot = (c >> 1) * 64 + (c & 1) * 32 + r;
    return (s * groups + grp) * 4096 + slot * 16 + inner;
}

// Gate/up: destination element o of [2*Ip][d] (logical), source gate or up.
template <typename T>
__global__ __launch_bounds__(256) void k_pack_gate_up(int64_t E, int64_t d, int64_t I,
                                                      int64_t Ip, const T* __restrict__ wg,
                                                      const T* __restrict__ wu,
                                                      char* __restrict__ out) {
    const int64_t per_e = 2 * Ip * d;
    const int64_t total = E * per_e;
    const int64_t groups = 2 * Ip / 32;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total;
         o += (int64_t)gridDim.x * blockDim.x) {
        const int64_t e = o / per_e;
        const int64_t rem = o - e * per_e;
        const int64_t p = rem / d, k = rem % d;
        const int64_t g = p / 32;
        const int64_t i = (g / 2) * 32 + (p % 32);
        T v = T(0);
        if (i < I) v = ((g & 1) ? wu : wg)[(e * I + i) * d + k];
        *reinterpret_cast<T*>(out + e * per_e * (int64_t)sizeof(T) +
                              blocked_offset(p, k, groups, sizeof(T))) = v;
    }
}

// Down: destination element of [d][Ip] (logical) from W_down, expert e's
// element (c, i) at wd[e * es + c * rs + i] ([E][d][I]: es = d*I, rs = I).
template <typename T>
__global__ __launch_bounds__(256) void k_pack_down(int64_t E, int64_t d, int64_t I, int64_t Ip,
                                                   int64_t es, int64_t rs,
                                                   const T* __restrict__ wd,
                                                   char* __restrict__ out) {
    const int64_t per_e = d * Ip;
    const int64_t total = E * per_e;
    const int64_t groups = d / 32;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total;
         o += (int64_t)gridDim.x * blockDim.x) {
        const int64_t e = o / per_e;
        const int64_t rem = o - e * per_e;
        const int64_t c = rem / Ip, i = rem % Ip;
        const T v = i < I ? wd[e * es + c * rs + i] : T(0);
        *reinterpret_cast<T*>(out + e * per_e * (int64_t)sizeof(T) +
                              blocked_offset(c, i, groups, sizeof(T))) = v;
    }
}

// Rows row0 .. row0 + n - 1 of a blocked bf16 [N][K] matrix (groups = N / 32
// row groups) from a row-major source [n][K] with rows ld elements apart.
__global__ __launch_bounds__(256) void k_pack_rows(int64_t n, int64_t K, int64_t groups,
                                                   int64_t row0, int64_t ld,
                                                   const uint16_t* __restrict__ src,
                                                   char* __restrict__ out) {
    const int64_t total = n * K;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total;
         o += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = o / K, k = o - (o / K) * K;
        *reinterpret_cast<uint16_t*>(out + blocked_offset(row0 + r, k, groups, 2)) =
            src[r * ld + k];
    }
}

template <typename T>
static hipError_t pack_t(int64_t E_all, int64_t e0, int64_t n, int64_t d, int64_t I,
                         const void* wg, const void* wu, const void* wd, int64_t es, int64_t rs,
                         void* packed, hipStream_t s) {
    const int64_t Ip = padded_I(I);
    const int64_t gu_e = 2 * Ip * d * (int64_t)sizeof(T), dn_e = d * Ip * (int64_t)sizeof(T);
    char* gu = reinterpret_cast<char*>(packed) + e0 * gu_e;
    char* dn = reinterpret_cast<char*>(packed) + E_all * gu_e + e0 * dn_e;
    const unsigned blocks = 4096;
    k_pack_gate_up<T><<<blocks, 256, 0, s>>>(n, d, I, Ip, reinterpret_cast<const T*>(wg),
                                              reinterpret_cast<const T*>(wu), gu);
    k_pack_down<T><<<blocks, 256, 0, s>>>(n, d, I, Ip, es, rs, reinterpret_cast<const T*>(wd),
                                           dn);
    return hipGetLastError();
}

hipError_t launch_pack_slots(readme_dtype dt, int64_t E_all, int64_t e0, int64_t n, int64_t d,
                             int64_t I, const void* wg, const void* wu, const void* wd,
                             int64_t wd_expert_stride, int64_t wd_row_stride, void* packed,
                             hipStream_t s) {
    if (dt == README_F32)
        return pack_t<uint32_t>(E_all, e0, n, d, I, wg, wu, wd, wd_expert_stride, wd_row_stride,
                                packed, s);
    return pack_t<uint16_t>(E_all, e0, n, d, I, wg, wu, wd, wd_expert_stride, wd_row_stride,
                            packed, s);
}

hipError_t launch_pack_rows_bf16(int64_t N, int64_t K, int64_t row0, int64_t n,
                                 const void* src, int64_t ld, void* packed, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const int64_t blocks = ceil_div(n * K, 256);
    k_pack_rows<<<(unsigned)(blocks < 4096 ? blocks : 4096), 256, 0, s>>>(
        n, K, N / 32, row0, ld, reinterpret_cast<const uint16_t*>(src),
        reinterpret_cast<char*>(packed));
    return hipGetLastError();
}

hipError_t launch_pack(readme_dtype dt, int64_t E, int64_t d, int64_t I, const void* wg,
                       const void* wu, const void* wd, void* packed, hipStream_t s) {
    return launch_pack_slots(dt, E, 0, E, d, I, wg, wu, wd, d * I, I, packed, s);
}

}  // namespace readme
