// readme_moe_ffn_fused without a caller workspace, for callers that cannot
// allocate device memory (code under graph capture, tight serving loops,
// harnesses that forbid allocation).  The intermediate h = silu(g) * u,
// the one scratch buffer of the FFN, lives in a file-scope device array of
// fixed size instead; every call on a GPU reuses that GPU's copy.
//
// The array's name is only a host-side stand-in for it: its device address
// is looked up once per device (hipGetSymbolAddress, with the device
// current) and that address is what the kernels receive.  Nothing here
// allocates or frees.
#include <mutex>

#include "common.hpp"
#include "internal.hpp"

static __device__ __align__(256) unsigned char scratch[README_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
void* g_scratch[kMaxDevices];  // device address of `scratch`, per device
std::mutex g_scratch_mu;

// Device address of the current device's scratch array (looked up on the
// first call on that device).
hipError_t scratch_address(void** out) {
    int dev = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return err;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (err != hipSuccess) return err;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return hipSuccess;
}

}  // namespace

extern "C" {

readme_status readme_moe_ffn_fused_noalloc(readme_dtype dt, int64_t T, int64_t d, int32_t E,
                                           int64_t I, const void* x, const int32_t* perm,
                                           const int32_t* offsets, const void* packed, void* y,
                                           void* stream) {
    using namespace readme;
    if (!(dt == README_F32 || dt == README_BF16) || T < 0 || d <= 0 || I < 1)
        return README_ERR_ARG;
    if (E < 1 || E > README_MAX_EXPERTS || d % 64 != 0 || T > INT32_MAX)
        return README_ERR_UNSUPPORTED;
    // h is T x padded(I) elements; beyond the fixed array the call is refused.
    const size_t h_bytes = (size_t)T * padded_I(I) * dtype_size(dt);
    if (h_bytes > (size_t)README_NOALLOC_SCRATCH_BYTES) return README_ERR_UNSUPPORTED;
    if (T == 0) return README_OK;
    if (!x || !perm || !offsets || !packed || !y) return README_ERR_ARG;
    const auto a16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; };
    if (!a16(x) || !a16(packed) || !a16(y)) return README_ERR_ARG;
    void* h = nullptr;
    if (scratch_address(&h) != hipSuccess) return README_ERR_HIP;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    // h needs no clearing: gate/up writes every column of every routed row,
    // and down reads only those rows.
    GemmArgs gu = gate_up_args(dt, T, d, E, I, x, offsets, packed, h);
    gu.a_rows = perm;
    hipError_t err = launch_grouped_gemm(dt == README_F32, EPI_GATE_UP_SILU, gu, s);
    if (err != hipSuccess) return README_ERR_HIP;
    GemmArgs dn = down_args(dt, T, d, E, I, h, offsets, packed, y);
    dn.c_rows = perm;
    err = launch_grouped_gemm(dt == README_F32, EPI_STORE, dn, s);
    return err == hipSuccess ? README_OK : README_ERR_HIP;
}

}  // extern "C"
