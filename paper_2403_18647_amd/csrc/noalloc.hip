// The skinny GEMM entry point for callers that cannot allocate device memory
// (code under stream capture, serving loops that forbid allocation): the same
// kernels as sdsat_linear, with the matrix-typed copy of X staged in a static
// device array instead of a caller-provided scratch buffer.
//
// Each GPU the library runs on holds its own copy of `scratch` (4 MiB) until
// the process ends.  Host code never passes the array's name to a kernel: the
// name is a host-side stand-in, so the device address of the current device's
// copy is looked up once per device (with that device current) and kept.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "../../include/sdsat.h"
#include "kernels.h"

namespace sdsat {

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's copy of `scratch`.
hipError_t scratch_ptr(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace
}  // namespace sdsat

extern "C" int sdsat_linear_noalloc(int32_t dtype, int32_t M, int32_t N, int32_t K, const float* d_x,
                                    const void* d_packed, float* d_y, void* hip_stream) {
    using namespace sdsat;
    if ((dtype != SDSAT_DTYPE_FP32 && dtype != SDSAT_DTYPE_BF16) || M < 1 || M > 64 || N < 1 || K < 1 || !d_x ||
        !d_packed || !d_y)
        return report_error(SDSAT_EINVAL, "bad linear_noalloc arguments");
    const int nt = (N + 15) / 16, ks = (K + 31) / 32;
    const size_t need = (size_t)M * ks * 32 * (dtype == SDSAT_DTYPE_BF16 ? 2 : 4);
    if (need > kNoAllocScratchBytes)
        return report_error(SDSAT_EINVAL, "linear_noalloc: M x K (padded to 32) elements exceed the 4 MiB static "
                                          "scratch");
    void* buf = nullptr;
    hipError_t e = scratch_ptr(&buf);
    if (e != hipSuccess)
        return report_error(SDSAT_EDEVICE, std::string("linear_noalloc scratch lookup: ") + hipGetErrorString(e));
    hipStream_t st = static_cast<hipStream_t>(hip_stream);
    // every element the GEMM reads (rows 0..M-1, columns 0..32*ks-1, pads zero) is rewritten here, so
    // nothing a previous call left in the array is read
    e = launch_to_elem_rows(dtype, d_x, M, K, buf, ks * 32, st);
    if (e != hipSuccess) return report_error(SDSAT_EDEVICE, std::string("linear_noalloc input: ") + hipGetErrorString(e));
    const GemmPlan p = plan_gemm(M, nt, ks);
    GemmArgs a{};
    a.M = M; a.N = N; a.K = K; a.n_tiles = nt; a.k_steps = ks; a.W = d_packed;
    a.xa = buf; a.ldx = ks * 32; a.y = d_y; a.ldy = N;
    e = launch_gemm(dtype, EP_STORE, p, a, st);
    if (e != hipSuccess) return report_error(SDSAT_EDEVICE, std::string("linear_noalloc launch: ") + hipGetErrorString(e));
    return SDSAT_OK;
}
