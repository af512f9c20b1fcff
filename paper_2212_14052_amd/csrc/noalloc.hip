// h3_statepass_conv_noalloc: state passing (Sec. 4.2, Algorithm 2) for
// callers that cannot allocate device memory.  Its scratch (chunk kernel,
// chunk end-states, initial-state tables and weights) lives in a file-scope
// device array of H3_NOALLOC_SCRATCH_BYTES instead of a caller workspace.
//
// In host code `scratch` names a host-side stand-in, not device memory: the
// array's device address is looked up once per device with
// hipGetSymbolAddress (that device current) and only that address is handed
// to kernels.  Every call on a device shares that device's array; calls that
// overlap in time on one device race on it.
#include <mutex>

#include "../../include/h3flash.h"
#include "internal.h"

namespace h3 {
namespace {

__device__ __align__(256) unsigned char scratch[H3_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices];   // device address of `scratch`, per device; null until looked up

// Device address of the current device's scratch array (looked up on the
// first call on that device).
int scratch_address(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return H3_EDEVICE;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return H3_EDEVICE;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return H3_OK;
}

}  // namespace
}  // namespace h3

extern "C" int h3_statepass_conv_noalloc(const void *u, const float *Abar, const float *Bbar, const float *C,
                                         const float *D, const float *x0, int B, int H, int L, int m, int chunk,
                                         int dtype, void *y, float *x_final, void *stream) {
    using namespace h3;
    const int st = statepass_check(u, Abar, Bbar, C, y, x_final, B, H, L, m, chunk, dtype);
    if (st != H3_OK) return st;
    if (statepass_workspace(B, H, L, m, chunk, dtype) > (size_t)H3_NOALLOC_SCRATCH_BYTES) return H3_EWORKSPACE;
    void *ws = nullptr;
    const int sa = scratch_address(&ws);
    if (sa != H3_OK) return sa;
    return statepass_run(u, Abar, Bbar, C, D, x0, B, H, L, m, chunk, dtype, y, x_final, (char *)ws,
                         (hipStream_t)stream);
}
