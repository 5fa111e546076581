// The spectral correction without a caller workspace: sc_correct_static runs
// sc_correct's kernels on a file-scope device array, for callers that cannot
// allocate device memory (code under HIP graph capture, serving loops that
// forbid allocation).  Nothing else in the library refers to the array.
#include "common.h"

#include <mutex>
#include <vector>

namespace acsc {
namespace {

constexpr size_t kStaticScratchBytes = static_cast<size_t>(SC_STATIC_SCRATCH_BYTES);

// Each device that runs the entry point holds its own copy of the array until
// the process ends.  In host code `scratch` names a host-side stand-in, never
// the device memory: kernels and copies get the address that
// hipGetSymbolAddress returns for the current device.
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

std::mutex g_mu;
std::vector<void *> g_addr;   // device ordinal -> that device's copy of `scratch`

int scratch_address(void **out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return set_error(ACSC_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
    std::lock_guard<std::mutex> lk(g_mu);
    if (static_cast<size_t>(dev) >= g_addr.size())
        g_addr.resize(static_cast<size_t>(dev) + 1, nullptr);
    if (!g_addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return set_error(ACSC_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                             hipGetErrorString(e));
        g_addr[dev] = p;
    }
    *out = g_addr[dev];
    return ACSC_OK;
}

}  // namespace
}  // namespace acsc

extern "C" int sc_correct_static(const void *G, acsc_dtype dt, int m, int n, const float *U, const float *d,
                                 const float *V, int r, float alpha, void *G_proj, hipStream_t stream)
{
    using namespace acsc;
    size_t need = 0;
    int rc = sc_adamw_workspace_size(m, n, r, dt, &need);   // validates dt, m, n, r (clears the error)
    if (rc)
        return rc;
    ACSC_CHECK_ARG(need <= kStaticScratchBytes, ACSC_ENOSPC,
                   "a %d x %d correction at r=%d needs %zu bytes of scratch; sc_correct_static holds %zu "
                   "(use sc_correct with a workspace)", m, n, r, need, kStaticScratchBytes);
    void *ws = nullptr;
    if ((rc = scratch_address(&ws)))
        return rc;
    return sc_correct(G, dt, m, n, U, d, V, r, alpha, G_proj, ws, kStaticScratchBytes, stream);
}
