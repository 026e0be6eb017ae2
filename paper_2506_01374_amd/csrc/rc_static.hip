// rc_launch_static: launching a plan with no device allocation, for callers
// that cannot allocate (code under HIP graph capture, tight serving loops).
//
// The workspace a plan needs (the gated MLP's hidden activations, the MoE
// routing tables and permuted rows, attention partial states, split-K
// partial sums) lives in one file-scope device array instead of a
// caller-allocated buffer.  Each device the library runs on holds its own
// copy of the array from the first call on that device until the process
// ends.  Host code never uses the array's name as an address: its device
// address is fetched once per device with hipGetSymbolAddress (with that
// device current) and kept; kernels receive that address as their
// workspace.
//
// No kernel of the library needs its workspace to start at zero (every part
// is written before it is read within one launch), so nothing is cleared.
// Every call on one device shares that device's array, which keeps the last
// call's contents: calls that overlap on one device (different streams, or
// host threads) race.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "rc_internal.h"

#define RC_STATIC_SCRATCH_BYTES ((size_t)64 << 20)

static __device__ __align__(256) unsigned char scratch[RC_STATIC_SCRATCH_BYTES];

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex g_static_mu;
void *g_scratch_ptr[MAX_DEVICES] = {};

// Device address of this device's copy of `scratch`, looked up once.
rc_status scratch_on_current_device(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return rc::fail(RC_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
    if (dev < 0 || dev >= MAX_DEVICES) return rc::fail(RC_ERR_UNSUPPORTED, "device index beyond 64");
    std::lock_guard<std::mutex> g(g_static_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        e = hipGetSymbolAddress((void **)&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr)
            return rc::fail(RC_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return RC_OK;
}

}  // namespace

extern "C" {

size_t rc_static_scratch_bytes(void) { return RC_STATIC_SCRATCH_BYTES; }

rc_status rc_launch_static(const rc_plan *p, const rc_args *a, void *stream) {
    if (!p || !a) return rc::fail(RC_ERR_INVALID_ARGUMENT, "null plan or args");
    size_t need = 0;
    rc_status r = rc_plan_workspace(p, &need);
    if (r != RC_OK) return r;
    if (need > RC_STATIC_SCRATCH_BYTES)
        return rc::fail(RC_ERR_OUT_OF_MEMORY, "plan needs a workspace of " + std::to_string(need) +
                                                  " bytes, more than the " +
                                                  std::to_string(RC_STATIC_SCRATCH_BYTES) +
                                                  "-byte static scratch; use rc_launch");
    void *ws = nullptr;
    if (need > 0) {
        r = scratch_on_current_device(&ws);
        if (r != RC_OK) return r;
    }
    return rc::launch_plan(p, a, ws, need > 0 ? RC_STATIC_SCRATCH_BYTES : 0, stream);
}

}  // extern "C"
