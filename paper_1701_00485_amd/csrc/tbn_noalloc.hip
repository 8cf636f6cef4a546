// tbn_noalloc.hip -- tbn_conv2d_fwd_noalloc: the forward pass with its workspace taken from
// a library-owned static device array instead of caller memory, for callers that cannot
// allocate device memory.  Each device holds its own copy of the array; its address is
// looked up once per device (with that device current) and cached.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>
#include <string>

#include "tbn.h"
#include "tbn_kernels.h"

namespace {

// Kernel-side scratch of the no-allocation forward pass.  Host code never uses this name as
// an address: it uses the per-device pointer from hipGetSymbolAddress below.
static __device__ __align__(256) uint8_t scratch[TBN_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of the current device's scratch array (looked up on the first call on
// that device).
tbn_status scratch_ptr(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return tbn::set_error(TBN_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices) return tbn::set_error(TBN_ERR_UNSUPPORTED, "device index beyond 63");
    void* p = g_scratch[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch[dev].load(std::memory_order_relaxed);
        if (!p) {
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess || !p)
                return tbn::set_error(TBN_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") +
                                                       hipGetErrorString(e));
            g_scratch[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return TBN_OK;
}

}  // namespace

extern "C" tbn_status tbn_conv2d_fwd_noalloc(const tbn_conv_desc* desc, const void* x, tbn_dtype xt,
                                             const uint32_t* codes, const float* alpha, const tbn_epilogue* ep,
                                             void* y, tbn_dtype yt, hipStream_t stream) {
    size_t need = 0;
    tbn_status st = tbn_workspace_size(TBN_OP_FWD, desc, &need);
    if (st != TBN_OK) return st;
    if (need > (size_t)TBN_NOALLOC_SCRATCH_BYTES)
        return tbn::set_error(TBN_ERR_WORKSPACE, "the layer needs " + std::to_string(need) +
                                                     " bytes of workspace, more than the " +
                                                     std::to_string((size_t)TBN_NOALLOC_SCRATCH_BYTES) +
                                                     " bytes of static scratch; call tbn_conv2d_fwd with a workspace");
    void* ws = nullptr;
    if (need) {
        st = scratch_ptr(&ws);
        if (st != TBN_OK) return st;
    }
    // the forward pass's workspace holds split-reduction partials or a bordered input copy,
    // both fully written before they are read: nothing in it has to start at zero
    return tbn_conv2d_fwd(desc, x, xt, codes, alpha, ep, y, yt, ws, need ? (size_t)TBN_NOALLOC_SCRATCH_BYTES : 0,
                          stream);
}
