// noalloc.hip -- ts_chain_marginals_noalloc: the marginals call for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops, harnesses that
// forbid allocation).  Instead of a caller-provided workspace it uses one file-scope device
// array of kScratchBytes per GPU, which the code object holds from the first call on that
// GPU until the process ends.  The kernels are those of ts_chain_marginals; they receive the
// array's device address (looked up once per device with hipGetSymbolAddress) exactly as
// they receive the caller's workspace there.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "internal.h"
#include "small.h"
#include "ts_chain.h"

namespace tsc {
namespace {

constexpr size_t kScratchBytes = (size_t)64 << 20;   // 64 MiB
constexpr int kMaxScratchDevices = 64;

// The scratch array.  In host code this name is a host-side stand-in, not a device address:
// only the pointer returned by hipGetSymbolAddress (per device) is ever passed to kernels.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// Device address of the calling thread's current device's copy of `scratch`.
hipError_t scratch_of_current_device(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!ptr) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace
}  // namespace tsc

using namespace tsc;

extern "C" {

size_t ts_chain_noalloc_scratch_bytes(void) { return kScratchBytes; }

ts_status ts_chain_marginals_noalloc(const float* pot, const int32_t* lengths, int64_t B,
                                     int64_t N, int64_t C, float* logZ, float* marg,
                                     void* stream) {
    // the same validation and plan as ts_chain_marginals, with the workspace size checked
    // against the scratch array before anything else touches the device
    const size_t need = ts_chain_workspace_bytes(TS_OP_MARGINALS, B, N, C);
    if (need > kScratchBytes) {
        // (sizes the plan rejects give 0 and fall through to the call's own checks)
        return report_error(
            TS_ERR_BAD_DIM, ("ts_chain_marginals_noalloc: this problem needs " +
                             std::to_string(need) + " bytes of scratch; the allocation-free "
                             "entry point holds at most " + std::to_string(kScratchBytes) +
                             " (use ts_chain_marginals with a workspace)").c_str());
    }
    void* ws = nullptr;
    if (need > 0) {
        const hipError_t e = scratch_of_current_device(&ws);
        if (e != hipSuccess)
            return report_error(
                TS_ERR_HIP, (std::string("ts_chain_marginals_noalloc: scratch address: ") +
                             hipGetErrorString(e)).c_str());
    }
    return ts_chain_marginals(pot, lengths, B, N, C, logZ, marg, ws, need, stream);
}

}  // extern "C"
