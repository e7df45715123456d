// htam_attend_transitions_noalloc: the fine stage with its workspace in a
// file-scope device array instead of a caller buffer, for callers that cannot
// allocate device memory (code under stream capture, tight serving loops).
//
// The array is the library's one piece of device memory of its own. Every
// GPU the library runs on holds its own copy for the life of the process, at
// its own address, which is looked up once per device with
// hipGetSymbolAddress; host code uses only that address, never the array's
// name (which in host code is a stand-in, not a device pointer). All calls on
// one GPU share the array: calls that overlap in time on one GPU race. The
// kernels clear every counter and table they read before reading it, so no
// state carries over from one call to the next.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "../../include/htam.h"
#include "internal.hpp"

namespace {

constexpr size_t kScratchBytes = size_t(HTAM_NOALLOC_SCRATCH_MIB) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_ptr[kMaxDevices] = {};

// The array's address on the current device (looked up on the first call on
// that device, with that device current); nullptr after reporting the error.
void *scratch_ptr() {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        htam::report_error(HTAM_ERR_DEVICE, "htam_attend_transitions_noalloc: no usable current device");
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            htam::report_error(HTAM_ERR_DEVICE, (std::string("htam_attend_transitions_noalloc: "
                                                             "hipGetSymbolAddress: ") +
                                                 hipGetErrorString(e)).c_str());
            return nullptr;
        }
        g_ptr[dev] = p;
    }
    return g_ptr[dev];
}

}  // namespace

extern "C" __attribute__((visibility("default"))) htam_status htam_attend_transitions_noalloc(
    const htam_bank *bank, const void *q, int32_t q_dtype, int32_t n_queries,
    const int32_t *sel_cluster, int32_t top_c, float tau, int32_t top_k, float *slot_max,
    float *slot_sum, float *cand_score, int32_t *cand_id, hipStream_t stream) {
    const size_t need = htam_attend_transitions_workspace_size(bank, n_queries, top_c, top_k);
    if (need > kScratchBytes) {
        // (argument errors give need == 0 and are reported by the call below)
        const std::string msg = "htam_attend_transitions_noalloc: this call needs " +
                                std::to_string(need) + " bytes of workspace, more than the " +
                                std::to_string(kScratchBytes) +
                                " bytes of the library's scratch array; use "
                                "htam_attend_transitions with a caller workspace";
        return (htam_status)htam::report_error(HTAM_ERR_WORKSPACE, msg.c_str());
    }
    void *ws = scratch_ptr();
    if (!ws) return HTAM_ERR_DEVICE;
    return htam_attend_transitions(bank, q, q_dtype, n_queries, sel_cluster, top_c, tau, top_k,
                                   slot_max, slot_sum, cand_score, cand_id, ws, kScratchBytes,
                                   stream);
}
