// tt_verify_noalloc: tt_verify for callers that cannot allocate device memory (code under HIP
// graph capture, tight serving loops, harnesses that forbid hipMalloc).  The verification's
// scratch (per-stream Q62 mass and selected row, per-chunk Q62 sums) lives in a file-scope
// device array of kNoallocScratchBytes instead of a caller workspace; the kernels are tt_verify's.
//
// Each GPU holds its own copy of the array until the process ends.  Its device address is
// looked up once per device (hipGetSymbolAddress, on the first call with that device current)
// and that address, never the array's host-side name, is what the kernels receive.  The
// scratch needs no initialisation (every launch writes what it reads), and every call on a
// GPU shares that GPU's array: calls that overlap in time on one GPU race.
#include <mutex>

#include "tt_internal.h"

namespace tt {
namespace {

constexpr size_t kNoallocScratchBytes = size_t(8) << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices] = {};

// The current device's scratch address, looked up on the device's first call; nullptr if the
// lookup fails.
void *device_scratch() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
        g_scratch_ptr[dev] = ptr;
    }
    return g_scratch_ptr[dev];
}

}  // namespace
}  // namespace tt

extern "C" int tt_verify_noalloc(int32_t n_streams, int32_t v_t, const int32_t *target_ids,
                                 const int32_t *target_off, const float *q, const float *target_probs,
                                 int64_t target_ld, const float *u_accept, const float *u_sample, int32_t max_m,
                                 int32_t *n_accepted, int32_t *out_token, float *residual, void *stream) {
    size_t need = 0;
    const int st = tt_verify_workspace_size(n_streams, v_t, &need);
    if (st != TT_OK) return st;
    if (need > tt::kNoallocScratchBytes) return TT_EWORKSPACE;
    void *ws = tt::device_scratch();
    if (ws == nullptr) return TT_ELAUNCH;
    return tt_verify(n_streams, v_t, target_ids, target_off, q, target_probs, target_ld, u_accept, u_sample, max_m,
                     n_accepted, out_token, residual, ws, tt::kNoallocScratchBytes, stream);
}
