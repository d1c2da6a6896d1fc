// Phase timing for kernel tuning, compiled in only with -DTT_PHASE_STAMPS (the library is
// built without it).  Lane 0 of a workgroup's wave 0 (TT_STAMP) or of the wave that reaches it
// (TT_STAMP_WAVE) records the 100 MHz real-time counter at numbered points of a kernel into a
// table of kStampSlots entries per workgroup (TT_STAMP_VAL records a value instead); the host
// reads a translation unit's table through tt_phase_stamps_<unit>(), exported only by such a
// build.
#pragma once

#include <hip/hip_runtime.h>

namespace tt {
constexpr int kStampSlots = 16;
constexpr int kStampBlocks = 8192;
}  // namespace tt

#ifdef TT_PHASE_STAMPS
static __device__ unsigned long long g_phase_stamps[tt::kStampBlocks * tt::kStampSlots];
#define TT_STAMPS_TABLE(unit)                                                                   \
    extern "C" void *tt_phase_stamps_##unit() {                                                 \
        void *p = nullptr;                                                                      \
        return hipGetSymbolAddress(&p, HIP_SYMBOL(g_phase_stamps)) == hipSuccess ? p : nullptr; \
    }
#define TT_STAMP_VAL(k, v)                                                 \
    do {                                                                   \
        if (threadIdx.x % 64 == 0 && blockIdx.x < tt::kStampBlocks)        \
            g_phase_stamps[blockIdx.x * tt::kStampSlots + (k)] = (v);      \
    } while (0)
#define TT_STAMP(k)                                    \
    do {                                               \
        if (threadIdx.x == 0)                          \
            TT_STAMP_VAL(k, __builtin_amdgcn_s_memrealtime()); \
    } while (0)
#define TT_STAMP_WAVE(k) TT_STAMP_VAL(k, __builtin_amdgcn_s_memrealtime())
#else
#define TT_STAMPS_TABLE(unit)
#define TT_STAMP_VAL(k, v) \
    do {                   \
    } while (0)
#define TT_STAMP(k) \
    do {            \
    } while (0)
#define TT_STAMP_WAVE(k) \
    do {                 \
    } while (0)
#endif
