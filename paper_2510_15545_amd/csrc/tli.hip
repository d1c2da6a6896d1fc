// Token-Level Intersection proposal rows (App. D Alg. 3) on gfx950.
//
// For each draft distribution q over V_d, q' over V_t is q(x) / S at y = d2t[x] for draft ids
// x in the vocabulary intersection and 0 elsewhere; S is the mass q puts on the intersection.
// Standard speculative sampling (App. D Alg. 4, tt_verify_dense) then runs with p and q'.
//
// Numerics: q is clamped to [0, 1] (NaN -> 0).  S is formed as the sampler forms its masses:
// every intersected q(x) is truncated to Q62 fixed point and the integers are summed exactly
// (128 bits per lane, so any row length and any order give the same sum), then the sum is
// rounded once to the nearest fp32 (ties to even).  q'(y) is the IEEE fp32 quotient
// q(x) / S; a row with S = 0 is written as zeros.
//
// One 1024-thread workgroup per row, two passes over the row:
//   1. coalesced reads of q and d2t (16-byte loads when the rows allow), Q62 sums in
//      registers, a wave and then a workgroup reduction of the 128-bit sums;
//   2. coalesced reads of t2d and writes of q' (16-byte stores when aligned), with q(x)
//      gathered from the row read in pass 1 (it is still in L2 or the Infinity Cache).
// The row is read from HBM once; the maps are shared by every row and stay in cache.
#include "verify_core.h"

namespace tt {
namespace {

using vcore::clamp01;
using vcore::q62;

constexpr int kThreads = 1024;
constexpr int kWave = 64;
constexpr int kUnroll = 4;  // 16-byte loads of each array a thread keeps in flight

struct U128 {
    uint64_t lo, hi;
};

__device__ __forceinline__ U128 add128(U128 a, U128 b) {
    U128 r;
    r.lo = a.lo + b.lo;
    r.hi = a.hi + b.hi + (r.lo < a.lo ? 1u : 0u);
    return r;
}

__device__ __forceinline__ U128 shfl_xor128(U128 v, int m) {
    U128 r;
    r.lo = __shfl_xor(v.lo, m);
    r.hi = __shfl_xor(v.hi, m);
    return r;
}

// N * 2^-62 rounded to the nearest fp32, ties to even (N < 2^128).
__device__ inline float q62_to_f32(U128 n) {
    if (n.hi == 0 && n.lo == 0) return 0.0f;
    const int bl = n.hi ? 128 - __clzll(n.hi) : 64 - __clzll(n.lo);  // bit length
    if (bl <= 24) return ldexpf((float)n.lo, -62);                   // exact
    const int sh = bl - 24;                                           // bits dropped, >= 1
    const uint64_t mant = sh >= 64 ? (n.hi >> (sh - 64)) : ((n.lo >> sh) | (n.hi << (64 - sh)));
    const int rb = sh - 1;  // the highest dropped bit
    const uint32_t round = (uint32_t)((rb >= 64 ? (n.hi >> (rb - 64)) : (n.lo >> rb)) & 1u);
    bool sticky;  // any dropped bit below the round bit
    if (rb == 0) sticky = false;
    else if (rb <= 64) sticky = (rb == 64 ? n.lo : (n.lo & ((1ull << rb) - 1))) != 0;
    else sticky = n.lo != 0 || (n.hi & ((1ull << (rb - 64)) - 1)) != 0;
    const uint64_t m = mant + ((round && (sticky || (mant & 1u))) ? 1u : 0u);  // may reach 2^24: still exact
    return ldexpf((float)m, sh - 62);
}

__global__ void __launch_bounds__(kThreads) tli_rows(TliArgs a, int vec_in, int vec_out) {
    const int r = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const float *q = a.draft_probs + (int64_t)r * a.draft_ld;
    float *out = a.q_out + (int64_t)r * a.q_ld;
    __shared__ U128 sh_part[kThreads / kWave];
    __shared__ float sh_S;

    // 1. exact Q62 sum of the intersected mass
    U128 acc{0, 0};
    auto add = [&](float x, int32_t m) {  // branch-free: the loads stay batched
        const uint64_t keep = 0ull - (uint64_t)(m >= 0);
        acc = add128(acc, U128{q62(clamp01(x)) & keep, 0});
    };
    int x0 = 0;
    if (vec_in) {
        const float4 *q4 = reinterpret_cast<const float4 *>(q);
        const int4 *m4 = reinterpret_cast<const int4 *>(a.d2t);
        const int n4 = a.v_d / 4;
        int k = tid;
        for (; k + (kUnroll - 1) * kThreads < n4; k += kUnroll * kThreads) {  // kUnroll loads of each in flight
            float4 v[kUnroll];
            int4 m[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                v[u] = q4[k + u * kThreads];
                m[u] = m4[k + u * kThreads];
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                add(v[u].x, m[u].x);
                add(v[u].y, m[u].y);
                add(v[u].z, m[u].z);
                add(v[u].w, m[u].w);
            }
        }
        for (; k < n4; k += kThreads) {
            const float4 v = q4[k];
            const int4 m = m4[k];
            add(v.x, m.x);
            add(v.y, m.y);
            add(v.z, m.z);
            add(v.w, m.w);
        }
        x0 = 4 * n4;
    }
    for (int x = x0 + tid; x < a.v_d; x += kThreads) add(q[x], a.d2t[x]);
    for (int m = kWave / 2; m > 0; m >>= 1) acc = add128(acc, shfl_xor128(acc, m));
    if (lane == 0) sh_part[wave] = acc;
    __syncthreads();
    if (tid == 0) {
        U128 tot{0, 0};
        for (int w = 0; w < kThreads / kWave; ++w) tot = add128(tot, sh_part[w]);
        sh_S = q62_to_f32(tot);
    }
    __syncthreads();
    const float S = sh_S;

    // 2. q' over the target vocabulary
    // every lane loads (q[0] outside the intersection) so the gathers of a batch stay in flight together
    auto gather = [&](int32_t x) -> float { return q[(x >= 0 && x < a.v_d) ? x : 0]; };
    auto value = [&](int32_t x, float g) -> float {
        return (x >= 0 && x < a.v_d && S > 0.0f) ? clamp01(g) / S : 0.0f;
    };
    int y0 = 0;
    if (vec_out) {
        const int4 *m4 = reinterpret_cast<const int4 *>(a.t2d);
        float4 *o4 = reinterpret_cast<float4 *>(out);
        const int n4 = a.v_t / 4;
        int k = tid;
        for (; k + (kUnroll - 1) * kThreads < n4; k += kUnroll * kThreads) {
            int4 m[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) m[u] = m4[k + u * kThreads];
            float4 g[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u)
                g[u] = make_float4(gather(m[u].x), gather(m[u].y), gather(m[u].z), gather(m[u].w));
#pragma unroll
            for (int u = 0; u < kUnroll; ++u)
                o4[k + u * kThreads] = make_float4(value(m[u].x, g[u].x), value(m[u].y, g[u].y),
                                                   value(m[u].z, g[u].z), value(m[u].w, g[u].w));
        }
        for (; k < n4; k += kThreads) {
            const int4 m = m4[k];
            const float4 g = make_float4(gather(m.x), gather(m.y), gather(m.z), gather(m.w));
            o4[k] = make_float4(value(m.x, g.x), value(m.y, g.y), value(m.z, g.z), value(m.w, g.w));
        }
        y0 = 4 * n4;
    }
    for (int y = y0 + tid; y < a.v_t; y += kThreads) {
        const int32_t x = a.t2d[y];
        out[y] = value(x, gather(x));
    }
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

int launch_tli_proposal(const TliArgs &a, hipStream_t stream) {
    if (a.n_rows == 0) return TT_OK;
    const int vec_in = aligned16(a.draft_probs) && aligned16(a.d2t) && a.draft_ld % 4 == 0;
    const int vec_out = aligned16(a.q_out) && aligned16(a.t2d) && a.q_ld % 4 == 0;
    hipLaunchKernelGGL(tli_rows, dim3(a.n_rows), dim3(kThreads), 0, stream, a, vec_in, vec_out);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

}  // namespace tt
