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

TT_STAMPS_TABLE(tli)

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

// S, the mass row q puts on the intersection: every intersected q(x) (clamped to [0, 1])
// truncated to Q62 and the integers summed exactly, rounded once to fp32.  Called by every
// thread of the workgroup (barriers inside); sh_part holds a partial sum per wave.
__device__ float row_mass(const float *q, const int32_t *d2t, int v_d, bool vec_in, U128 *sh_part, float *sh_S) {
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    U128 acc{0, 0};
    auto add = [&](float x, int32_t m) {  // branch-free: the loads stay batched
        const uint64_t keep = 0ull - (uint64_t)(m >= 0);
        acc = add128(acc, U128{q62(clamp01(x)) & keep, 0});
    };
    int x0 = 0;
    if (vec_in) {
        const float4 *q4 = reinterpret_cast<const float4 *>(q);
        const int4 *m4 = reinterpret_cast<const int4 *>(d2t);
        const int n4 = v_d / 4;
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
    for (int x = x0 + tid; x < v_d; x += kThreads) add(q[x], d2t[x]);
    for (int m = kWave / 2; m > 0; m >>= 1) acc = add128(acc, shfl_xor128(acc, m));
    if (lane == 0) sh_part[wave] = acc;
    __syncthreads();
    if (tid == 0) {
        U128 tot{0, 0};
        for (int w = 0; w < kThreads / kWave; ++w) tot = add128(tot, sh_part[w]);
        *sh_S = q62_to_f32(tot);
    }
    __syncthreads();
    return *sh_S;
}

// q'(y) for the draft id x = t2d[y] whose mass g = q(x) was gathered (g = 0 when x lies
// outside [0, v_d): the entry is 0 either way); 0 when S is not positive.
__device__ __forceinline__ float qprime(float g, float S) { return S > 0.0f ? clamp01(g) / S : 0.0f; }

__global__ void __launch_bounds__(kThreads) tli_rows(TliArgs a, int vec_in, int vec_out) {
    const int r = blockIdx.x;
    const int tid = threadIdx.x;
    const float *q = a.draft_probs + (int64_t)r * a.draft_ld;
    float *out = a.q_out + (int64_t)r * a.q_ld;
    __shared__ U128 sh_part[kThreads / kWave];
    __shared__ float sh_S;

    // 1. exact Q62 sum of the intersected mass
    const float S = row_mass(q, a.d2t, a.v_d, vec_in != 0, sh_part, &sh_S);

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

// ------------------------------------------------------------------ fused verification
// Standard speculative sampling (App. D Alg. 4) with the TLI proposal of each drafted
// position formed where it is used, so q' rows are never written: one 1024-thread workgroup
// per stream.
//   acceptance: q'_j(t_j) = q_j(t2d[t_j]) / S_j, one gathered draft mass per position; S_j
//     from draft_mass (wave 0 tests 64 positions per ballot) or, without it, by a pass over
//     draft row j (the whole workgroup, row after row until the first rejection);
//   residual: the chunk sums of max(0, p - q') over target row gamma, q' gathered through t2d
//     from draft row gamma (the bonus row as is after full acceptance), the row read in
//     vcore::load_chunk's element order (a 16-byte load instruction covers 1 KB; a chunk's sum
//     does not depend on the order), then the exact inverse-CDF sample by wave 0, which reads
//     the crossing chunk again in position order -- the arithmetic of tt_verify_dense element
//     for element.
constexpr int kWaves = kThreads / kWave;

struct TliVerifyParams {
    TliVerifyArgs a;
    int32_t nc, vec_t, vec_d;
};

// The 16 draft ids t2d of a lane's elements x0 .. x0+15 (x0 = c*1024 + lane*16; -1 past v_t).
__device__ __forceinline__ void load_x(const TliVerifyArgs &a, int x0, bool vec, int32_t (&xs)[16]) {
    if (vec && x0 + 16 <= a.v_t) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int4 t = *reinterpret_cast<const int4 *>(a.t2d + x0 + 4 * q);
            xs[4 * q] = t.x;
            xs[4 * q + 1] = t.y;
            xs[4 * q + 2] = t.z;
            xs[4 * q + 3] = t.w;
        }
    } else {
#pragma unroll
        for (int k = 0; k < 16; ++k) xs[k] = x0 + k < a.v_t ? a.t2d[x0 + k] : -1;
    }
}

// Their target probabilities (0 past v_t) and ids (the sampler's crossing chunk, in position order).
__device__ __forceinline__ void load_px(const TliVerifyArgs &a, const float *prow, int x0, bool vec, float (&pv)[16],
                                        int32_t (&xs)[16]) {
    vcore::read16(prow, x0, a.v_t, vec, pv);
    load_x(a, x0, vec, xs);
}

// The draft masses q(x) at the 16 ids (0 for an id outside [0, v_d), or without a draft row).
// Only the lanes that keep an id load (the intersection is often a small part of V_t).
__device__ __forceinline__ void gather16(const TliVerifyArgs &a, const float *drow, const int32_t (&xs)[16],
                                         float (&gv)[16]) {
#pragma unroll
    for (int k = 0; k < 16; ++k) gv[k] = (drow != nullptr && xs[k] >= 0 && xs[k] < a.v_d) ? drow[xs[k]] : 0.0f;
}

// Q62 residual entries q62(clamp01(p - q')) of the 16 elements (q' = qprime(g, S); 0 past v_t,
// where p = g = 0).
__device__ __forceinline__ uint64_t residual16(const float (&pv)[16], const float (&gv)[16], float S, int x0, int vt,
                                               uint64_t (&qv)[16]) {
    uint64_t sum = 0;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        qv[k] = x0 + k < vt ? q62(clamp01(pv[k] - qprime(gv[k], S))) : 0ull;
        sum += qv[k];
    }
    return sum;
}

// The row pass in vcore::load_chunk's element order (lane l holds elements 256 u + 4 l + j of a
// chunk, so each 16-byte load instruction covers 1 KB of the row): the target probabilities
// with the non-temporal hint, the 16 ids t2d in the same order (-1 past v_t).
__device__ __forceinline__ void load_px_strided(const TliVerifyArgs &a, const float *prow, int c, bool vec,
                                                float4 (&pv)[4], int32_t (&xs)[16]) {
    const int lane = threadIdx.x % kWave;
    const int xb = c * vcore::kChunk;
    vcore::load_chunk(prow, xb, lane, a.v_t, vec, pv);
    if (vec && xb + vcore::kChunk <= a.v_t) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int4 t = *reinterpret_cast<const int4 *>(a.t2d + xb + u * 256 + lane * 4);
            xs[4 * u] = t.x;
            xs[4 * u + 1] = t.y;
            xs[4 * u + 2] = t.z;
            xs[4 * u + 3] = t.w;
        }
    } else {
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            const int y = xb + (k >> 2) * 256 + lane * 4 + (k & 3);
            xs[k] = y < a.v_t ? a.t2d[y] : -1;
        }
    }
}

// Q62 sum of the 16 residual entries in that order (p = g = 0 past v_t gives 0).
__device__ __forceinline__ uint64_t residual_sum_strided(const float4 (&pv)[4], const float (&gv)[16], float S) {
    uint64_t sum = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        sum += q62(clamp01(pv[u].x - qprime(gv[4 * u], S))) + q62(clamp01(pv[u].y - qprime(gv[4 * u + 1], S))) +
               q62(clamp01(pv[u].z - qprime(gv[4 * u + 2], S))) + q62(clamp01(pv[u].w - qprime(gv[4 * u + 3], S)));
    }
    return sum;
}

__global__ void __launch_bounds__(kThreads) verify_tli_row(TliVerifyParams p) {
    const TliVerifyArgs &a = p.a;
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    extern __shared__ uint64_t sh_part[];  // nc chunk sums (Q62)
    __shared__ U128 sh_red[kWaves];
    __shared__ float sh_S, sh_Sr;
    __shared__ int sh_ok, sh_gamma, sh_ctr, sh_rej;

    TT_STAMP(0);
    const int t0 = a.target_off[b];
    const int M = a.target_off[b + 1] - t0;
    if (!(M >= 0 && M <= a.max_m)) {
        if (tid == 0) {
            a.n_accepted[b] = -1;
            a.out_token[b] = -1;
        }
        return;
    }
    if (wave == kWaves - 1) {  // every proposal's id inside the target vocabulary
        bool ok = true;
        for (int base = 0; ok && base < M; base += kWave) {
            const int j = base + lane;
            ok = !__any(j < M && (a.target_ids[t0 + j] < 0 || a.target_ids[t0 + j] >= a.v_t));
        }
        if (lane == 0) {
            sh_ok = ok ? 1 : 0;
            sh_ctr = kWaves;
        }
    }
    int gamma = M;
    float S_r = 0.0f;
    if (a.draft_mass != nullptr) {
        if (wave == 0) {
            for (int base = 0; base < M && gamma == M; base += kWave) {
                const int j = base + lane;
                bool rej = false;
                float Sj = 0.0f;
                if (j < M) {
                    const int tok = a.target_ids[t0 + j];
                    const float uj = a.u_accept[t0 + j];
                    Sj = a.draft_mass[t0 + j];
                    if (tok >= 0 && tok < a.v_t) {
                        const float pt = a.target_probs[(int64_t)(t0 + b + j) * a.target_ld + tok];
                        const int32_t x = a.t2d[tok];
                        const float g = (x >= 0 && x < a.v_d) ? a.draft_probs[(int64_t)(t0 + j) * a.draft_ld + x] : 0.0f;
                        const float qj = qprime(g, Sj);
                        rej = !((qj <= 0.0f) || (uj < pt / qj));
                    }
                }
                const unsigned long long rm = __ballot(rej);
                if (rm != 0ull) {
                    const int l = __ffsll(rm) - 1;
                    gamma = base + l;
                    S_r = __shfl(Sj, l);
                }
            }
            if (lane == 0) {
                sh_gamma = gamma;
                sh_Sr = S_r;
            }
        }
        __syncthreads();
        if (!sh_ok) {
            if (tid == 0) {
                a.n_accepted[b] = -1;
                a.out_token[b] = -1;
            }
            return;
        }
        gamma = sh_gamma;
        S_r = sh_Sr;
    } else {
        __syncthreads();
        if (!sh_ok) {
            if (tid == 0) {
                a.n_accepted[b] = -1;
                a.out_token[b] = -1;
            }
            return;
        }
        for (int j = 0; j < M; ++j) {  // S_j of each tested row, formed as tt_tli_proposal forms it
            const float *drow = a.draft_probs + (int64_t)(t0 + j) * a.draft_ld;
            const float Sj = row_mass(drow, a.d2t, a.v_d, p.vec_d != 0, sh_red, &sh_S);
            if (tid == 0) {
                const int tok = a.target_ids[t0 + j];
                const float pt = a.target_probs[(int64_t)(t0 + b + j) * a.target_ld + tok];
                const int32_t x = a.t2d[tok];
                const float g = (x >= 0 && x < a.v_d) ? drow[x] : 0.0f;
                const float qj = qprime(g, Sj);
                sh_rej = !((qj <= 0.0f) || (a.u_accept[t0 + j] < pt / qj)) ? 1 : 0;
            }
            __syncthreads();
            if (sh_rej) {
                gamma = j;
                S_r = Sj;
                break;
            }
        }
    }
    TT_STAMP(1);
    // residual (or bonus) row: Q62 chunk sums of max(0, p - q') into LDS
    const bool vec = p.vec_t != 0;
    const float *prow = a.target_probs + (int64_t)(t0 + b + gamma) * a.target_ld;
    const float *drow = gamma < M ? a.draft_probs + (int64_t)(t0 + gamma) * a.draft_ld : nullptr;
    const int nc = p.nc;
    {
        // each wave: chunk c's probabilities and draft masses, chunk cn's probabilities and ids
        // in flight behind them (a chunk's gathers wait for its ids only)
        float4 pv[4], pn[4];
        float gv[16];
        int32_t xs[16];
        int c = wave, cn = nc;
        if (c < nc) {
            load_px_strided(a, prow, c, vec, pv, xs);
            gather16(a, drow, xs, gv);
            cn = vcore::next_chunk(&sh_ctr, c, kWaves);
            if (cn < nc) load_px_strided(a, prow, cn, vec, pn, xs);
        }
        while (c < nc) {
            uint64_t acc = residual_sum_strided(pv, gv, S_r);
            acc = vcore::wave_total(acc);
            if (lane == kWave - 1) sh_part[c] = acc;
            c = cn;
            if (c < nc) {
#pragma unroll
                for (int u = 0; u < 4; ++u) pv[u] = pn[u];
                gather16(a, drow, xs, gv);
                cn = vcore::next_chunk(&sh_ctr, c, kWaves);
                if (cn < nc) load_px_strided(a, prow, cn, vec, pn, xs);
            }
        }
    }
    if (wave < 12) TT_STAMP_WAVE(4 + wave);
    __syncthreads();
    TT_STAMP(2);
    if (wave != 0) return;
    uint64_t Z, T, base;
    int cs;
    const int st = vcore::find_crossing(nc, [&](int c) { return sh_part[c]; }, a.u_sample[b], Z, T, cs, base);
    int token;
    if (st == 1) {
        token = vcore::wave_first_argmax(prow, a.v_t);
    } else if (st == 2) {
        token = a.v_t - 1;
    } else {
        const int x0 = cs * vcore::kChunk + lane * 16;
        float pv[16], gv[16];
        int32_t xs[16];
        load_px(a, prow, x0, vec, pv, xs);
        gather16(a, drow, xs, gv);
        uint64_t qv[16];
        const uint64_t sum = residual16(pv, gv, S_r, x0, a.v_t, qv);
        const uint64_t lincl = vcore::wave_inclusive_scan(sum) + base;
        const uint64_t lexcl = lincl - sum;
        const unsigned long long lhit = __ballot(lexcl <= T && T < lincl);
        if (lhit == 0ull) {
            token = a.v_t - 1;
        } else {
            const int tl = __ffsll(lhit) - 1;
            uint64_t run = lexcl;
            int k_at = 0;
#pragma unroll
            for (int k = 0; k < 16; ++k) {
                run += qv[k];
                k_at += run <= T ? 1 : 0;
            }
            token = __builtin_amdgcn_readlane(x0 + k_at, tl);
        }
    }
    if (lane == 0) {
        a.n_accepted[b] = gamma;
        a.out_token[b] = token;
    }
    TT_STAMP(3);
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

int launch_verify_tli(const TliVerifyArgs &a, hipStream_t stream) {
    if (a.n_streams == 0) return TT_OK;
    TliVerifyParams p;
    p.a = a;
    p.nc = (a.v_t + vcore::kChunk - 1) / vcore::kChunk;
    p.vec_t = aligned16(a.target_probs) && aligned16(a.t2d) && a.target_ld % 4 == 0;
    p.vec_d = aligned16(a.draft_probs) && aligned16(a.d2t) && a.draft_ld % 4 == 0;
    hipLaunchKernelGGL(verify_tli_row, dim3(a.n_streams), dim3(kThreads), 8 * (size_t)p.nc, stream, p);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

}  // namespace tt
