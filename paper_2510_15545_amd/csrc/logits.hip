// Verification from bf16 target logits with a temperature on gfx950: the target softmax of
// Sec. 3's acceptance rule and App. D Alg. 4's residual is formed inside the verification
// (App. F lists the sampling temperatures), so the caller never materialises fp32
// probability rows.
//
// Arithmetic (every step specified, so any summation order gives the same token):
//   x      = fp32(bf16 logit) * inv_temp; NaN counts as minus infinity
//   m      = max x over the row
//   e(x)   = sexp(x - m): Cody-Waite reduction x = k ln2 + r (k = rint(x log2 e), r by two
//            fused multiply-adds), the degree-6 Taylor polynomial of exp(r) by Horner's
//            rule with fused multiply-adds, scaling by 2^k; 0 below -87
//   e39    = floor(e * 2^39), summed exactly in 64 bits (rows of at most 2^23 entries)
//   S      = sum * 2^-39 rounded once to the nearest fp32 (ties to even)
//   P(t_j) = e(t_j) / S; accept while q_j <= 0 or u_j < P(t_j) / q_j
//   after a rejection at r the entry t_r of the residual is
//            floor(clamp(e(t_r) - q_r S, 0, 1) * 2^39), proportional to max(0, P - q_r e_t);
//            after full acceptance the bonus row's e39 is sampled as is
//   token  = first index whose prefix exceeds floor(u * Z); first largest x when Z = 0.
//
// One 1024-thread workgroup per stream walks its rows 0, 1, ... until the first rejection
// (each row: a max pass, then a pass of chunk sums into LDS -- the second read mostly from
// the caches), then wave 0 samples: the chunk sums lane-blocked, the crossing chunk's
// e39 recomputed from its 1024 logits.  A lane reads 16 consecutive bf16 (two 16-byte loads).
#include "verify_core.h"

namespace tt {
namespace {

using vcore::exact_threshold;
using vcore::lane_value;
using vcore::wave_inclusive_scan;

constexpr int kThreads = 1024;
constexpr int kWave = 64;
constexpr int kWaves = kThreads / kWave;
constexpr int kChunk = 1024;  // logits per chunk: one wave, 16 per lane

__device__ __forceinline__ float bf16_value(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

// exp(x) for x <= 0 as specified above (0 for x < -87 and NaN)
__device__ __forceinline__ float sexp(float x) {
    if (!(x >= -87.0f)) return 0.0f;
    const float kf = rintf(x * 0x1.715476p+0f);
    float r = fmaf(-kf, 0x1.62e430p-1f, x);
    r = fmaf(-kf, -0x1.05c610p-29f, r);
    float p = 0x1.6c16c2p-10f;
    p = fmaf(p, r, 0x1.111112p-7f);
    p = fmaf(p, r, 0x1.555556p-5f);
    p = fmaf(p, r, 0x1.555556p-3f);
    p = fmaf(p, r, 0.5f);
    p = fmaf(p, r, 1.0f);
    p = fmaf(p, r, 1.0f);
    return ldexpf(p, (int)kf);
}

// floor(e * 2^39) for e in [0, 1] (exact: the high word is trunc(e * 2^7), the low word the
// remainder scaled by 2^32)
__device__ __forceinline__ uint64_t q39(float e) {
    const float s = e * 128.0f;
    const uint32_t hi = (uint32_t)s;
    const uint32_t lo = (uint32_t)((s - (float)hi) * 4294967296.0f);
    return ((uint64_t)hi << 32) | lo;
}

// n * 2^-39 rounded to the nearest fp32, ties to even
__device__ inline float q39_to_f32(uint64_t n) {
    if (n == 0) return 0.0f;
    const int bl = 64 - __clzll(n);
    if (bl <= 24) return ldexpf((float)n, -39);
    const int sh = bl - 24;
    uint64_t mant = n >> sh;
    const uint64_t rem = n & ((1ull << sh) - 1), half = 1ull << (sh - 1);
    if (rem > half || (rem == half && (mant & 1u))) ++mant;
    return ldexpf((float)mant, sh - 39);
}

__device__ __forceinline__ float scaled(uint32_t bits16, float it) {
    const float x = bf16_value(bits16) * it;
    return x == x ? x : -INFINITY;
}

// The 16 logits of a lane in chunk c (elements c*1024 + lane*16 + k, zero bits past v).
__device__ __forceinline__ void load16(const uint16_t *row, int x0, int v, bool vec, uint32_t (&w)[8]) {
    if (vec && x0 + 16 <= v) {
        const uint4 a = *reinterpret_cast<const uint4 *>(row + x0);
        const uint4 b = *reinterpret_cast<const uint4 *>(row + x0 + 8);
        w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
        w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
    } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const uint32_t lo = x0 + 2 * k < v ? row[x0 + 2 * k] : 0u;
            const uint32_t hi = x0 + 2 * k + 1 < v ? row[x0 + 2 * k + 1] : 0u;
            w[k] = lo | (hi << 16);
        }
    }
}

// bf16 element k (0..15) of a lane's 16
__device__ __forceinline__ uint32_t elem(const uint32_t (&w)[8], int k) {
    return (k & 1) ? (w[k >> 1] >> 16) : (w[k >> 1] & 0xFFFFu);
}

struct LogitsParams {
    LogitsArgs a;
    int32_t nc, vec;
};

__global__ void __launch_bounds__(kThreads) verify_logits_row(LogitsParams p) {
    const LogitsArgs &a = p.a;
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    extern __shared__ uint64_t sh_part[];  // nc chunk sums of e39
    __shared__ float sh_red[kWaves];
    __shared__ int sh_ok;
    __shared__ float sh_m;
    __shared__ int sh_next;  // 1: accepted, go to the next row
    __shared__ uint64_t sh_Z;
    __shared__ int sh_t;
    __shared__ float sh_rt;

    const int t0 = a.target_off[b];
    const int M = a.target_off[b + 1] - t0;
    const float it = a.inv_temp[b];
    const int v = a.v_t, nc = p.nc;
    const bool vec = p.vec != 0;
    if (wave == 0) {
        bool ok = M >= 0 && M <= a.max_m && it > 0.0f;
        for (int base = 0; ok && base < M; base += kWave) {
            const int j = base + lane;
            const bool bad = j < M && (a.target_ids[t0 + j] < 0 || a.target_ids[t0 + j] >= v);
            ok = !__any(bad);
        }
        if (lane == 0) sh_ok = ok ? 1 : 0;
    }
    __syncthreads();
    if (!sh_ok) {
        if (tid == 0) {
            a.n_accepted[b] = -1;
            a.out_token[b] = -1;
        }
        return;
    }
    for (int j = 0; j <= M; ++j) {
        const uint16_t *row = a.logits + (int64_t)(t0 + b + j) * a.ld;
        // pass 1: the row's largest x
        float m = -INFINITY;
        for (int c = wave; c < nc; c += kWaves) {
            uint32_t w[8];
            const int x0 = c * kChunk + lane * 16;
            load16(row, x0, v, vec, w);
#pragma unroll
            for (int k = 0; k < 16; ++k)
                if (x0 + k < v) m = fmaxf(m, scaled(elem(w, k), it));
        }
        for (int off = kWave / 2; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
        if (lane == 0) sh_red[wave] = m;
        __syncthreads();
        if (tid == 0) {
            float mm = -INFINITY;
            for (int k = 0; k < kWaves; ++k) mm = fmaxf(mm, sh_red[k]);
            sh_m = mm;
        }
        __syncthreads();
        m = sh_m;
        // pass 2: chunk sums of e39
        for (int c = wave; c < nc; c += kWaves) {
            uint32_t w[8];
            const int x0 = c * kChunk + lane * 16;
            load16(row, x0, v, vec, w);
            uint64_t acc = 0;
#pragma unroll
            for (int k = 0; k < 16; ++k)
                acc += x0 + k < v ? q39(sexp(scaled(elem(w, k), it) - m)) : 0ull;
            acc = wave_inclusive_scan(acc);
            if (lane == kWave - 1) sh_part[c] = acc;
        }
        __syncthreads();
        // S, the acceptance test of position j, and the residual's entry at t_j
        if (wave == 0) {
            uint64_t local = 0;
            for (int c = lane; c < nc; c += kWave) local += sh_part[c];
            const uint64_t Sq = lane_value(wave_inclusive_scan(local), kWave - 1);
            if (lane == 0) {
                const float S = q39_to_f32(Sq);
                int next = 0;
                uint64_t Z = Sq;
                int t = -1;
                float et = 0.0f, rt = 0.0f;
                if (j < M) {
                    t = a.target_ids[t0 + j];
                    const float qj = a.q[t0 + j];
                    et = sexp(scaled(row[t], it) - m);
                    const float P = et / S;
                    if (qj <= 0.0f || a.u_accept[t0 + j] < P / qj) {
                        next = 1;
                    } else {
                        rt = fminf(fmaxf(et - qj * S, 0.0f), 1.0f);  // NaN -> 0
                        const uint64_t before = q39(et), after = q39(rt);
                        Z = Sq - before + after;
                        sh_part[t / kChunk] = sh_part[t / kChunk] - before + after;
                    }
                }
                sh_next = next;
                sh_Z = Z;
                sh_t = next ? -1 : t;
                sh_rt = rt;
            }
        }
        __syncthreads();
        if (sh_next) continue;
        // sample row j (wave 0)
        if (wave == 0) {
            const uint64_t Z = sh_Z;
            const int t = sh_t;
            int token = 0;
            if (Z == 0) {  // no mass: the first largest x
                float bv = -INFINITY;
                int bi = INT_MAX;
                for (int x = lane; x < v; x += kWave) {
                    const float xv = scaled(row[x], it);
                    if (xv > bv) {
                        bv = xv;
                        bi = x;
                    }
                }
                for (int off = kWave / 2; off > 0; off >>= 1) {
                    const float ov = __shfl_xor(bv, off);
                    const int oi = __shfl_xor(bi, off);
                    if (ov > bv || (ov == bv && oi < bi)) {
                        bv = ov;
                        bi = oi;
                    }
                }
                token = bi == INT_MAX ? 0 : bi;
            } else {
                const uint64_t T = exact_threshold(a.u_sample[b], Z);
                // chunk sums lane-blocked: lane l holds chunks [l*per, (l+1)*per)
                const int per = (nc + kWave - 1) / kWave;
                const int ca = lane * per < nc ? lane * per : nc;
                const int cb = ca + per < nc ? ca + per : nc;
                uint64_t local = 0;
                for (int c = ca; c < cb; ++c) local += sh_part[c];
                const uint64_t incl = wave_inclusive_scan(local);
                const uint64_t excl = incl - local;
                const unsigned long long hit = __ballot(excl <= T && T < incl);
                int cs = 0;
                uint64_t base = 0;
                if (hit != 0ull) {
                    const int owner = __ffsll(hit) - 1;
                    if (lane == owner) {
                        uint64_t run = excl;
                        cs = ca;
                        base = excl;
                        for (int c = ca; c < cb; ++c) {
                            const uint64_t nx = run + sh_part[c];
                            if (nx > T) break;
                            cs = c + 1;
                            base = nx;
                            run = nx;
                        }
                    }
                    cs = __builtin_amdgcn_readlane(cs, owner);
                    base = lane_value(base, owner);
                    // the crossing chunk: lane holds elements cs*1024 + lane*16 + [0, 16)
                    const int x0 = cs * kChunk + lane * 16;
                    uint32_t w[8];
                    load16(row, x0, v, vec, w);
                    const float mm = sh_m;
                    const uint64_t adj = q39(sh_rt);
                    uint64_t qv[16];
                    uint64_t sum = 0;
#pragma unroll
                    for (int k = 0; k < 16; ++k) {
                        uint64_t e = x0 + k < v ? q39(sexp(scaled(elem(w, k), it) - mm)) : 0ull;
                        if (x0 + k == t) e = adj;
                        qv[k] = e;
                        sum += e;
                    }
                    const uint64_t lincl = wave_inclusive_scan(sum) + base;
                    const uint64_t lexcl = lincl - sum;
                    const unsigned long long lhit = __ballot(lexcl <= T && T < lincl);
                    if (lhit != 0ull) {
                        const int tl = __ffsll(lhit) - 1;
                        uint64_t run = lexcl;
                        int k_at = 0;
#pragma unroll
                        for (int k = 0; k < 16; ++k) {
                            run += qv[k];
                            k_at += run <= T ? 1 : 0;
                        }
                        token = __builtin_amdgcn_readlane(x0 + k_at, tl);
                    } else {
                        token = v - 1;
                    }
                } else {
                    token = v - 1;  // only if the sums wrapped (rows longer than allowed)
                }
            }
            if (lane == 0) {
                a.n_accepted[b] = j;
                a.out_token[b] = token;
            }
        }
        return;
    }
}

}  // namespace

int launch_verify_logits(const LogitsArgs &a, hipStream_t stream) {
    if (a.n_streams == 0) return TT_OK;
    LogitsParams p;
    p.a = a;
    p.nc = (a.v_t + kChunk - 1) / kChunk;
    p.vec = ((reinterpret_cast<uintptr_t>(a.logits) & 15u) == 0 && (a.ld % 8) == 0) ? 1 : 0;
    hipLaunchKernelGGL(verify_logits_row, dim3(a.n_streams), dim3(kThreads), 8 * (size_t)p.nc, stream, p);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

}  // namespace tt
