// Vocabulary-wide lossless speculative sampling on gfx950.
//
// Per stream b (Sec. 3 "Standard Speculative Sampling", Sec. 4.2.2-4.2.3, App. D Alg. 4):
//   gamma  = number of leading proposals with u_j < P_t(t_j) / q_j (fp32), first rejection stops
//   r      = gamma; R(x) = max(0, P_t[r](x) - q_r [x == t_r]) if r < M, else P_t[M](x)
//   token  = inverse-CDF sample of R with the uniform u_sample[b]
//
// The row of stream b is read once from HBM.  It is cut into chunks of 1024 floats
// (one wave, 16 floats per lane, 16-byte loads).  Each chunk's residual mass is
// accumulated in exact Q62 fixed point (R quantised by truncation), so chunk sums and
// their prefix are independent of summation order and the sampled token is
// bit-identical to a sequential scan.  Sampling forms Z and T = floor(u * Z) exactly,
// scans the chunk sums to the crossing chunk, re-reads that one chunk (4 KiB) and
// scans it to the crossing index.  Row loads carry the non-temporal hint: every row
// is read once, and for 256 rows of 151,936 floats that cut the kernel from 34.6 to
// 30.6 us against ordinary loads.
//
// Two launch shapes:
//   row path    (at least one stream per CU): one 1024-thread workgroup per stream
//               runs the acceptance scan once, streams its whole row with 16 waves,
//               keeps the chunk sums in LDS and one wave samples.  One kernel.
//   split path  (fewer streams): verify_stream over B x S workgroups (every workgroup
//               of a stream recomputes gamma, streams its share of the row and stores
//               chunk sums), then verify_sample with one wave per stream.  The kernel
//               boundary publishes the chunk sums: an in-kernel hand-off between
//               workgroups needs an agent-scope release, which on gfx950 writes back
//               the XCD's whole L2 (one per workgroup made the kernel 5-10x slower).
// Sampling runs in one wave with DPP prefix sums and no LDS or barriers.
// In the split path workgroup id -> (stream, split) is XCD-aware: the hardware deals
// workgroup ids round-robin over the 8 XCDs, so XCD x receives the contiguous work range
// [x * G/8, (x+1) * G/8) and a stream's splits share one XCD.
#include <climits>
#include <cmath>

#include "tt_internal.h"

#ifndef TT_VERIFY_TARGET_WG
#define TT_VERIFY_TARGET_WG 2048  // split path: workgroups to aim for
#endif
#ifndef TT_VERIFY_ROW_MIN_STREAMS
#define TT_VERIFY_ROW_MIN_STREAMS 256  // row path from this many streams up
#endif
#ifndef TT_VERIFY_PREFETCH
#define TT_VERIFY_PREFETCH 1  // chunks each wave keeps in flight ahead of the one it sums
#endif
#ifndef TT_VERIFY_NT_LOADS
#define TT_VERIFY_NT_LOADS 1  // row loads carry the non-temporal hint (0: ordinary loads)
#endif

namespace tt {
namespace {

constexpr int kWave = 64;
constexpr int kSplitThreads = 256;
constexpr int kRowThreads = 1024;
constexpr int kChunk = 1024;
constexpr int kXcds = 8;

struct VParams {
    VerifyArgs a;
    uint64_t *zsum;
    int32_t *rsel;
    uint64_t *partials;
    int32_t nc, splits, cpw, work_items, vec4;
};

__device__ __forceinline__ float clamp01(float x) { return fminf(fmaxf(x, 0.0f), 1.0f); }

// floor(r * 2^62) for r in [0, 1]: the high word is trunc(r * 2^30), the low word the
// fraction of r * 2^30 scaled by 2^32 and truncated (every step is exact in fp32).
__device__ __forceinline__ uint64_t q62(float r) {
    const float s = r * 0x1p30f;
    const uint32_t hi = (uint32_t)s;
    const uint32_t lo = (uint32_t)(__builtin_amdgcn_fractf(s) * 0x1p32f);
    return ((uint64_t)hi << 32) | (uint64_t)lo;
}

// floor(u * Z) exactly: u = mant * 2^-sh from its IEEE fields, 128-bit product.
__device__ __forceinline__ uint64_t exact_threshold(float u, uint64_t Z) {
    if (!(u > 0.0f)) return 0;
    if (u >= 1.0f) return Z - 1;
    const uint32_t bits = __float_as_uint(u);
    const uint32_t e = (bits >> 23) & 0xFFu;
    uint64_t m = bits & 0x7FFFFFu;
    int sh;
    if (e == 0) {
        sh = 149;
    } else {
        m |= 0x800000u;
        sh = 150 - (int)e;  // >= 24 because u < 1
    }
    if (sh >= 128) return 0;
    const uint64_t lo = m * Z;
    const uint64_t hi = __umul64hi(m, Z);
    const uint64_t T = (sh >= 64) ? (hi >> (sh - 64)) : ((lo >> sh) | (hi << (64 - sh)));
    return T < Z ? T : Z - 1;
}

// v + (v shifted across lanes by a DPP control); lanes without a source add 0.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint64_t dpp_add(uint64_t v) {
    const uint32_t lo = __builtin_amdgcn_update_dpp(0u, (uint32_t)v, CTRL, ROW_MASK, 0xF, true);
    const uint32_t hi = __builtin_amdgcn_update_dpp(0u, (uint32_t)(v >> 32), CTRL, ROW_MASK, 0xF, true);
    return v + (((uint64_t)hi << 32) | lo);
}

// Inclusive prefix sum over the 64 lanes (prefix sums inside each row of 16 lanes, then
// row broadcasts); lane 63 holds the total.
__device__ __forceinline__ uint64_t wave_inclusive_scan(uint64_t v) {
    v = dpp_add<0x111, 0xF>(v);  // row_shr:1
    v = dpp_add<0x112, 0xF>(v);  // row_shr:2
    v = dpp_add<0x114, 0xF>(v);  // row_shr:4
    v = dpp_add<0x118, 0xF>(v);  // row_shr:8
    v = dpp_add<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
    v = dpp_add<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
    return v;
}

__device__ __forceinline__ uint64_t lane_value(uint64_t v, int lane) {
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, lane);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}

// First index of the maximum over the row (NaN never wins); 0 if nothing exceeds -inf.
// One wave.
__device__ int wave_first_argmax(const float *row, int vt) {
    const int lane = threadIdx.x % kWave;
    float bv = -INFINITY;
    int bi = INT_MAX;
    for (int x = lane; x < vt; x += kWave) {
        const float v = row[x];
        if (v > bv) {
            bv = v;
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
    return bi == INT_MAX ? 0 : bi;
}

// Acceptance scan by one wave: gamma (first rejection, else M); false if the stream is
// invalid (M outside [0, max_m] or an id outside [0, v_t)).
__device__ __forceinline__ bool accept_scan(const VerifyArgs &a, int b, int t0, int M, int lane, int &gamma) {
    gamma = M;
    if (M < 0 || M > a.max_m) return false;
    for (int base = 0; base < M; base += kWave) {
        const int j = base + lane;
        bool bad = false, rej = false;
        if (j < M) {
            const int tok = a.target_ids[t0 + j];
            if (tok < 0 || tok >= a.v_t) {
                bad = true;
            } else {
                const float pt = a.target_probs[(int64_t)(t0 + b + j) * a.target_ld + tok];
                const float qj = a.q[t0 + j];
                const float ratio = pt / qj;
                rej = !((qj <= 0.0f) || (a.u_accept[t0 + j] < ratio));
            }
        }
        if (__any(bad)) return false;
        const unsigned long long rm = __ballot(rej);
        if (rm != 0ull && gamma == M) gamma = base + __ffsll(rm) - 1;
    }
    return true;
}

// The four 16-byte loads of one lane for chunk starting at xb (guarded at the row end).
__device__ __forceinline__ void load_chunk(const float *row, int xb, int lane, int vt, bool vec, float4 (&v)[4]) {
    if (vec && xb + kChunk <= vt) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const float4 *src = reinterpret_cast<const float4 *>(row + xb + u * 256 + lane * 4);
#if TT_VERIFY_NT_LOADS
            typedef float f4v __attribute__((ext_vector_type(4)));
            const f4v t = __builtin_nontemporal_load(reinterpret_cast<const f4v *>(src));
            v[u] = make_float4(t.x, t.y, t.z, t.w);
#else
            v[u] = *src;
#endif
        }
    } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int x = xb + u * 256 + lane * 4;
            v[u].x = x < vt ? row[x] : 0.0f;
            v[u].y = x + 1 < vt ? row[x + 1] : 0.0f;
            v[u].z = x + 2 < vt ? row[x + 2] : 0.0f;
            v[u].w = x + 3 < vt ? row[x + 3] : 0.0f;
        }
    }
}

// Q62 sums of chunks c0 + wave, c0 + wave + stride, ... < c1 (one chunk ahead in flight);
// lane 63 hands each sum to store(c, sum).
template <class Store>
__device__ __forceinline__ void sum_chunk(const float4 (&v)[4], const float *row, int c, int rtok, float rq,
                                          Store &store) {
    const int lane = threadIdx.x % kWave;
    uint64_t acc = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u)
        acc += q62(clamp01(v[u].x)) + q62(clamp01(v[u].y)) + q62(clamp01(v[u].z)) + q62(clamp01(v[u].w));
    acc = wave_inclusive_scan(acc);
    if (lane == kWave - 1) {
        const int xb = c * kChunk;
        if (rtok >= xb && rtok < xb + kChunk) {  // the rejected proposal loses q_r of its mass
            const float pr = row[rtok];
            acc += q62(clamp01(pr - rq)) - q62(clamp01(pr));
        }
        store(c, acc);
    }
}

// Q62 sums of chunks c0 + wave, c0 + wave + stride, ... < c1, with TT_VERIFY_PREFETCH
// chunks in flight ahead of the one being summed; lane 63 hands each sum to store(c, sum).
template <class Store>
__device__ __forceinline__ void stream_chunks(const float *row, int vt, bool vec, int c0, int c1, int stride,
                                              int rtok, float rq, Store store) {
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    int c = c0 + wave;
#if TT_VERIFY_PREFETCH >= 2
    float4 v0[4], v1[4], v2[4];
    if (c < c1) load_chunk(row, c * kChunk, lane, vt, vec, v0);
    if (c + stride < c1) load_chunk(row, (c + stride) * kChunk, lane, vt, vec, v1);
    for (; c < c1; c += stride) {
        if (c + 2 * stride < c1) load_chunk(row, (c + 2 * stride) * kChunk, lane, vt, vec, v2);
        sum_chunk(v0, row, c, rtok, rq, store);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            v0[u] = v1[u];
            v1[u] = v2[u];
        }
    }
#else
    float4 v[4], nx[4];
    if (c < c1) load_chunk(row, c * kChunk, lane, vt, vec, v);
    for (; c < c1; c += stride) {
        const int cn = c + stride;
        if (cn < c1) load_chunk(row, cn * kChunk, lane, vt, vec, nx);
        sum_chunk(v, row, c, rtok, rq, store);
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = nx[u];
    }
#endif
}

// Inverse-CDF sample of the row from its nc chunk sums part(c), by one wave: every lane
// returns the token and *Zout the Q62 mass.  Chunk sums are scanned lane-blocked, the
// crossing chunk is re-read as 16 consecutive floats per lane and scanned the same way.
template <class Part>
__device__ int wave_sample(const float *row, int vt, int nc, Part part, float u, int rtok, float rq,
                           uint64_t *Zout) {
    const int lane = threadIdx.x % kWave;
    const int per = (nc + kWave - 1) / kWave;
    const int ca = lane * per < nc ? lane * per : nc;
    const int cb = ca + per < nc ? ca + per : nc;
    uint64_t local = 0;
    for (int c = ca; c < cb; ++c) local += part(c);
    const uint64_t incl = wave_inclusive_scan(local);
    const uint64_t Z = lane_value(incl, kWave - 1);
    *Zout = Z;
    if (Z == 0) return wave_first_argmax(row, vt);
    const uint64_t T = exact_threshold(u, Z);
    // lane whose block of chunks holds the crossing, then the chunk inside it
    const uint64_t excl = incl - local;
    const unsigned long long hit = __ballot(excl <= T && T < incl);
    if (hit == 0ull) return vt - 1;  // only if the Q62 mass wrapped (not a probability row)
    const int owner = __ffsll(hit) - 1;
    int cs = nc;
    uint64_t base = 0;
    if (lane == owner) {
        uint64_t run = excl;
        for (int c = ca; c < cb; ++c) {
            const uint64_t nx = run + part(c);
            if (run <= T && nx > T) {
                cs = c;
                base = run;
                break;
            }
            run = nx;
        }
    }
    cs = __builtin_amdgcn_readlane(cs, owner);
    base = lane_value(base, owner);
    // the crossing chunk: lane holds elements cs*1024 + lane*16 + [0, 16)
    const int x0 = cs * kChunk + lane * 16;
    uint64_t qv[16];
    uint64_t sum = 0;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const int x = x0 + k;
        const float pv = x < vt ? row[x] : 0.0f;
        qv[k] = q62(clamp01(pv - (x == rtok ? rq : 0.0f)));
        sum += qv[k];
    }
    const uint64_t lincl = wave_inclusive_scan(sum) + base;
    const uint64_t lexcl = lincl - sum;
    const unsigned long long lhit = __ballot(lexcl <= T && T < lincl);
    if (lhit == 0ull) return vt - 1;
    const int tl = __ffsll(lhit) - 1;
    int tok = vt - 1;
    if (lane == tl) {
        uint64_t run = lexcl;
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            run += qv[k];
            if (run > T) {
                tok = x0 + k;
                break;
            }
        }
    }
    return __builtin_amdgcn_readlane(tok, tl);
}

// ------------------------------------------------------------------ row path
__global__ void __launch_bounds__(kRowThreads) verify_row(VParams p) {
    const VerifyArgs &a = p.a;
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    extern __shared__ uint64_t sh_part[];  // nc chunk sums
    __shared__ int sh_gamma, sh_ok;

    const int t0 = a.target_off[b];
    const int M = a.target_off[b + 1] - t0;
    const float us = a.u_sample[b];
    if (wave == 0) {
        int gamma;
        const bool ok = accept_scan(a, b, t0, M, lane, gamma);
        if (lane == 0) {
            sh_gamma = gamma;
            sh_ok = ok ? 1 : 0;
        }
    }
    __syncthreads();
    if (!sh_ok) {
        if (tid == 0) {
            a.n_accepted[b] = -1;
            a.out_token[b] = -1;
            p.rsel[b] = -1;
        }
        return;
    }
    const int r = sh_gamma;
    const int vt = a.v_t;
    const float *row = a.target_probs + (int64_t)(t0 + b + r) * a.target_ld;
    const int rtok = r < M ? a.target_ids[t0 + r] : -1;
    const float rq = r < M ? a.q[t0 + r] : 0.0f;
    stream_chunks(row, vt, p.vec4 != 0, 0, p.nc, kRowThreads / kWave, rtok, rq,
                  [&](int c, uint64_t s) { sh_part[c] = s; });
    __syncthreads();
    if (wave != 0) return;
    uint64_t Z;
    const int token = wave_sample(row, vt, p.nc, [&](int c) { return sh_part[c]; }, us, rtok, rq, &Z);
    if (tid == 0) {
        a.n_accepted[b] = r;
        a.out_token[b] = token;
        p.zsum[b] = Z;
        p.rsel[b] = r;
    }
}

// ------------------------------------------------------------------ split path
__global__ void __launch_bounds__(kSplitThreads) verify_stream(VParams p) {
    const VerifyArgs &a = p.a;
    const int G = gridDim.x;
    const int g = blockIdx.x;
    const int work = (g % kXcds) * (G / kXcds) + g / kXcds;
    if (work >= p.work_items) return;
    const int b = work / p.splits, s = work % p.splits;
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    __shared__ int sh_gamma, sh_ok;

    const int t0 = a.target_off[b];
    const int M = a.target_off[b + 1] - t0;
    if (wave == 0) {  // every workgroup of the stream recomputes gamma
        int gamma;
        const bool ok = accept_scan(a, b, t0, M, lane, gamma);
        if (lane == 0) {
            sh_gamma = gamma;
            sh_ok = ok ? 1 : 0;
        }
    }
    __syncthreads();
    if (!sh_ok) {
        if (s == 0 && tid == 0) {
            a.n_accepted[b] = -1;
            a.out_token[b] = -1;
            p.rsel[b] = -1;
        }
        return;
    }
    const int r = sh_gamma;
    if (s == 0 && tid == 0) p.rsel[b] = r;
    const float *row = a.target_probs + (int64_t)(t0 + b + r) * a.target_ld;
    const int rtok = r < M ? a.target_ids[t0 + r] : -1;
    const float rq = r < M ? a.q[t0 + r] : 0.0f;
    const int c0 = s * p.cpw;
    const int c1 = (c0 + p.cpw) < p.nc ? (c0 + p.cpw) : p.nc;
    uint64_t *out = p.partials + (int64_t)b * p.nc;
    stream_chunks(row, a.v_t, p.vec4 != 0, c0, c1, kSplitThreads / kWave, rtok, rq,
                  [&](int c, uint64_t sum) { out[c] = sum; });
}

// One wave per stream: exact threshold, crossing chunk, crossing index.
__global__ void __launch_bounds__(kWave) verify_sample(VParams p) {
    const VerifyArgs &a = p.a;
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const uint64_t *part = p.partials + (int64_t)b * p.nc;
    const int r = p.rsel[b];
    const int t0 = a.target_off[b];
    const int M = a.target_off[b + 1] - t0;
    const float us = a.u_sample[b];
    if (r < 0) return;  // sentinel stream, outputs already written (uniform per workgroup)
    const float *row = a.target_probs + (int64_t)(t0 + b + r) * a.target_ld;
    const int rtok = r < M ? a.target_ids[t0 + r] : -1;
    const float rq = r < M ? a.q[t0 + r] : 0.0f;
    uint64_t Z;
    const int token = wave_sample(row, a.v_t, p.nc, [&](int c) { return part[c]; }, us, rtok, rq, &Z);
    if (tid == 0) {
        a.n_accepted[b] = r;
        a.out_token[b] = token;
        p.zsum[b] = Z;
    }
}

// Optional normalised residual row: res[x] = R(x) / fp32(Z * 2^-62), one-hot when Z = 0.
__global__ void __launch_bounds__(kSplitThreads) residual_write(VParams p, int rsplit) {
    const VerifyArgs &a = p.a;
    const int b = blockIdx.x / rsplit, sidx = blockIdx.x % rsplit;
    if (a.n_accepted[b] < 0) return;
    const int r = p.rsel[b];
    const uint64_t Z = p.zsum[b];
    const int tok = a.out_token[b];
    const int t0 = a.target_off[b];
    const int M = a.target_off[b + 1] - t0;
    const float *row = a.target_probs + (int64_t)(t0 + b + r) * a.target_ld;
    const int rtok = r < M ? a.target_ids[t0 + r] : -1;
    const float rq = r < M ? a.q[t0 + r] : 0.0f;
    float *res = a.residual + (int64_t)b * a.target_ld;
    const int vt = a.v_t;
    const int per = (vt + rsplit - 1) / rsplit;
    const int x0 = sidx * per;
    const int x1 = (x0 + per) < vt ? (x0 + per) : vt;
    if (Z == 0) {
        for (int x = x0 + (int)threadIdx.x; x < x1; x += kSplitThreads) res[x] = (x == tok) ? 1.0f : 0.0f;
        return;
    }
    const float zf = (float)Z * 0x1p-62f;
    for (int x = x0 + (int)threadIdx.x; x < x1; x += kSplitThreads)
        res[x] = clamp01(row[x] - (x == rtok ? rq : 0.0f)) / zf;
}

inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

}  // namespace

VerifyLayout verify_layout(int32_t n_streams, int32_t v_t) {
    VerifyLayout L;
    const size_t n = n_streams > 0 ? (size_t)n_streams : 0;
    L.n_chunks = v_t > 0 ? (int32_t)((v_t + kChunk - 1) / kChunk) : 0;
    size_t off = 0;
    L.zsum = off;
    off = align256(off + 8 * n);
    L.rsel = off;
    off = align256(off + 4 * n);
    L.partials = off;
    off = align256(off + 8 * n * (size_t)L.n_chunks);
    L.total = off;
    return L;
}

int launch_verify(const VerifyArgs &a, hipStream_t stream) {
    const VerifyLayout L = verify_layout(a.n_streams, a.v_t);
    if (a.workspace == nullptr || a.workspace_bytes < L.total) return TT_EWORKSPACE;
    uint8_t *ws = static_cast<uint8_t *>(a.workspace);
    VParams p;
    p.a = a;
    p.zsum = reinterpret_cast<uint64_t *>(ws + L.zsum);
    p.rsel = reinterpret_cast<int32_t *>(ws + L.rsel);
    p.partials = reinterpret_cast<uint64_t *>(ws + L.partials);
    p.nc = L.n_chunks;
    p.vec4 = ((reinterpret_cast<uintptr_t>(a.target_probs) & 15u) == 0 && (a.target_ld % 4) == 0) ? 1 : 0;
    const size_t row_lds = 8 * (size_t)p.nc;
    if (a.n_streams >= TT_VERIFY_ROW_MIN_STREAMS && row_lds <= 64 * 1024) {
        p.splits = 1;
        p.cpw = p.nc;
        p.work_items = a.n_streams;
        hipLaunchKernelGGL(verify_row, dim3(a.n_streams), dim3(kRowThreads), row_lds, stream, p);
        if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
    } else {
        // splits per stream: aim for TT_VERIFY_TARGET_WG workgroups, at least one chunk per wave
        constexpr int kWaves = kSplitThreads / kWave;
        int max_splits = (p.nc + kWaves - 1) / kWaves;
        int splits = (TT_VERIFY_TARGET_WG + a.n_streams - 1) / a.n_streams;
        if (splits > max_splits) splits = max_splits;
        if (splits < 1) splits = 1;
        p.cpw = (p.nc + splits - 1) / splits;
        p.splits = (p.nc + p.cpw - 1) / p.cpw;
        p.work_items = a.n_streams * p.splits;
        const int grid = ((p.work_items + kXcds - 1) / kXcds) * kXcds;
        hipLaunchKernelGGL(verify_stream, dim3(grid), dim3(kSplitThreads), 0, stream, p);
        if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
        hipLaunchKernelGGL(verify_sample, dim3(a.n_streams), dim3(kWave), 0, stream, p);
        if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
    }
    if (a.residual != nullptr) {
        int rsplit = (a.v_t + 8191) / 8192;
        if (rsplit < 1) rsplit = 1;
        hipLaunchKernelGGL(residual_write, dim3(a.n_streams * rsplit), dim3(kSplitThreads), 0, stream, p, rsplit);
        if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
    }
    return TT_OK;
}

}  // namespace tt
