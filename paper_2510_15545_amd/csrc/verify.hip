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
// bit-identical to a sequential scan.
//
// Two kernels, ordered by the stream:
//   verify_stream  grid B x S: every workgroup of stream b recomputes gamma_b (M_b
//                  scalar gathers), then streams its share of row gamma_b and stores one
//                  Q62 sum per chunk.  Split 0 records gamma_b.
//   verify_sample  grid B: forms Z and T = floor(u * Z) exactly, scans the chunk sums to
//                  the crossing chunk, re-reads that one chunk (4 KiB) and scans it to the
//                  crossing index.
// The kernel boundary publishes the chunk sums; an in-kernel hand-off between
// workgroups would need agent-scope fences, which on gfx950 write back and invalidate
// the whole L2 of an XCD.
//
// Workgroup id -> (stream, split) is XCD-aware: the hardware deals workgroup ids
// round-robin over the 8 XCDs, so XCD x receives the contiguous work range
// [x * G/8, (x+1) * G/8) and a stream's splits share one XCD.
#include <climits>
#include <cmath>

#include "tt_internal.h"

namespace tt {
namespace {

constexpr int kWave = 64;
constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kChunk = 1024;
constexpr int kXcds = 8;
constexpr int kTargetWorkgroups = 2048;

struct VParams {
    VerifyArgs a;
    uint64_t *zsum;
    int32_t *rsel;
    uint64_t *partials;
    int32_t nc, splits, cpw, work_items, vec4;
};

__device__ __forceinline__ float clamp01(float x) { return fminf(fmaxf(x, 0.0f), 1.0f); }

// floor(r * 2^62) for r in [0, 1]: the high word is trunc(r * 2^30), the low word the
// truncated fraction scaled by 2^32 (both conversions are exact).
__device__ __forceinline__ uint64_t q62(float r) {
    const float s = r * 0x1p30f;
    const uint32_t hi = (uint32_t)s;
    const float fr = s - (float)hi;
    const uint32_t lo = (uint32_t)(fr * 0x1p32f);
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

// Sum over the wave; the total lands in lane 63 (row prefix sums, then row broadcasts).
__device__ __forceinline__ uint64_t wave_sum_to_last(uint64_t v) {
    v = dpp_add<0x111, 0xF>(v);  // row_shr:1
    v = dpp_add<0x112, 0xF>(v);  // row_shr:2
    v = dpp_add<0x114, 0xF>(v);  // row_shr:4
    v = dpp_add<0x118, 0xF>(v);  // row_shr:8
    v = dpp_add<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
    v = dpp_add<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
    return v;
}

// Exclusive scan over the workgroup in thread order; *total receives the full sum.
__device__ __forceinline__ uint64_t block_exclusive_scan(uint64_t v, uint64_t *total, uint64_t *sh) {
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    uint64_t incl = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const uint64_t n = __shfl_up(incl, off);
        if (lane >= off) incl += n;
    }
    if (lane == kWave - 1) sh[wave] = incl;
    __syncthreads();
    uint64_t wbase = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        const uint64_t s = sh[w];
        if (w < wave) wbase += s;
        tot += s;
    }
    __syncthreads();
    *total = tot;
    return wbase + incl - v;
}

// First index of the maximum (NaN never wins); 0 if no element exceeds -inf.
__device__ int block_first_argmax(const float *row, int vt, float *shv, int *shi) {
    float bv = -INFINITY;
    int bi = INT_MAX;
    for (int x = threadIdx.x; x < vt; x += kThreads) {
        const float v = row[x];
        if (v > bv) {
            bv = v;
            bi = x;
        }
    }
    shv[threadIdx.x] = bv;
    shi[threadIdx.x] = bi;
    __syncthreads();
    for (int w = kThreads / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) {
            const float ov = shv[threadIdx.x + w];
            const int oi = shi[threadIdx.x + w];
            const float mv = shv[threadIdx.x];
            const int mi = shi[threadIdx.x];
            if (ov > mv || (ov == mv && oi < mi)) {
                shv[threadIdx.x] = ov;
                shi[threadIdx.x] = oi;
            }
        }
        __syncthreads();
    }
    const int r = shi[0];
    __syncthreads();
    return r == INT_MAX ? 0 : r;
}

// The four 16-byte loads of one lane for chunk starting at xb (guarded at the row end).
__device__ __forceinline__ void load_chunk(const float *row, int xb, int lane, int vt, bool vec, float4 (&v)[4]) {
    if (vec && xb + kChunk <= vt) {
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const float4 *>(row + xb + u * 256 + lane * 4);
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

__global__ void __launch_bounds__(kThreads) verify_stream(VParams p) {
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

    // ---- phase A: acceptance scan (every workgroup of the stream, redundantly)
    if (wave == 0) {
        bool ok = M >= 0 && M <= a.max_m;
        int gamma = M;
        if (ok) {
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
                if (__any(bad)) {
                    ok = false;
                    break;
                }
                const unsigned long long rm = __ballot(rej);
                if (rm != 0ull && gamma == M) gamma = base + __ffsll(rm) - 1;
            }
        }
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
    const int vt = a.v_t;
    const float *row = a.target_probs + (int64_t)(t0 + b + r) * a.target_ld;
    const int rtok = r < M ? a.target_ids[t0 + r] : -1;
    const float rq = r < M ? a.q[t0 + r] : 0.0f;

    // ---- phase B: stream this workgroup's chunks (one chunk ahead), Q62 chunk sums
    const int c0 = s * p.cpw;
    const int c1 = (c0 + p.cpw) < p.nc ? (c0 + p.cpw) : p.nc;
    const bool vec = p.vec4 != 0;
    float4 v[4], nx[4];
    int c = c0 + wave;
    if (c < c1) load_chunk(row, c * kChunk, lane, vt, vec, v);
    for (; c < c1; c += kWaves) {
        const int cn = c + kWaves;
        if (cn < c1) load_chunk(row, cn * kChunk, lane, vt, vec, nx);
        uint64_t acc = 0;
#pragma unroll
        for (int u = 0; u < 4; ++u)
            acc += q62(clamp01(v[u].x)) + q62(clamp01(v[u].y)) + q62(clamp01(v[u].z)) + q62(clamp01(v[u].w));
        acc = wave_sum_to_last(acc);
        if (lane == kWave - 1) {
            const int xb = c * kChunk;
            if (rtok >= xb && rtok < xb + kChunk) {  // the rejected proposal loses q_r of its mass
                const float pr = row[rtok];
                acc += q62(clamp01(pr - rq)) - q62(clamp01(pr));
            }
            p.partials[(int64_t)b * p.nc + c] = acc;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = nx[u];
    }
}

// One workgroup per stream: exact threshold, crossing chunk, crossing index.
__global__ void __launch_bounds__(kThreads) verify_sample(VParams p) {
    const VerifyArgs &a = p.a;
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    __shared__ int sh_chunk, sh_tok;
    __shared__ uint64_t sh_base;
    __shared__ uint64_t sh_scan[kWaves];
    __shared__ float sh_av[kThreads];
    __shared__ int sh_ai[kThreads];

    // loads that do not depend on gamma first: the chunk sums, offsets, the uniform
    const int nc = p.nc;
    const uint64_t *part = p.partials + (int64_t)b * nc;
    const int per = (nc + kThreads - 1) / kThreads;
    const int ca = tid * per < nc ? tid * per : nc;
    const int cb = ca + per < nc ? ca + per : nc;
    uint64_t local = 0;
    for (int c = ca; c < cb; ++c) local += part[c];
    const int r = p.rsel[b];
    const int t0 = a.target_off[b];
    const int M = a.target_off[b + 1] - t0;
    const float us = a.u_sample[b];
    if (r < 0) return;  // sentinel stream, outputs already written (uniform per workgroup)
    const int vt = a.v_t;
    const float *row = a.target_probs + (int64_t)(t0 + b + r) * a.target_ld;
    const int rtok = r < M ? a.target_ids[t0 + r] : -1;
    const float rq = r < M ? a.q[t0 + r] : 0.0f;
    if (tid == 0) sh_chunk = nc;
    uint64_t Z;
    const uint64_t base = block_exclusive_scan(local, &Z, sh_scan);

    int token;
    if (Z == 0) {
        token = block_first_argmax(row, vt, sh_av, sh_ai);
    } else {
        const uint64_t T = exact_threshold(us, Z);
        uint64_t run = base;
        for (int c = ca; c < cb; ++c) {
            const uint64_t nx = run + part[c];
            if (run <= T && nx > T) atomicMin(&sh_chunk, c);
            run = nx;
        }
        __syncthreads();
        const int cs = sh_chunk;
        if (cs < nc && ca <= cs && cs < cb) {
            uint64_t run2 = base;
            for (int c = ca; c < cs; ++c) run2 += part[c];
            sh_base = run2;
        }
        if (tid == 0) sh_tok = INT_MAX;
        __syncthreads();
        if (cs < nc) {
            const int x0 = cs * kChunk + tid * 4;
            uint64_t qv[4];
            uint64_t loc = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int x = x0 + k;
                const float pv = x < vt ? row[x] : 0.0f;
                qv[k] = q62(clamp01(pv - (x == rtok ? rq : 0.0f)));
                loc += qv[k];
            }
            uint64_t tot2;
            uint64_t pre = block_exclusive_scan(loc, &tot2, sh_scan) + sh_base;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                pre += qv[k];
                if (pre > T) {
                    atomicMin(&sh_tok, x0 + k);
                    break;
                }
            }
            __syncthreads();
        }
        token = (sh_tok == INT_MAX) ? vt - 1 : sh_tok;
    }
    if (tid == 0) {
        a.n_accepted[b] = r;
        a.out_token[b] = token;
        p.zsum[b] = Z;
    }
}

// Optional normalised residual row: res[x] = R(x) / fp32(Z * 2^-62), one-hot when Z = 0.
__global__ void __launch_bounds__(kThreads) residual_write(VParams p, int rsplit) {
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
        for (int x = x0 + (int)threadIdx.x; x < x1; x += kThreads) res[x] = (x == tok) ? 1.0f : 0.0f;
        return;
    }
    const float zf = (float)Z * 0x1p-62f;
    for (int x = x0 + (int)threadIdx.x; x < x1; x += kThreads)
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
    // splits per stream: aim for ~kTargetWorkgroups workgroups, at least one chunk per wave
    int max_splits = (p.nc + kWaves - 1) / kWaves;
    int splits = (kTargetWorkgroups + a.n_streams - 1) / a.n_streams;
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    p.cpw = (p.nc + splits - 1) / splits;
    p.splits = (p.nc + p.cpw - 1) / p.cpw;
    p.work_items = a.n_streams * p.splits;
    p.vec4 = ((reinterpret_cast<uintptr_t>(a.target_probs) & 15u) == 0 && (a.target_ld % 4) == 0) ? 1 : 0;
    const int grid = ((p.work_items + kXcds - 1) / kXcds) * kXcds;
    hipLaunchKernelGGL(verify_stream, dim3(grid), dim3(kThreads), 0, stream, p);
    if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
    hipLaunchKernelGGL(verify_sample, dim3(a.n_streams), dim3(kThreads), 0, stream, p);
    if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
    if (a.residual != nullptr) {
        int rsplit = (a.v_t + 8191) / 8192;
        if (rsplit < 1) rsplit = 1;
        hipLaunchKernelGGL(residual_write, dim3(a.n_streams * rsplit), dim3(kThreads), 0, stream, p, rsplit);
        if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
    }
    return TT_OK;
}

}  // namespace tt
