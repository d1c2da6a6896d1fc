// Device building blocks of the vocabulary-wide sampler, shared by the verify kernels
// and the fused step kernel: exact Q62 fixed point, wave scans, chunk streaming and
// the inverse-CDF sample.  Internal to the library.
#pragma once

#include <climits>
#include <cmath>

#include "stamps.h"
#include "tt_internal.h"

#ifndef TT_VERIFY_NT_LOADS
#define TT_VERIFY_NT_LOADS 1  // row loads carry the non-temporal hint (0: ordinary loads)
#endif

namespace tt {
namespace vcore {

constexpr int kWave = 64;
constexpr int kChunk = 1024;  // floats per chunk: one wave, 16 per lane

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

// v plus v shifted across lanes by a DPP control (32 bits; lanes without a source add 0).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_add32(uint32_t v) {
    return v + __builtin_amdgcn_update_dpp(0u, v, CTRL, ROW_MASK, 0xF, true);
}

__device__ __forceinline__ uint32_t wave_scan32(uint32_t v) {
    v = dpp_add32<0x111, 0xF>(v);  // row_shr:1
    v = dpp_add32<0x112, 0xF>(v);  // row_shr:2
    v = dpp_add32<0x114, 0xF>(v);  // row_shr:4
    v = dpp_add32<0x118, 0xF>(v);  // row_shr:8
    v = dpp_add32<0x142, 0xA>(v);  // row_bcast:15
    v = dpp_add32<0x143, 0xC>(v);  // row_bcast:31
    return v;
}

// The wave's total of v modulo 2^64, in lane 63 only: v's bits 0-21, 22-43 and 44-63 are
// summed as 32-bit values (64 of them stay below 2^28) by three DPP scans, half the
// instructions of the 64-bit scan.
__device__ __forceinline__ uint64_t wave_total(uint64_t v) {
    const uint32_t a = wave_scan32((uint32_t)v & 0x3FFFFFu);
    const uint32_t b = wave_scan32((uint32_t)(v >> 22) & 0x3FFFFFu);
    const uint32_t c = wave_scan32((uint32_t)(v >> 44));
    return (uint64_t)a + ((uint64_t)b << 22) + ((uint64_t)c << 44);
}

__device__ __forceinline__ uint64_t lane_value(uint64_t v, int lane) {
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, lane);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}

// First index of the maximum over the row (NaN never wins); 0 if nothing exceeds -inf.
// One wave.
__device__ inline int wave_first_argmax(const float *row, int vt) {
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

// Q62 sum of one loaded chunk c; lane 63 hands it to store(c, sum).  The rejected
// proposal's token rtok loses q_r = rq of its mass: rp is its entry P(rtok), which the
// acceptance test has already gathered, so the chunk holding it needs no second load.
template <class Store>
__device__ __forceinline__ void sum_chunk(const float4 (&v)[4], int c, int rtok, float rq, float rp, Store &store) {
    const int lane = threadIdx.x % kWave;
    uint64_t acc = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u)
        acc += q62(clamp01(v[u].x)) + q62(clamp01(v[u].y)) + q62(clamp01(v[u].z)) + q62(clamp01(v[u].w));
    acc = wave_total(acc);
    if (lane == kWave - 1) {
        const int xb = c * kChunk;
        if (rtok >= xb && rtok < xb + kChunk) acc += q62(clamp01(rp - rq)) - q62(clamp01(rp));
        store(c, acc);
    }
}

// The chunk a wave takes after its current one.  With an LDS counter (next != nullptr,
// initialised by the caller to c0 + the number of waves before a barrier) chunks are handed
// out in order to whichever wave asks first, so waves that the memory system serves faster
// take more of the row; without one the wave strides by the number of waves.
__device__ __forceinline__ int next_chunk(int *next, int c, int stride) {
    if (next == nullptr) return c + stride;
    int n = 0;
    if (threadIdx.x % kWave == 0) n = atomicAdd(next, 1);
    return __builtin_amdgcn_readfirstlane(n);
}

// Q62 sums of chunks [c0, c1): wave w starts at c0 + w and keeps one chunk in flight ahead of
// the one it sums; lane 63 hands each sum to store(c, sum).
template <class Store>
__device__ __forceinline__ void stream_chunks(const float *row, int vt, bool vec, int c0, int c1, int stride,
                                              int rtok, float rq, float rp, Store store, int *next = nullptr) {
    const int lane = threadIdx.x % kWave, wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    int c = c0 + wave;
    if (c >= c1) return;
    float4 v[4], nx[4];
    load_chunk(row, c * kChunk, lane, vt, vec, v);
    int cn = next_chunk(next, c, stride);
    for (;;) {
        int cnn = c1;
        if (cn < c1) {
            load_chunk(row, cn * kChunk, lane, vt, vec, nx);
            cnn = next_chunk(next, cn, stride);
        }
        sum_chunk(v, c, rtok, rq, rp, store);
        if (cn >= c1) break;
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = nx[u];
        c = cn;
        cn = cnn;
    }
}

// 16 consecutive floats row[x0 .. x0 + 16) (zero past vt).
__device__ __forceinline__ void read16(const float *row, int x0, int vt, bool vec, float (&pv)[16]) {
    if (vec && x0 + 16 <= vt) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 t = *reinterpret_cast<const float4 *>(row + x0 + 4 * q);
            pv[4 * q] = t.x;
            pv[4 * q + 1] = t.y;
            pv[4 * q + 2] = t.z;
            pv[4 * q + 3] = t.w;
        }
    } else {
#pragma unroll
        for (int k = 0; k < 16; ++k) pv[k] = x0 + k < vt ? row[x0 + k] : 0.0f;
    }
}

// Dense proposal (standard speculative sampling over one vocabulary): the residual is
// max(0, p - q) elementwise over two rows.  Q62 sum of one loaded chunk of each row.
template <class Store>
__device__ __forceinline__ void sum_chunk_dense(const float4 (&vp)[4], const float4 (&vq)[4], int c, Store &store) {
    uint64_t acc = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u)
        acc += q62(clamp01(vp[u].x - vq[u].x)) + q62(clamp01(vp[u].y - vq[u].y)) +
               q62(clamp01(vp[u].z - vq[u].z)) + q62(clamp01(vp[u].w - vq[u].w));
    acc = wave_total(acc);
    if (threadIdx.x % kWave == kWave - 1) store(c, acc);
}

// As stream_chunks for the dense residual: chunks [c0, c1) of both rows, one chunk of each
// ahead in flight.
template <class Store>
__device__ __forceinline__ void stream_chunks_dense(const float *prow, const float *qrow, int vt, bool vec, int c0,
                                                    int c1, int stride, Store store, int *next = nullptr) {
    const int lane = threadIdx.x % kWave, wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    int c = c0 + wave;
    if (c >= c1) return;
    float4 vp[4], vq[4], np_[4], nq[4];
    load_chunk(prow, c * kChunk, lane, vt, vec, vp);
    load_chunk(qrow, c * kChunk, lane, vt, vec, vq);
    int cn = next_chunk(next, c, stride);
    while (c < c1) {
        int cnn = c1;
        if (cn < c1) {
            load_chunk(prow, cn * kChunk, lane, vt, vec, np_);
            load_chunk(qrow, cn * kChunk, lane, vt, vec, nq);
            cnn = next_chunk(next, cn, stride);
        }
        sum_chunk_dense(vp, vq, c, store);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            vp[u] = np_[u];
            vq[u] = nq[u];
        }
        c = cn;
        cn = cnn;
    }
}

// Z (the row's Q62 mass), T = floor(u * Z) and the chunk cs holding the crossing, with the
// mass `base` of the chunks before it, from the nc chunk sums part(c), by one wave.  Chunk
// sums are scanned lane-blocked (lane l holds chunks [l * per, (l + 1) * per)); searches
// inside a lane are branch-free counts.  Returns 0 when cs is found, 1 when Z = 0, 2 when no
// chunk holds the crossing (the Q62 mass wrapped: not a probability row).  Z, T, cs and base
// are the same in every lane.
template <class Part>
__device__ __forceinline__ int find_crossing(int nc, Part part, float u, uint64_t &Z, uint64_t &T, int &cs,
                                             uint64_t &base) {
    constexpr int kPerMax = 4;  // chunk sums kept in registers per lane (rows up to 256K floats)
    const int lane = threadIdx.x % kWave;
    const int per = (nc + kWave - 1) / kWave;
    const int ca = lane * per < nc ? lane * per : nc;
    const int cb = ca + per < nc ? ca + per : nc;
    uint64_t ps[kPerMax];
    uint64_t local = 0;
    if (per <= kPerMax) {
#pragma unroll
        for (int k = 0; k < kPerMax; ++k) {
            ps[k] = ca + k < cb ? part(ca + k) : 0ull;
            local += ps[k];
        }
    } else {
        for (int c = ca; c < cb; ++c) local += part(c);
    }
    const uint64_t incl = wave_inclusive_scan(local);
    Z = lane_value(incl, kWave - 1);
    T = 0;
    cs = 0;
    base = 0;
    if (Z == 0) return 1;
    T = exact_threshold(u, Z);
    // lane whose block of chunks holds the crossing, then the chunk inside it
    const uint64_t excl = incl - local;
    const unsigned long long hit = __ballot(excl <= T && T < incl);
    if (hit == 0ull) return 2;
    const int owner = __ffsll(hit) - 1;
    int c_at = ca;
    uint64_t b_at = excl;
    if (per <= kPerMax) {
        uint64_t run = excl;
#pragma unroll
        for (int k = 0; k < kPerMax; ++k) {  // chunks of this lane wholly at or below T
            const bool below = ca + k < cb && run + ps[k] <= T;
            c_at += below ? 1 : 0;
            b_at = below ? run + ps[k] : b_at;
            run += ps[k];
        }
    } else if (lane == owner) {
        uint64_t run = excl;
        for (int c = ca; c < cb; ++c) {
            const uint64_t nx = run + part(c);
            if (nx > T) break;
            c_at = c + 1;
            b_at = nx;
            run = nx;
        }
    }
    cs = __builtin_amdgcn_readlane(c_at, owner);
    base = lane_value(b_at, owner);
    return 0;
}

// Inverse-CDF sample of the row from its nc chunk sums part(c), by one wave: every lane
// returns the token and *Zout the Q62 mass.  The residual is max(0, row - qrow) when qrow
// is given (dense proposal), else row less rq at the rejected proposal rtok (one-hot).  The
// crossing chunk's row values come as 16 consecutive floats per lane from chunk16(cs, x0, pv)
// (wave_sample: read again from the row) and are scanned.
template <class Part, class Chunk16>
__device__ inline int wave_sample_with(const float *row, const float *qrow, int vt, int nc, bool vec, Part part,
                                       Chunk16 chunk16, float u, int rtok, float rq, uint64_t *Zout) {
    const int lane = threadIdx.x % kWave;
    uint64_t Z, T, base;
    int cs;
    const int st = find_crossing(nc, part, u, Z, T, cs, base);
    *Zout = Z;
    if (st == 1) return wave_first_argmax(row, vt);
    if (st == 2) return vt - 1;
    // the crossing chunk: lane holds elements cs*1024 + lane*16 + [0, 16)
    const int x0 = cs * kChunk + lane * 16;
    float pv[16], dv[16];
    chunk16(cs, x0, pv);
    if (qrow != nullptr) {
        read16(qrow, x0, vt, vec, dv);
    } else {
#pragma unroll
        for (int k = 0; k < 16; ++k) dv[k] = x0 + k == rtok ? rq : 0.0f;
    }
    uint64_t qv[16];
    uint64_t sum = 0;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        qv[k] = x0 + k < vt ? q62(clamp01(pv[k] - dv[k])) : 0ull;
        sum += qv[k];
    }
    const uint64_t lincl = wave_inclusive_scan(sum) + base;
    const uint64_t lexcl = lincl - sum;
    const unsigned long long lhit = __ballot(lexcl <= T && T < lincl);
    if (lhit == 0ull) return vt - 1;
    const int tl = __ffsll(lhit) - 1;
    // in the crossing lane: the number of leading elements whose inclusive prefix is <= T
    uint64_t run = lexcl;
    int k_at = 0;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        run += qv[k];
        k_at += run <= T ? 1 : 0;
    }
    return __builtin_amdgcn_readlane(x0 + k_at, tl);
}

template <class Part>
__device__ inline int wave_sample(const float *row, const float *qrow, int vt, int nc, bool vec, Part part, float u,
                                  int rtok, float rq, uint64_t *Zout) {
    return wave_sample_with(
        row, qrow, vt, nc, vec, part, [&](int, int x0, float(&pv)[16]) { read16(row, x0, vt, vec, pv); }, u, rtok,
        rq, Zout);
}

}  // namespace vcore
}  // namespace tt
