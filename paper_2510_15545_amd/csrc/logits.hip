// Verification from bf16 target logits with a temperature on gfx950: the target softmax of
// Sec. 3's acceptance rule and App. D Alg. 4's residual is formed inside the verification
// (App. F lists the sampling temperatures), so the caller never materialises fp32
// probability rows.
//
// Arithmetic (every step specified, so any summation order gives the same token), in base 2:
//   c      = inv_temp * log2(e) (fp32, once per stream); y = fp32(bf16 logit) * c, NaN counts
//            as minus infinity (no mass, never the max)
//   mu     = max y over the row, or L * log2(e) for a caller's log-sum-exp L (natural units)
//   z      = fma(logit, c, 31 - mu) held in [-1, 31]: the logit's scaled base-2 exponent
//   2^z    = p * 2^k, k = rint(z), p the degree-5 Taylor polynomial of 2^(z - k) (Horner, FMAs)
//   e31    = floor(p * 2^k), the weight in Q31, summed exactly in 64 bits (rows <= 2^23 entries)
//   E      = p * 2^(k - 31) (0 for z < 0); S = sum * 2^-31 rounded once to fp32 (ties to even)
//   P(t_j) = E(t_j) / S (E(t_j) with L); accept while q_j <= 0 or u_j < P(t_j) / q_j
//   after a rejection at r the entry t_r of the residual is
//            floor(clamp(E(t_r) - q_r S, 0, 1) * 2^31), proportional to max(0, P - q_r e_t);
//            after full acceptance the bonus row's e31 is sampled as is
//   token  = first index whose prefix exceeds floor(u * Z); first largest y when Z = 0.
//
// One 1024-thread workgroup per stream.  Without normalisers it walks its rows 0, 1, ...
// until the first rejection (each row: a max pass, then a pass of chunk sums into LDS -- the
// second read mostly from the caches).  With per-row log-sum-exp values L from the caller
// (an LM head can emit them with its logits) it uses m = L and S = 1: the acceptance test
// needs one gathered logit per position and only the residual (or bonus) row is read, once.
// Wave 0 samples: the chunk sums lane-blocked, the crossing chunk's e31 recomputed from its
// 1024 logits.  In the row passes a lane reads 16 bf16 with two 16-byte loads, each load
// instruction covering 1 KB of the row; the sampler reads 16 consecutive bf16 a lane.
#include "verify_core.h"

TT_STAMPS_TABLE(logits)

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

constexpr float kLog2e = 0x1.715476p+0f;  // log2(e) rounded to fp32

// 2^z = p * 2^k for z held in [-1, 31] (NaN gives p * 2^k < 1, a zero weight): k = rint(z),
// f = z - k in [-1/2, 1/2] (exact), p = 1 + f ln2 + ... + (f ln2)^5 / 5! by Horner's rule.
__device__ __forceinline__ float exp2_parts(float z, int &k) {
    z = fminf(fmaxf(z, -1.0f), 31.0f);
    const float kf = rintf(z);
    const float f = z - kf;
    float p = 0x1.5d87fep-10f;
    p = fmaf(p, f, 0x1.3b2ab6p-7f);
    p = fmaf(p, f, 0x1.c6b08ep-5f);
    p = fmaf(p, f, 0x1.ebfbe0p-3f);
    p = fmaf(p, f, 0x1.62e430p-1f);
    p = fmaf(p, f, 1.0f);
    k = (int)kf;
    return p;
}

// floor(2^z): the weight in Q31 of a logit whose scaled exponent is z (p * 2^k < 2^32)
__device__ __forceinline__ uint32_t e31_at(float z) {
    int k;
    const float p = exp2_parts(z, k);
    return (uint32_t)ldexpf(p, k);
}

// E = 2^(z - 31) as fp32, 0 when z < 0 or NaN (where the Q31 weight is 0)
__device__ __forceinline__ float weight_at(float z) {
    if (!(z >= 0.0f)) return 0.0f;
    int k;
    const float p = exp2_parts(z, k);
    return ldexpf(p, k - 31);
}

// floor(r * 2^31) for r in [0, 1]
__device__ __forceinline__ uint32_t q31(float r) { return (uint32_t)ldexpf(r, 31); }

// n * 2^-31 rounded to the nearest fp32, ties to even
__device__ inline float q31_to_f32(uint64_t n) {
    if (n == 0) return 0.0f;
    const int bl = 64 - __clzll(n);
    if (bl <= 24) return ldexpf((float)n, -31);
    const int sh = bl - 24;
    uint64_t mant = n >> sh;
    const uint64_t rem = n & ((1ull << sh) - 1), half = 1ull << (sh - 1);
    if (rem > half || (rem == half && (mant & 1u))) ++mant;
    return ldexpf((float)mant, sh - 31);
}

// y = logit * c.  A NaN y is left as is: fmaxf ignores it in the max pass and it never
// compares greater in the first-argmax fallback; its scaled exponent gives a zero weight.
__device__ __forceinline__ float scaled(uint32_t bits16, float c) { return bf16_value(bits16) * c; }

// the scaled exponent z of a logit: fma(logit, c, b31) with b31 = 31 - mu
__device__ __forceinline__ float expo(uint32_t bits16, float c, float b31) { return fmaf(bf16_value(bits16), c, b31); }

// 16 consecutive logits x0 .. x0 + 15 of a lane (the sampler's crossing chunk; zero bits past v).
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

// The 16 bf16 a lane takes of chunk c in the row passes: elements 512 u + 8 lane + j (u < 2,
// j < 8), so that each of the two 16-byte load instructions covers 1 KB of the row (16
// consecutive logits a lane would make each span 2 KB); 0 past v.  NT: the non-temporal hint
// (the row's last read).  A chunk's sums and maximum do not depend on the order.
template <bool NT>
__device__ __forceinline__ void load16s(const uint16_t *row, int c, int lane, int v, bool vec, uint32_t (&w)[8]) {
    const int xb = c * kChunk;
    if (vec && xb + kChunk <= v) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const uint4 *src = reinterpret_cast<const uint4 *>(row + xb + u * 512 + lane * 8);
            uint4 t;
            if constexpr (NT) {
                typedef unsigned int u4v __attribute__((ext_vector_type(4)));
                const u4v q = __builtin_nontemporal_load(reinterpret_cast<const u4v *>(src));
                t = make_uint4(q.x, q.y, q.z, q.w);
            } else {
                t = *src;
            }
            w[4 * u] = t.x;
            w[4 * u + 1] = t.y;
            w[4 * u + 2] = t.z;
            w[4 * u + 3] = t.w;
        }
    } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int x = xb + (k >> 2) * 512 + lane * 8 + 2 * (k & 3);
            const uint32_t lo = x < v ? row[x] : 0u;
            const uint32_t hi = x + 1 < v ? row[x + 1] : 0u;
            w[k] = lo | (hi << 16);
        }
    }
}

// Index of element k (0..15) of a lane's 16 in chunk c, in load16s's order.
__device__ __forceinline__ int elem_index_s(int c, int lane, int k) {
    return c * kChunk + (k >> 3) * 512 + lane * 8 + (k & 7);
}

// bf16 element k (0..15) of a lane's 16
__device__ __forceinline__ uint32_t elem(const uint32_t (&w)[8], int k) {
    return (k & 1) ? (w[k >> 1] >> 16) : (w[k >> 1] & 0xFFFFu);
}

struct LogitsParams {
    LogitsArgs a;
    int32_t nc, vec;
};

// Per-row table of the Q31 weights.  For a fixed scale and offset the weight of a logit is a
// function of its 16 bits, so the row pass looks it up instead of evaluating the exponential:
// the table holds e31_at(expo(bits)) for every pattern whose magnitude lies in [2^-20, 2^8)
// (exponent fields 107 .. 134, 3,584 patterns a sign), as 64-bit entries that add straight into
// the 64-bit sums.  Each sign owns a half of 4,096 slots (32 KiB, so the pattern's sign bit,
// left in place, is the byte offset of its half); slot 0 and slot 3,585 of a half are sentinels,
// 2^40 (a weight is at most 2^31: z <= 31), onto which magnitudes outside the domain clamp
// (tiny values, |x| >= 256, infinities, NaNs).  A lane group whose sum reaches 2^40 met one and
// is summed again from the formula.
constexpr uint32_t kMagLo = 107u << 7;  // bf16 magnitude bits of 2^-20
constexpr uint32_t kTabMags = 28u << 7;
constexpr int kTabHalf = 4096;
constexpr int kTabSlots = 2 * kTabHalf;
constexpr uint64_t kSentinel = 1ull << 40;

__device__ __forceinline__ void build_table(uint64_t *tab, float sc, float b31) {
    for (int i = threadIdx.x; i < kTabSlots; i += kThreads) {
        const uint32_t s = (uint32_t)i / kTabHalf, j = (uint32_t)i % kTabHalf;
        if (j > kTabMags + 1) continue;  // never addressed
        uint64_t e = kSentinel;
        if (j > 0 && j <= kTabMags) e = e31_at(expo((s << 15) | (kMagLo + j - 1), sc, b31));
        tab[i] = e;
    }
}

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// The LDS byte offsets of the two bf16 in a 32-bit word (low half first), both formed at once
// with packed 16-bit operations: the magnitude clamped to the domain's frame, rebased and
// scaled to a byte offset, and the pattern's sign bit kept as the half's offset.
__device__ __forceinline__ uint32_t tab_offsets(uint32_t w) {
    u16x2 t = __builtin_bit_cast(u16x2, w & 0x7FFF7FFFu);
    t = __builtin_elementwise_max(t, (u16x2)(unsigned short)(kMagLo - 1));
    t = __builtin_elementwise_min(t, (u16x2)(unsigned short)(kMagLo + kTabMags));
    // (t - (kMagLo - 1)) * 8, modulo 2^16 (the true value is below 2^15)
    t = t * (u16x2)(unsigned short)8 - (u16x2)(unsigned short)((kMagLo - 1) * 8);
    return __builtin_bit_cast(uint32_t, t) | (w & 0x80008000u);
}

__device__ __forceinline__ uint64_t tab_at(const uint64_t *tab, uint32_t byte_off) {
    return *reinterpret_cast<const uint64_t *>(reinterpret_cast<const char *>(tab) + byte_off);
}

// The 16 weights of a lane's logits x0 .. x0+15 (0 past v) into e; a sentinel for a logit
// outside the table's domain is replaced by the formula's weight.
__device__ __forceinline__ void lane_weights(const uint64_t *tab, const uint32_t (&w)[8], int x0, int v, float sc,
                                             float b31, uint64_t (&e)[16]) {
    uint64_t any = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const uint32_t o = tab_offsets(w[k]);
        e[2 * k] = x0 + 2 * k < v ? tab_at(tab, o & 0xFFFFu) : 0u;
        e[2 * k + 1] = x0 + 2 * k + 1 < v ? tab_at(tab, o >> 16) : 0u;
        any |= e[2 * k] | e[2 * k + 1];
    }
    if (any >= kSentinel) {
#pragma unroll
        for (int k = 0; k < 16; ++k) e[k] = x0 + k < v ? e31_at(expo(elem(w, k), sc, b31)) : 0u;
    }
}

// As lane_weights for a lane's 16 logits of chunk c in load16s's order.
__device__ __forceinline__ void lane_weights_s(const uint64_t *tab, const uint32_t (&w)[8], int c, int v, float sc,
                                               float b31, uint64_t (&e)[16]) {
    const int lane = threadIdx.x % kWave;
    uint64_t any = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const uint32_t o = tab_offsets(w[k]);
        e[2 * k] = elem_index_s(c, lane, 2 * k) < v ? tab_at(tab, o & 0xFFFFu) : 0u;
        e[2 * k + 1] = elem_index_s(c, lane, 2 * k + 1) < v ? tab_at(tab, o >> 16) : 0u;
        any |= e[2 * k] | e[2 * k + 1];
    }
    if (any >= kSentinel) {
#pragma unroll
        for (int k = 0; k < 16; ++k) e[k] = elem_index_s(c, lane, k) < v ? e31_at(expo(elem(w, k), sc, b31)) : 0u;
    }
}

// The wave's total of per-lane sums of 16 weights (each at most 2^35), in lane 63: the low 20
// and the high 15 bits are summed as 32-bit values (64 of them stay below 2^26 and 2^21).
__device__ __forceinline__ uint64_t chunk_total(uint64_t a) {
    const uint32_t lo = vcore::wave_scan32((uint32_t)a & 0xFFFFFu);
    const uint32_t hi = vcore::wave_scan32((uint32_t)(a >> 20));
    return ((uint64_t)hi << 20) + lo;
}

// The row's weight table, then its chunk sums of e31 into sh_part.  Every wave first issues the
// loads of its first two chunks, so that their latency passes while the table is built; waves
// take chunks from the LDS counter *next (which the caller sets to kWaves before a barrier that
// precedes the call; wave w starts at chunk w), one chunk in flight ahead of the one summed.
__device__ __forceinline__ void chunk_sums(const uint16_t *row, int v, int nc, bool vec, float sc, float b31,
                                           uint64_t *tab, uint64_t *sh_part, int *next) {
    const int lane = threadIdx.x % kWave, wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    uint32_t w[8] = {}, nx[8] = {};
    int c = wave, cn = nc, cnn = nc;  // chunk summed, chunk in flight, the one after it
    if (c < nc) {
        load16s<true>(row, c, lane, v, vec, w);
        cn = vcore::next_chunk(next, c, kWaves);
        if (cn < nc) {
            load16s<true>(row, cn, lane, v, vec, nx);
            cnn = vcore::next_chunk(next, cn, kWaves);
        }
    }
    build_table(tab, sc, b31);
    __syncthreads();
    while (c < nc) {
        uint64_t acc = 0;
        if ((c + 1) * kChunk <= v) {
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const uint32_t o = tab_offsets(w[k]);
                acc += tab_at(tab, o & 0xFFFFu) + tab_at(tab, o >> 16);
            }
            if (acc >= kSentinel) {  // a logit outside the table's domain: the lane group by the formula
                acc = 0;
#pragma unroll
                for (int k = 0; k < 16; ++k) acc += e31_at(expo(elem(w, k), sc, b31));
            }
        } else {  // the row's ragged end
            uint64_t e[16];
            lane_weights_s(tab, w, c, v, sc, b31, e);
#pragma unroll
            for (int k = 0; k < 16; ++k) acc += e[k];
        }
        acc = chunk_total(acc);
        if (lane == kWave - 1) sh_part[c] = acc;
        c = cn;
        if (c < nc) {
#pragma unroll
            for (int k = 0; k < 8; ++k) w[k] = nx[k];
            cn = cnn;
            if (cn < nc) {
                load16s<true>(row, cn, lane, v, vec, nx);
                cnn = vcore::next_chunk(next, cn, kWaves);
            }
        }
    }
}

// Inverse-CDF sample of a row from its chunk sums (one wave).  When t >= 0 the entry at t
// counts adj instead of the before its chunk sum holds (the residual's entry); Z is the row's
// total so adjusted.  The first largest x when Z = 0.
__device__ inline int sample_row(const uint16_t *row, int v, int nc, bool vec, float sc, float b31,
                                 const uint64_t *tab, int t, uint64_t adj, uint64_t before, float u,
                                 const uint64_t *sh_part) {
    const int lane = threadIdx.x % kWave;
    // chunk sums lane-blocked: lane l holds chunks [l*per, (l+1)*per)
    const int per = (nc + kWave - 1) / kWave;
    const int ca = lane * per < nc ? lane * per : nc;
    const int cb = ca + per < nc ? ca + per : nc;
    const int ct = t >= 0 ? t / kChunk : -1;
    uint64_t local = 0;
    for (int c = ca; c < cb; ++c) local += sh_part[c];
    if (ct >= ca && ct < cb) local = local - before + adj;
    const uint64_t incl = wave_inclusive_scan(local);
    const uint64_t Z = lane_value(incl, kWave - 1);
    if (Z == 0) {
        float bv = -INFINITY;
        int bi = INT_MAX;
        for (int x = lane; x < v; x += kWave) {
            const float xv = scaled(row[x], sc);
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
        return bi == INT_MAX ? 0 : bi;
    }
    const uint64_t T = exact_threshold(u, Z);
    const uint64_t excl = incl - local;
    const unsigned long long hit = __ballot(excl <= T && T < incl);
    if (hit == 0ull) return v - 1;  // only if the sums wrapped (rows longer than allowed)
    const int owner = __ffsll(hit) - 1;
    int cs = ca;
    uint64_t base_sum = excl;
    if (lane == owner) {
        uint64_t run = excl;
        for (int c = ca; c < cb; ++c) {
            const uint64_t nx = run + (c == ct ? sh_part[c] - before + adj : sh_part[c]);
            if (nx > T) break;
            cs = c + 1;
            base_sum = nx;
            run = nx;
        }
    }
    cs = __builtin_amdgcn_readlane(cs, owner);
    base_sum = lane_value(base_sum, owner);
    // the crossing chunk: lane holds elements cs*1024 + lane*16 + [0, 16)
    const int x0 = cs * kChunk + lane * 16;
    uint32_t w[8];
    load16(row, x0, v, vec, w);
    uint64_t qv[16];
    lane_weights(tab, w, x0, v, sc, b31, qv);
    uint64_t sum = 0;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        if (x0 + k == t) qv[k] = adj;
        sum += qv[k];
    }
    const uint64_t lincl = wave_inclusive_scan(sum) + base_sum;
    const uint64_t lexcl = lincl - sum;
    const unsigned long long lhit = __ballot(lexcl <= T && T < lincl);
    if (lhit == 0ull) return v - 1;
    const int tl = __ffsll(lhit) - 1;
    uint64_t run = lexcl;
    int k_at = 0;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        run += qv[k];
        k_at += run <= T ? 1 : 0;
    }
    return __builtin_amdgcn_readlane(x0 + k_at, tl);
}

__global__ void __launch_bounds__(kThreads) verify_logits_row(LogitsParams p) {
    const LogitsArgs &a = p.a;
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    extern __shared__ uint64_t sh_part[];  // nc chunk sums of e31
    __shared__ float sh_red[kWaves];
    __shared__ int sh_ok, sh_r;
    __shared__ float sh_m, sh_L, sh_q, sh_P;
    __shared__ int sh_next;  // 1: accepted, go to the next row
    __shared__ uint64_t sh_before, sh_adj;
    __shared__ int sh_t, sh_x;
    __shared__ int sh_ctr;  // the row pass's chunk counter
    __shared__ uint64_t sh_tab[kTabSlots];  // the row's weight table

    const int t0 = a.target_off[b];
    const int M = a.target_off[b + 1] - t0;
    const float it = a.inv_temp[b];
    const float cb = it * kLog2e;  // the stream's base-2 scale
    const int v = a.v_t, nc = p.nc;
    const bool vec = p.vec != 0;
    TT_STAMP(0);
    if (!(M >= 0 && M <= a.max_m && it > 0.0f)) {
        if (tid == 0) {
            a.n_accepted[b] = -1;
            a.out_token[b] = -1;
        }
        return;
    }
    if (wave == kWaves - 1) {  // every proposal's id inside the vocabulary (beside wave 0's scan)
        bool ok = true;
        for (int base = 0; ok && base < M; base += kWave) {
            const int j = base + lane;
            const bool bad = j < M && (a.target_ids[t0 + j] < 0 || a.target_ids[t0 + j] >= v);
            ok = !__any(bad);
        }
        if (lane == 0) sh_ok = ok ? 1 : 0;
    }
    if (a.lse != nullptr) {
        // normalisers given: the acceptance test from one gathered logit per position, then
        // one pass over the residual (or bonus) row
        // (the rejecting lane's L, t, q, P and logit, or the bonus row's L, go to LDS with
        // gamma, so the row pass and the residual entry need no further dependent load; an id
        // outside the vocabulary is not gathered, and the stream then ends as a sentinel)
        if (wave == 0) {
            const float L_bonus = a.lse[t0 + b + M];
            int gamma = M, t_r = -1, x_r = 0;
            float L_r = L_bonus, q_r = 0.0f, P_r = 0.0f;
            for (int base = 0; base < M && gamma == M; base += kWave) {
                const int j = base + lane;
                bool rej = false;
                int tj = 0, xj = 0;
                float Lj = 0.0f, qj = 0.0f, P = 0.0f;
                if (j < M) {
                    const int64_t r = t0 + b + j;
                    tj = a.target_ids[t0 + j];
                    Lj = a.lse[r];
                    qj = a.q[t0 + j];
                    if (tj >= 0 && tj < v) {
                        xj = a.logits[r * a.ld + tj];
                        P = fminf(fmaxf(weight_at(expo(xj, cb, 31.0f - Lj * kLog2e)), 0.0f), 1.0f);
                        rej = !(qj <= 0.0f || a.u_accept[t0 + j] < P / qj);
                    }
                }
                const unsigned long long rm = __ballot(rej);
                if (rm != 0ull) {
                    const int src = __ffsll(rm) - 1;
                    gamma = base + src;
                    t_r = __builtin_amdgcn_readlane(tj, src);
                    x_r = __builtin_amdgcn_readlane(xj, src);
                    L_r = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(Lj), src));
                    q_r = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(qj), src));
                    P_r = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(P), src));
                }
            }
            if (lane == 0) {
                sh_ctr = kWaves;
                sh_r = gamma;
                sh_t = t_r;
                sh_x = x_r;
                sh_L = L_r;
                sh_q = q_r;
                sh_P = P_r;
            }
        }
        __syncthreads();
        TT_STAMP(1);
        if (!sh_ok) {
            if (tid == 0) {
                a.n_accepted[b] = -1;
                a.out_token[b] = -1;
            }
            return;
        }
        const int r = sh_r;
        const int64_t rr = t0 + b + r;
        const uint16_t *row = a.logits + rr * a.ld;
        const float L = sh_L;
        const float b31 = 31.0f - L * kLog2e;
        chunk_sums(row, v, nc, vec, cb, b31, sh_tab, sh_part, &sh_ctr);
        if (wave < 12) TT_STAMP_WAVE(4 + wave);
        __syncthreads();
        TT_STAMP(2);
        if (wave != 0) return;
        int t = -1;
        uint64_t adj = 0, before = 0;
        if (r < M) {  // the rejected proposal loses q_r of its mass: its entry is E(t) - q_r, clamped
            t = sh_t;
            adj = q31(fminf(fmaxf(sh_P - sh_q, 0.0f), 1.0f));
            before = e31_at(expo((uint32_t)sh_x, cb, b31));  // the weight the chunk sums counted at t
        }
        const int token = sample_row(row, v, nc, vec, cb, b31, sh_tab, t, adj, before, a.u_sample[b], sh_part);
        if (lane == 0) {
            a.n_accepted[b] = r;
            a.out_token[b] = token;
        }
        TT_STAMP(3);
        return;
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
        uint32_t w[8] = {}, nx[8] = {};
        if (wave < nc) load16s<false>(row, wave, lane, v, vec, w);
        for (int c = wave; c < nc; c += kWaves) {
            if (c + kWaves < nc) load16s<false>(row, c + kWaves, lane, v, vec, nx);
            if ((c + 1) * kChunk <= v) {
#pragma unroll
                for (int k = 0; k < 16; ++k) m = fmaxf(m, scaled(elem(w, k), cb));
            } else {
#pragma unroll
                for (int k = 0; k < 16; ++k)
                    if (elem_index_s(c, lane, k) < v) m = fmaxf(m, scaled(elem(w, k), cb));
            }
#pragma unroll
            for (int k = 0; k < 8; ++k) w[k] = nx[k];
        }
        for (int off = kWave / 2; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
        if (lane == 0) sh_red[wave] = m;
        __syncthreads();
        if (tid == 0) {
            float mm = -INFINITY;
            for (int k = 0; k < kWaves; ++k) mm = fmaxf(mm, sh_red[k]);
            sh_m = mm;
            sh_ctr = kWaves;
        }
        __syncthreads();
        m = sh_m;
        // pass 2: chunk sums of e31
        const float b31 = 31.0f - m;
        chunk_sums(row, v, nc, vec, cb, b31, sh_tab, sh_part, &sh_ctr);
        __syncthreads();
        // S, the acceptance test of position j, and the residual's entry at t_j
        if (wave == 0) {
            uint64_t local = 0;
            for (int c = lane; c < nc; c += kWave) local += sh_part[c];
            const uint64_t Sq = lane_value(wave_inclusive_scan(local), kWave - 1);
            if (lane == 0) {
                const float S = q31_to_f32(Sq);
                int next = 0;
                uint64_t before = 0, adj = 0;
                int t = -1;
                if (j < M) {
                    t = a.target_ids[t0 + j];
                    const float qj = a.q[t0 + j];
                    const float et = weight_at(expo(row[t], cb, b31));
                    const float P = et / S;
                    if (qj <= 0.0f || a.u_accept[t0 + j] < P / qj) {
                        next = 1;
                    } else {
                        const float rt = fminf(fmaxf(et - qj * S, 0.0f), 1.0f);  // NaN -> 0
                        before = e31_at(expo(row[t], cb, b31));
                        adj = q31(rt);
                    }
                }
                sh_next = next;
                sh_before = before;
                sh_t = next ? -1 : t;
                sh_adj = adj;
            }
        }
        __syncthreads();
        if (sh_next) continue;
        if (wave == 0) {
            const int token = sample_row(row, v, nc, vec, cb, b31, sh_tab, sh_t, sh_adj, sh_before, a.u_sample[b], sh_part);
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
    // the chunk sums (up to 64 KiB at the longest rows) sit beside the 64 KiB weight table in LDS
    const size_t lds = 8 * (size_t)p.nc;
    if (hipFuncSetAttribute(reinterpret_cast<const void *>(&verify_logits_row),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
        return TT_ELAUNCH;
    hipLaunchKernelGGL(verify_logits_row, dim3(a.n_streams), dim3(kThreads), lds, stream, p);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

}  // namespace tt
