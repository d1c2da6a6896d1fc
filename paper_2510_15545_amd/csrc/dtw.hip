// Dynamic Token Warping on gfx950 for pairs of any length: one 256-thread workgroup per
// (draft, proxy-target) pair, small enough in LDS that several pairs share a compute unit.
//
// Computes Alg. 1 of the paper (cumulative cost C over draft x target tokens with the
// Sakoe-Chiba band, Sec. 4.1) using the byte-level Levenshtein token distance of App. H,
// then the backtrack from (K, M) and the mapping of App. A.2.
//
// Work decomposition:
//   * Staging: every thread loads tokens (draft or target) -- id, byte offsets, bytes --
//     validates them and packs each into a fixed-width LDS slot.
//   * Draft rows are processed in strips of 64 with lane r of wave 0 owning row
//     i = i0 + r.  Wave 0 sweeps the strip's anti-diagonals: at step t lane r finishes
//     cell (i0 + r, jlo(i0) + t - r).  C(i-1, j) arrives from lane r-1 through a DPP wave
//     shift (lane 0 takes the previous strip's last row from LDS through the shift's
//     fill operand), C(i-1, j-1) is the value received one step earlier and C(i, j-1)
//     is the lane's own previous value.  The step is branch-free.
//   * Token distances: the strip's steps are cut into chunks of 64.  While wave 0 sweeps
//     chunk c, waves 1-3 evaluate the distances of chunk c + 1 into the other half of a
//     double buffer ([lane][step / 4] dwords, one byte per step, bit 7 set for cells
//     outside the band so the sweep needs no band arithmetic).  One barrier per chunk.
//   * Token distance: per-byte match masks of a packed token come from SWAR byte
//     comparison.  When every draft token of a wave's cells has at most two bytes (nearly
//     always for natural-language tokens), a closed form over the target token's match
//     masks for those bytes gives the distance; otherwise the bit-parallel edit-distance
//     recurrence (Myers 1999, in Hyyro's 2001 global-distance form) runs with the longer
//     token as the pattern (one bit per byte, at most 64) and the shorter one as the text.
//     Each thread loads the target tokens of its four cells together before computing.
//   * Each cell's predecessor choice is two bits (up: C(i-1, j) < C(i-1, j-1); left:
//     C(i, j-1) below both), shifted into a per-lane register, 16 steps per dword, and
//     stored straight from registers into the caller's workspace, row-major by draft row.
//   * Backtrack (wave 0), one row per step: inside row i the path runs left from its
//     entry column to the highest column whose move is not a left move,
//     then enters row i-1.  The walk runs in scalar registers: per row the code word
//     holding the entry cell is read (an LDS broadcast), the steps past it are masked and
//     the lowest set bit of the not-left flags gives the highest column.  The other waves stage the next strip's code words
//     into LDS meanwhile (rows of more than 64 words are read from the workspace).  Path
//     cells and map entries are then written by all threads with binary searches over
//     the rows' runs.
//
// LDS layout (bytes, each region 16-byte aligned):
//   tslot [max_m + 8][TB + 4] / tlen [max_m + 8]  target token bytes and lengths: 4 empty
//                                      slots on each side, a pad dword per slot when the plan fits
//                                      that way
//   dslot [max_k][TB] / dlen [max_k]   draft token bytes and lengths
//   row0, row1 [64 + max_m + 136] int32 C of the row above the strip / of the strip's last
//                                      row, by column with a 64-entry front pad
//   cost  2 x [64][17] u32             token distances of a chunk, double-buffered; during
//                                      the backtrack two strips of code words (2 x [64][RW])
//                                      when RW <= 64
//   path  [max_k] x 2 u32              per row: run (first column << 16 | entry column),
//                                      then the index of its first path cell
// Workspace: per pair max_k rows of RW = ceil(W / 16) + 1 code words, W the widest band
// row the bounds allow.
#include "dtw_common.h"

#ifndef TT_ALIGN_ROWS
#define TT_ALIGN_ROWS 1  // 0: short pairs also take the strip kernel
#endif

namespace tt {
namespace {

using dtw::kInf;
using dtw::kWave;
using dtw::read_slot;
using dtw::stage_token;
using dtw::token_distance;
// Workgroup size: wave 0 sweeps and walks, the other waves evaluate distances.  Eight waves
// at 64 VGPRs keep four workgroups on a compute unit; the register-hungry wide token slots
// use four.
template <int TB>
constexpr int band_threads() {
    return TB <= 16 ? 512 : 256;
}
constexpr int kChunk = 64;                       // sweep steps per cost chunk
constexpr int kOrderThreads = 256;               // dispatch-order ranks: threads per workgroup
constexpr int kOrderSplit = 4;                   // lanes counting one pair's rank
constexpr int kOrderPairsPerGroup = kOrderThreads / kOrderSplit;
constexpr int kOrderMax = 2048;                  // pairs it orders (11-bit index in the key); more keep their order
constexpr int kGroups = kChunk / 4;              // cost dwords per lane and chunk
constexpr int kCostStride = kGroups + 1;         // dwords per lane in a chunk buffer (odd: no bank conflicts)
constexpr int kRowFront = 64;                    // row buffers hold columns -64 .. max_m + 135
constexpr int kRowBack = 136;
constexpr size_t kLdsLimit = 160 * 1024 - 1024;  // gfx950 LDS per workgroup, less static use
constexpr uint32_t kOutOfBand = 0x80808080u;     // four cost bytes with the out-of-band bit
constexpr int kTPad = 4;                         // empty target slots before column 1 and after column M

__host__ __device__ inline size_t align16(size_t v) { return (v + 15) & ~size_t(15); }

struct LdsPlan {
    size_t tslot, tlen, dslot, dlen, row0, row1, cost, path, total;
    int tstride;  // dwords per target token slot
};

__host__ __device__ inline int band_half_width_bound(int32_t max_k, int32_t max_m, int32_t w) {
    int mx = max_k > max_m ? max_k : max_m;
    if (w < 0) return mx;
    int widen = mx - 1;  // largest possible |K - M|
    int L = w > widen ? w : widen;
    return L < mx ? L : mx;
}

// Code words stored per draft row: a band row of W cells starts anywhere inside a word.
__host__ __device__ inline int row_words_bound(int32_t max_k, int32_t max_m, int32_t w) {
    const long long L = band_half_width_bound(max_k, max_m, w);
    long long W = 2 * L + 1;
    if (W > max_m) W = max_m;
    return (int)((W + 15) / 16) + 1;
}

// Target token slots take TB / 4 + 1 dwords when the plan fits the LDS that way: the helper
// lanes of a row read slots four apart, which an odd stride spreads over distinct banks (a
// stride of TB / 4 dwords puts two lanes on every bank they use); else TB / 4.
__host__ __device__ inline LdsPlan plan_lds_with(int32_t max_k, int32_t max_m, int32_t w, int tb, int tstride) {
    LdsPlan p;
    size_t off = 0;
    p.tstride = tstride;
    p.tslot = off;
    off = align16(off + 4 * ((size_t)max_m + 2 * kTPad) * tstride);
    p.tlen = off;
    off = align16(off + (size_t)max_m + 2 * kTPad);
    p.dslot = off;
    off = align16(off + (size_t)max_k * tb);
    p.dlen = off;
    off = align16(off + (size_t)max_k);
    p.row0 = off;
    off = align16(off + 4 * ((size_t)kRowFront + max_m + kRowBack));
    p.row1 = off;
    off = align16(off + 4 * ((size_t)kRowFront + max_m + kRowBack));
    // distances of two chunks during the sweep; two strips of code words during the
    // backtrack when a row has at most 64 of them
    const int rw = row_words_bound(max_k, max_m, w);
    const size_t cost_bytes = 2 * 4 * (size_t)kWave * kCostStride;
    const size_t stage_bytes = rw <= kWave ? 2 * 4 * (size_t)kWave * rw : 0;
    p.cost = off;
    off = align16(off + (cost_bytes > stage_bytes ? cost_bytes : stage_bytes));
    p.path = off;
    off = align16(off + 8 * (size_t)max_k);
    p.total = off;
    return p;
}

__host__ __device__ inline LdsPlan plan_lds(int32_t max_k, int32_t max_m, int32_t w, int tb) {
    const LdsPlan wide = plan_lds_with(max_k, max_m, w, tb, tb / 4 + 1);
    return wide.total <= kLdsLimit ? wide : plan_lds_with(max_k, max_m, w, tb, tb / 4);
}

struct Band {
    int K, M, L, W;
    __device__ __forceinline__ int jlo(int i) const { return (i - L) > 1 ? (i - L) : 1; }
    __device__ __forceinline__ int jhi(int i) const { return (i + L) < M ? (i + L) : M; }
};

// Geometry of the strip starting at draft row i0.
struct Strip {
    int i0, R, jfirst, nchunks;
};

__device__ __forceinline__ Strip strip_at(const Band &g, int s) {
    Strip st;
    st.i0 = 1 + s * kWave;
    st.R = (g.K - st.i0 + 1) < kWave ? (g.K - st.i0 + 1) : kWave;
    st.jfirst = g.jlo(st.i0);
    const int steps = (g.jhi(st.i0 + st.R - 1) - st.jfirst + 1) + st.R - 1;
    st.nchunks = (steps + kChunk - 1) / kChunk;
    return st;
}

// Bits 0 .. n-1 set (n <= 32).
__device__ __forceinline__ uint32_t low_mask(int n) { return n >= 32 ? 0xFFFFFFFFu : ((1u << n) - 1u); }

// Edit distance between a draft token of at most two bytes (the text, xm bytes: c1 = byte 0
// broadcast in bc1, c2 = byte 1 in bc2) and a target token (the pattern, yn bytes in yw, lim
// its bit mask), in closed form over the pattern positions E1, E2 that equal c1, c2:
//   xm = 0 or yn = 0   d = xm + yn
//   xm = 1             d = yn - [E1 != 0]
//   xm = 2, yn = 1     d = 2 - [E1 | E2 != 0]
//   xm = 2, yn >= 2    d = yn - 2 + (0 if some a < b has E1[a] and E2[b];
//                                    1 else if E1 has a bit below yn - 1 or E2 a bit above 0;
//                                    2 else)
// (for yn >= 2 the two text bytes go to two increasing pattern positions, the other yn - 2
// bytes are deleted, and each costs 1 unless it matches; an alignment that inserts a text
// byte costs at least yn).
template <int TB>
__device__ __forceinline__ uint32_t closed_distance(const uint32_t (&yw)[TB / 4], int yn, uint32_t lim, uint32_t bc1,
                                                    uint32_t bc2, int xm) {
    const uint32_t e1 = dtw::match_mask<TB>(yw, bc1) & lim;
    const uint32_t e2 = dtw::match_mask<TB>(yw, bc2) & lim;
    const uint32_t low1 = e1 & (0u - e1);                   // lowest position matching c1
    const bool in_order = (e2 & ~((low1 << 1) - 1u)) != 0;  // c2 matches further on
    const bool one = (e1 & (lim >> 1)) != 0 || (e2 & ~1u) != 0;
    const uint32_t two = yn - 2 + (in_order ? 0u : (one ? 1u : 2u));
    const uint32_t d2 = yn == 1 ? 2u - ((e1 | e2) != 0 ? 1u : 0u) : two;
    const uint32_t d1 = (uint32_t)yn - (e1 != 0 ? 1u : 0u);
    return (xm == 0 || yn == 0) ? (uint32_t)(xm + yn) : (xm == 1 ? d1 : d2);
}

// The same distance by Myers' recurrence with D(0, j) = j over the text's bytes, read at the
// end from the vertical deltas; the loop leaves once no lane of the wave has bytes left.
template <int TB>
__device__ __forceinline__ uint32_t myers_distance(const uint32_t (&pw)[TB / 4], const uint32_t (&tw)[TB / 4], int tn,
                                                   uint32_t lim) {
    uint32_t vp = 0xFFFFFFFFu, vn = 0;
#pragma unroll
    for (int k = 0; k < TB; ++k) {
        const bool act = k < tn;
        if (!__any(act)) break;
        const uint32_t bc = __builtin_amdgcn_perm(0u, tw[k >> 2], (uint32_t)(k & 3) * 0x01010101u);
        const uint32_t eq = dtw::match_mask<TB>(pw, bc) & lim;
        const uint32_t xv = eq | vn;
        const uint32_t xh = (((eq & vp) + vp) ^ vp) | eq;
        const uint32_t hp = ((vn | ~(xh | vp)) << 1) | 1u;
        const uint32_t hn = (vp & xh) << 1;
        const uint32_t nvp = hn | ~(xv | hp);
        const uint32_t nvn = hp & xv;
        vp = act ? nvp : vp;
        vn = act ? nvn : vn;
    }
    return (uint32_t)(tn + __popc(vp & lim) - __popc(vn & lim));
}

// Token distances of chunk T0 / 64 of strip st: cell (i0 + r, jfirst + t - r) for
// t in [T0, T0 + 64) goes to byte t & 3 of dword buf[r][(t - T0) / 4]; out-of-band
// cells get 0x80.  Threads h, h + nh, ... each take four consecutive steps of one row, and
// consecutive threads consecutive steps: a wave's lanes then leave the band together
// (rows in consecutive lanes would diverge at every band edge).  The four cells of a thread
// load their target tokens together (columns clamped into [1, M], results masked) and take
// the closed form with the draft token as the text unless some lane of the wave has a draft
// token of more than two bytes.
template <int TB>
__device__ __forceinline__ void chunk_costs(const Band &g, const Strip &st, int T0, uint32_t *buf,
                                            const uint32_t *tslot, int ts, const uint8_t *tlen, const uint32_t *dslot,
                                            const uint8_t *dlen, int h, int nh) {
    for (int item = h; item < st.R * kGroups; item += nh) {
        const int r = item / kGroups, gq = item % kGroups;
        const int i = st.i0 + r;
        const int jl = g.jlo(i), jh = g.jhi(i);
        const int jb = st.jfirst + T0 + 4 * gq - r;  // column of the item's first step
        uint32_t packed = kOutOfBand;
        if (jb <= jh && jb + 3 >= jl) {
            uint32_t xw[TB / 4];
            read_slot<TB>(dslot + (i - 1) * (TB / 4), xw);
            const int xm = dlen[i - 1];
            if constexpr (TB <= 32) {
                const bool closed = !__any(xm > 2);  // uniform: the wave's draft tokens have at most two bytes
                const uint32_t bc1 = __builtin_amdgcn_perm(0u, xw[0], 0u);
                const uint32_t bc2 = __builtin_amdgcn_perm(0u, xw[0], 0x01010101u);
                constexpr int kBatch = TB <= 8 ? 4 : 1;  // target slots loaded together (within 64 VGPRs)
                uint32_t d[4];
#pragma unroll
                for (int u0 = 0; u0 < 4; u0 += kBatch) {
                    uint32_t yw[kBatch][TB / 4];
                    int yn[kBatch];
#pragma unroll
                    for (int v = 0; v < kBatch; ++v) {  // jb - 1 + kTPad >= 0: the item meets the band
                        const int sl = jb + u0 + v - 1 + kTPad;
                        read_slot<TB>(tslot + sl * ts, yw[v]);
                        yn[v] = tlen[sl];
                    }
#pragma unroll
                    for (int v = 0; v < kBatch; ++v) {
                        if (closed) {
                            d[u0 + v] = closed_distance<TB>(yw[v], yn[v], low_mask(yn[v]), bc1, bc2, xm);
                        } else {
                            const bool swap = yn[v] > xm;
                            uint32_t pw[TB / 4], tw[TB / 4];
#pragma unroll
                            for (int q = 0; q < TB / 4; ++q) {
                                pw[q] = swap ? yw[v][q] : xw[q];
                                tw[q] = swap ? xw[q] : yw[v][q];
                            }
                            d[u0 + v] = myers_distance<TB>(pw, tw, swap ? xm : yn[v], low_mask(swap ? yn[v] : xm));
                        }
                    }
                }
                packed = 0;
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int j = jb + u;
                    packed |= ((j >= jl && j <= jh) ? d[u] : 0x80u) << (8 * u);
                }
            } else {
#pragma unroll 1
                for (int u = 0; u < 4; ++u) {
                    const int j = jb + u;
                    if (j >= jl && j <= jh) {
                        uint32_t yw[TB / 4];
                        read_slot<TB>(tslot + (j - 1 + kTPad) * ts, yw);
                        const uint32_t d = (uint32_t)token_distance<TB>(xw, xm, yw, tlen[j - 1 + kTPad]);
                        packed = (packed & ~(0xFFu << (8 * u))) | (d << (8 * u));
                    }
                }
            }
        }
        buf[r * kCostStride + gq] = packed;
    }
}

// Per-lane state of the strip sweep (wave 0, lane r = row i0 + r).
struct Sweep {
    int cur;         // C of the lane's latest cell
    int above_prev;  // C(i-1, j-1) of the next cell
    uint32_t cw;     // predecessor codes of the latest 16 steps
    uint32_t oob;    // kOutOfBand for lanes past the strip's last row
    int kr0;         // first stored code word of the row (in steps / 16 of the strip)
    bool act, last;
    uint32_t *prow;  // the row's code words in the workspace
};

// Steps T0 .. T0 + 63 of the sweep.  rowIn / rowOut point at column 0 of the row buffers,
// which are infinite past column M far enough for lane 0's reads of C(i0 - 1, j).
__device__ __forceinline__ void sweep_chunk(Sweep &sw, const uint32_t *buf, const int *rowIn, int *rowOut, int T0,
                                            int jfirst, int rw) {
    const int lane = threadIdx.x;
    const uint32_t *myc = buf + lane * kCostStride;
    const int *rin = rowIn + jfirst + T0;  // lane 0's C(i0 - 1, j) at the chunk's steps
    uint32_t dw = myc[0] | sw.oob;
    int rv[4] = {rin[0], rin[1], rin[2], rin[3]};
#pragma unroll
    for (int gq = 0; gq < kGroups; ++gq) {
        // the next group's inputs (the last group reads the buffer's pad column)
        const uint32_t dwn = myc[gq + 1] | sw.oob;
        const int rvn[4] = {rin[4 * gq + 4], rin[4 * gq + 5], rin[4 * gq + 6], rin[4 * gq + 7]};
        int c[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int d = ((int)(dw << (24 - 8 * u))) >> 24;  // negative outside the band
            const int above = __builtin_amdgcn_update_dpp(rv[u], sw.cur, 0x138 /* wave_shr:1 */, 0xF, 0xF, false);
            const int diag = sw.above_prev;
            sw.above_prev = above;
            // ties: diagonal, then (i-1, j), then (i, j-1); each choice bit is the sign of a
            // difference shifted into the code word (values stay below 2^31)
            const int m1 = above < diag ? above : diag;
            sw.cw = __builtin_amdgcn_alignbit(sw.cw, (uint32_t)(above - diag), 31);  // up
            sw.cw = __builtin_amdgcn_alignbit(sw.cw, (uint32_t)(sw.cur - m1), 31);   // left
            const int best = sw.cur < m1 ? sw.cur : m1;
            sw.cur = d < 0 ? kInf : d + best;
            c[u] = sw.cur;
        }
        // keep the code word current every group: left to itself the compiler defers the
        // choice bits of 16 steps to the store and holds all their operands live
        asm volatile("" : "+v"(sw.cw));
        if (sw.last) {  // the strip's last row feeds the next strip
            int *dst = rowOut + (jfirst + T0 + 4 * gq - lane);
            dst[0] = c[0];
            dst[1] = c[1];
            dst[2] = c[2];
            dst[3] = c[3];
        }
        if ((gq & 3) == 3) {  // 16 steps make code word k of the row
            const int k = (T0 >> 4) + (gq >> 2) - sw.kr0;
            if (sw.act && (unsigned)k < (unsigned)rw) sw.prow[k] = sw.cw;
        }
        dw = dwn;
#pragma unroll
        for (int u = 0; u < 4; ++u) rv[u] = rvn[u];
    }
}

template <int TB, int TS>
__global__ void __launch_bounds__(band_threads<TB>()) __attribute__((amdgpu_waves_per_eu(band_threads<TB>() / 64)))
dtw_band(AlignArgs a, LdsPlan lp, uint32_t *gcodes, size_t gcode_stride,
                                                     int rw, const int32_t *order) {
    constexpr int kThreads = band_threads<TB>();
    constexpr int kHelpers = kThreads - kWave;
    extern __shared__ __align__(16) uint8_t lds[];
    const int b = order != nullptr ? order[blockIdx.x] : (int)blockIdx.x;  // pairs in descending work
    const int tid = threadIdx.x, lane = tid % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);  // uniform: wave-level branches stay scalar
    const int d0 = a.draft_off[b], K = a.draft_off[b + 1] - d0;
    const int t0 = a.target_off[b], M = a.target_off[b + 1] - t0;

    uint32_t *tslot = reinterpret_cast<uint32_t *>(lds + lp.tslot);
    constexpr int ts = TS;  // dwords per target token slot (lp.tstride)
    uint8_t *tlen = lds + lp.tlen;
    uint32_t *dslot = reinterpret_cast<uint32_t *>(lds + lp.dslot);
    uint8_t *dlen = lds + lp.dlen;
    int *rowIn = reinterpret_cast<int *>(lds + lp.row0) + kRowFront;
    int *rowOut = reinterpret_cast<int *>(lds + lp.row1) + kRowFront;
    uint32_t *costbuf = reinterpret_cast<uint32_t *>(lds + lp.cost);  // two halves of kWave * kCostStride
    uint32_t *seg = reinterpret_cast<uint32_t *>(lds + lp.path);  // [K]: first column << 16 | entry column
    uint32_t *poff = seg + a.max_k;                               // [K]: index of the row's first path cell
    __shared__ int votes[kThreads / kWave];
    __shared__ int s_imin, s_n;

    // ---- staging + validation: one token (draft or target) per thread and pass
    const bool shape_ok = K >= 1 && K <= a.max_k && M >= 1 && M <= a.max_m;
    int bad = shape_ok ? 0 : 1;
    if (shape_ok) {
        for (int e = tid; e < K + M; e += kThreads) {
            const bool ok = e < K ? stage_token<TB>(a.vd, a.draft_ids[d0 + e], dslot + e * (TB / 4), dlen + e)
                                  : stage_token<TB>(a.vt, a.target_ids[t0 + e - K], tslot + (e - K + kTPad) * ts,
                                                    tlen + (e - K + kTPad));
            bad |= ok ? 0 : 1;
        }
        // the empty slots around the target tokens (read by items that straddle the band's ends)
        if (tid < 2 * kTPad * ts) {
            const int sl = tid / ts, q = tid % ts;
            const int slot = sl < kTPad ? sl : M + sl;  // 0 .. kTPad-1 and M + kTPad .. M + 2 kTPad - 1
            tslot[slot * ts + q] = 0u;
            if (q == 0) tlen[slot] = 0;
        }
    }
    if (dtw::block_or(bad, votes, kThreads / kWave)) {
        if (tid == 0) {
            a.cost[b] = -1;
            a.path_len[b] = 0;
        }
        for (int j = tid; j < M; j += kThreads) a.map[t0 + j] = -1;
        return;
    }

    // ---- band geometry for this pair
    Band g;
    g.K = K;
    g.M = M;
    const int mx = K > M ? K : M;
    g.L = (a.w < 0) ? mx : (a.w > abs(K - M) ? a.w : abs(K - M));
    if (g.L > mx) g.L = mx;
    g.W = (2 * g.L + 1 < M) ? 2 * g.L + 1 : M;
    const int nstrips = (K + kWave - 1) / kWave;
    uint32_t *parked = gcodes + (size_t)b * gcode_stride;  // code words of row i at (i - 1) * rw

    // ---- chunked sweep: wave 0 sweeps a chunk while waves 1-3 evaluate the next one
    if (wave == 0) {
        for (int j = lane - kRowFront; j < M + kRowBack; j += kWave) {
            rowIn[j] = (j == 0) ? 0 : kInf;  // C(0, j)
            rowOut[j] = kInf;
        }
    }
    Strip st = strip_at(g, 0);
    chunk_costs<TB>(g, st, 0, costbuf, tslot, ts, tlen, dslot, dlen, tid, kThreads);
    __syncthreads();
    // the sweep is the critical path: its wave wins issue arbitration on its SIMD
    if (wave == 0) __builtin_amdgcn_s_setprio(3);
    int gidx = 0;  // chunks swept so far (selects the buffer half)
    Sweep sw;
    for (int s = 0; s < nstrips; ++s) {
        if (wave == 0) {
            const int i = st.i0 + lane;
            sw.act = lane < st.R;
            sw.last = lane == st.R - 1;
            sw.oob = sw.act ? 0u : kOutOfBand;
            sw.kr0 = sw.act ? (g.jlo(i) - st.jfirst + lane) >> 4 : 0;
            sw.prow = parked + (size_t)(sw.act ? i - 1 : 0) * rw;
            sw.cur = kInf;
            sw.above_prev = (lane == 0) ? rowIn[st.jfirst - 1] : kInf;
            sw.cw = 0;
        }
        const Strip nxt = (s + 1 < nstrips) ? strip_at(g, s + 1) : st;
        for (int c = 0; c < st.nchunks; ++c) {
            uint32_t *cur_buf = costbuf + (gidx & 1) * kWave * kCostStride;
            uint32_t *next_buf = costbuf + ((gidx + 1) & 1) * kWave * kCostStride;
            if (wave == 0) {
                sweep_chunk(sw, cur_buf, rowIn, rowOut, c * kChunk, st.jfirst, rw);
            } else if (c + 1 < st.nchunks) {
                chunk_costs<TB>(g, st, (c + 1) * kChunk, next_buf, tslot, ts, tlen, dslot, dlen, tid - kWave, kHelpers);
            } else if (s + 1 < nstrips) {
                chunk_costs<TB>(g, nxt, 0, next_buf, tslot, ts, tlen, dslot, dlen, tid - kWave, kHelpers);
            }
            __syncthreads();
            ++gidx;
        }
        int *tmp = rowIn;  // the strip's last row is the next strip's row above
        rowIn = rowOut;
        rowOut = tmp;
        if (wave == 0 && s + 1 < nstrips) {
            for (int j = lane - kRowFront; j < M + kRowBack; j += kWave) rowOut[j] = kInf;
        }
        st = nxt;
    }

    // ---- backtrack (wave 0): inside row i the path runs left from its entry column e to
    // the highest column x <= e whose move is not (i, j-1); it enters row i-1 at x - 1
    // after a diagonal move and at x after an (i-1, j) move
    __builtin_amdgcn_s_waitcnt(0);  // wave 0's code-word stores are complete before they are read back
    const int cost_km = wave == 0 ? rowIn[M] : 0;  // C(K, M), read before the row buffers are reused
    int e = M;      // entry column of the row being walked (uniform over wave 0)
    int first = 1;  // first row on the path
    // Wave 0 walks rows rtop down to i0 of one strip with uniform (scalar) state; word(rr, k)
    // is code word k of row i0 + rr, read by every lane at the same address.  The run of
    // row i0 + l is recorded in lane l and the strip's records are written at the end.
    // Returns true while the path goes on below the strip.
    auto walk_strip = [&](int i0, int rtop, auto word) -> bool {
        const int jf = g.jlo(i0);
        uint32_t rec = 0;
        bool more = true;
        int r = rtop;
        for (; r >= i0; --r) {
            const int rr = r - i0;
            const int kr0 = (g.jlo(r) - jf + rr) >> 4;  // the row's first code word, in strip steps / 16
            const int te = e - jf + rr;                 // sweep step of the entry cell
            int k = (te >> 4) - kr0;
            // the checks below never fire on codes the sweep wrote (the entry column lies inside
            // the row's band, and the band's first cell is not a left move); they are folded into
            // one flag so the walk's dependent chain has a single branch per row
            int bad = (uint32_t)k >= (uint32_t)rw ? 1 : 0;
            k = bad ? 0 : k;
            uint32_t w = __builtin_amdgcn_readfirstlane(word(rr, k));
            // cells whose move is not (i, j-1), at steps <= te
            uint32_t m = ~w & 0x55555555u & (0xFFFFFFFFu << (30 - 2 * (te & 15)));
            if (m == 0u) {
                while (m == 0u && k > 0) {  // the run continues into the word below
                    --k;
                    w = __builtin_amdgcn_readfirstlane(word(rr, k));
                    m = ~w & 0x55555555u;
                }
                bad |= m == 0u ? 1 : 0;
            }
            const int pos = m != 0u ? __builtin_ctz(m) : 0;
            const int x = jf + 16 * (kr0 + k) + ((30 - pos) >> 1) - rr;
            rec = lane == rr ? (((uint32_t)x << 16) | (uint32_t)e) : rec;
            e = x - (int)((~w >> (pos + 1)) & 1u);  // x after an (i-1, j) move, x - 1 after a diagonal
            if ((bad | (e < 1 ? 1 : 0) | (r == 1 ? 1 : 0)) != 0) {
                more = false;
                r -= bad ? 0 : 1;  // a bad row is not on the path; otherwise this row was the last
                break;
            }
        }
        // rows r + 1 .. rtop were walked
        if (lane + i0 > r && lane + i0 <= rtop) seg[i0 - 1 + lane] = rec;
        if (!more) first = r + 1;
        return more;
    };
    // One row of the walk for any row r (the code words' step numbering is that of the 64-row
    // strip holding r): entry column e, the row's code words at rowwords; returns the entry
    // column of row r - 1 and the row's run record, and raises bad on codes the sweep cannot
    // have written (see walk_strip).
    auto row_step = [&](int r, int ein, const uint32_t *rowwords, uint32_t &rec_out, int &bad) -> int {
        const int i0s = 1 + ((r - 1) & ~(kWave - 1));
        const int rr = r - i0s;
        const int jf = g.jlo(i0s);
        const int kr0 = (g.jlo(r) - jf + rr) >> 4;
        const int te = ein - jf + rr;
        int k = (te >> 4) - kr0;
        bad = (uint32_t)k >= (uint32_t)rw ? 1 : 0;
        k = bad ? 0 : k;
        uint32_t w = __builtin_amdgcn_readfirstlane(rowwords[k]);
        uint32_t m = ~w & 0x55555555u & (0xFFFFFFFFu << (30 - 2 * (te & 15)));
        if (m == 0u) {
            while (m == 0u && k > 0) {
                --k;
                w = __builtin_amdgcn_readfirstlane(rowwords[k]);
                m = ~w & 0x55555555u;
            }
            bad |= m == 0u ? 1 : 0;
        }
        const int pos = m != 0u ? __builtin_ctz(m) : 0;
        const int x = jf + 16 * (kr0 + k) + ((30 - pos) >> 1) - rr;
        rec_out = ((uint32_t)x << 16) | (uint32_t)ein;
        return x - (int)((~w >> (pos + 1)) & 1u);
    };
    // Segment-parallel walk (code words of up to 64 rows per segment staged in LDS): the rows
    // are cut into segments of kSeg; a group of segments is staged into the LDS the sweep no
    // longer needs (token tables, row buffers, distance buffers), and every wave walks one
    // segment at the same time, the topmost from its known entry column and the others from a
    // guess on the line from (1, 1) to (K, M), recording each row's entry column (in poff) and
    // run (in seg).  Wave 0 then corrects the segments top-down: entering a segment at its true
    // column it re-walks rows only until its entry column meets the recorded one; from there the
    // recorded walk is the true walk, because a row's exit depends only on its entry column.
    // Optimal paths from nearby columns merge within a few rows, so the correction is short.
    constexpr int kSeg = 32;
    constexpr int kWaves = kThreads / kWave;
    uint32_t *scr = reinterpret_cast<uint32_t *>(lds + lp.tslot);
    const int scr_words = (int)((lp.path - lp.tslot) / 4);
    int par = scr_words / (kSeg * rw);
    par = par < kWaves ? par : kWaves;
    __shared__ int s_exit[kWaves], s_more, s_first, s_etrue;
    if (rw <= kWave && par >= 2 && K > kSeg) {
        const int nseg = (K + kSeg - 1) / kSeg;
        if (tid == 0) {
            s_more = 1;
            s_first = 1;
            s_etrue = M;
        }
        for (int top = nseg - 1; top >= 0; top -= par) {
            __syncthreads();  // s_more / s_etrue published; the previous group's buffers are free
            if (!s_more) break;  // uniform
            const int nsg = top + 1 < par ? top + 1 : par;
            const int sg = top - wave;  // this wave's segment
            const int lo = sg * kSeg + 1;
            const int hi = (lo + kSeg - 1) < K ? (lo + kSeg - 1) : K;
            uint32_t *buf = scr + wave * kSeg * rw;
            if (wave < nsg) {
                const uint32_t *src = parked + (size_t)(lo - 1) * rw;
                for (int q = lane; q < (hi - lo + 1) * rw; q += kWave) buf[q] = src[q];
            }
            __syncthreads();
            if (wave < nsg) {  // speculative walk of the segment, uniform state per wave
                int ew;
                if (wave == 0) {
                    ew = s_etrue;
                } else {  // the line from (1, 1) to (K, M), clamped into row hi's band
                    ew = 1 + (int)(((long long)(hi - 1) * (M - 1)) / (K - 1));
                    ew = ew < g.jlo(hi) ? g.jlo(hi) : (ew > g.jhi(hi) ? g.jhi(hi) : ew);
                }
                uint32_t rec = 0, ent = 0;
                int badw = 0;
                for (int r = hi; r >= lo; --r) {
                    uint32_t rc;
                    int bad;
                    const int en = row_step(r, ew, buf + (r - lo) * rw, rc, bad);
                    ent = lane == r - lo ? (uint32_t)ew : ent;
                    rec = lane == r - lo ? rc : rec;
                    if (bad) {
                        badw = 1;
                        break;
                    }
                    ew = en;
                    if (r == 1) break;
                }
                if (lane < hi - lo + 1) {
                    seg[lo - 1 + lane] = rec;
                    poff[lo - 1 + lane] = badw ? 0xFFFFFFFFu : ent;  // never an entry column: forces a re-walk
                }
                if (lane == 0) s_exit[wave] = ew;
            }
            __syncthreads();
            if (wave == 0) {  // corrections, top-down
                int et = s_etrue;
                bool more = true;
                int fst = 1;
                for (int w = 0; w < nsg && more; ++w) {
                    const int lo2 = (top - w) * kSeg + 1;
                    const int hi2 = (lo2 + kSeg - 1) < K ? (lo2 + kSeg - 1) : K;
                    const uint32_t *b2 = scr + w * kSeg * rw;
                    bool met = false;
                    for (int r = hi2; r >= lo2; --r) {
                        if ((uint32_t)et == poff[r - 1]) {  // the recorded walk is the true walk from here
                            met = true;
                            break;
                        }
                        uint32_t rc;
                        int bad;
                        const int en = row_step(r, et, b2 + (r - lo2) * rw, rc, bad);
                        if (bad) {  // as in walk_strip: row r is not on the path
                            more = false;
                            fst = r + 1;
                            break;
                        }
                        if (lane == 0) {
                            seg[r - 1] = rc;
                            poff[r - 1] = (uint32_t)et;
                        }
                        et = en;
                        if (et < 1 || r == 1) {
                            more = false;
                            fst = r;
                            break;
                        }
                    }
                    if (met) {
                        et = s_exit[w];
                        if (lo2 == 1) more = false;  // the recorded walk reached row 1
                    } else if (more && lo2 == 1) {
                        more = false;
                    }
                }
                if (lane == 0) {
                    s_etrue = et;
                    s_more = more ? 1 : 0;
                    if (!more) s_first = fst;
                }
            }
        }
        __syncthreads();
        first = s_first;
    } else if (rw <= kWave) {
        // each strip's code words are staged into the freed cost buffers by the other waves
        // while wave 0 walks the strip below it in the other half
        uint32_t *stg = costbuf;
        auto copy_strip = [&](int s, int h, int nh) {
            const int i0 = 1 + s * kWave;
            const int R = (K - i0 + 1) < kWave ? (K - i0 + 1) : kWave;
            const uint32_t *src = parked + (size_t)(i0 - 1) * rw;
            uint32_t *dst = stg + (s & 1) * kWave * rw;
            for (int e2 = h; e2 < R * rw; e2 += nh) dst[e2] = src[e2];
        };
        copy_strip(nstrips - 1, tid, kThreads);
        __syncthreads();
        bool walking = true;  // uniform over wave 0
        for (int s = nstrips - 1; s >= 0; --s) {
            if (wave != 0) {
                if (s >= 1) copy_strip(s - 1, tid - kWave, kHelpers);
            } else if (walking) {
                const int i0 = 1 + s * kWave;
                const uint32_t *half = stg + (s & 1) * kWave * rw;
                const int rtop = (K < i0 + kWave - 1) ? K : i0 + kWave - 1;
                walking = walk_strip(i0, rtop, [&](int rr, int k) { return half[rr * rw + k]; });
            }
            __syncthreads();
        }
    } else if (wave == 0) {
        // rows of more than 64 code words: read straight from the workspace
        for (int s = nstrips - 1; s >= 0; --s) {
            const int i0 = 1 + s * kWave;
            const int rtop = (K < i0 + kWave - 1) ? K : i0 + kWave - 1;
            auto word = [&](int rr, int k) { return parked[(size_t)(i0 - 1 + rr) * rw + k]; };
            if (!walk_strip(i0, rtop, word)) break;
        }
    }
    if (wave == 0) {
        if (lane == 0) a.cost[b] = cost_km;  // C(K, M), from the last strip's last row
        // rows first..K are on the path: path offsets
        int carry = 0;
        for (int r0 = first - 1; r0 < K; r0 += kWave) {
            const int r = r0 + lane;
            const uint32_t sv = r < K ? seg[r] : 0u;
            const int len = r < K ? (int)(sv & 0xFFFFu) - (int)(sv >> 16) + 1 : 0;
            const int incl = dtw::wave_prefix_sum(len) + carry;
            if (r < K) poff[r] = (uint32_t)(incl - len);
            carry = __builtin_amdgcn_readlane(incl, kWave - 1);
        }
        if (lane == 0) {
            s_imin = first;
            s_n = carry;
            a.path_len[b] = carry;
        }
    }
    __syncthreads();
    const int imin = s_imin;
    const int n = s_n < K + M - 1 ? s_n : K + M - 1;  // a path has at most K + M - 1 cells
    // ---- path cells and map entries, all threads: binary searches over the rows' runs
    int32_t *pp = a.path + 2 * ((size_t)d0 + (size_t)t0);
    for (int q = tid; q < n; q += kThreads) {
        int lo = imin - 1, hi = K - 1;  // last row r with poff[r] <= q
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if ((int)poff[mid] <= q) lo = mid;
            else hi = mid - 1;
        }
        const int x = (int)(seg[lo] >> 16);
        pp[2 * q] = lo;
        pp[2 * q + 1] = x - 1 + (q - (int)poff[lo]);
    }
    for (int j = tid + 1; j <= M; j += kThreads) {
        int lo = imin - 1, hi = K - 1;  // last row r whose run starts at or before column j
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if ((int)(seg[mid] >> 16) <= j) lo = mid;
            else hi = mid - 1;
        }
        a.map[t0 + j - 1] = lo;
    }
}

// Dispatch order for the strip kernel: pairs by descending band work K * W (in units of 16
// cells), ties by index.  Workgroups are handed to compute units in launch order, so the
// longest pairs start first and the short ones fill in around them (on the 1,024 long pairs:
// 393 us in generator order, about 254 us sorted).  Every 256-thread workgroup builds all n
// 32-bit keys (work class, index) in LDS and ranks its own 64 pairs: a pair's slot is the number
// of keys below its own, counted by four lanes over a quarter of the keys each with broadcast
// LDS reads.
__device__ __forceinline__ uint32_t order_key(const AlignArgs &a, int i) {
    const int K = a.draft_off[i + 1] - a.draft_off[i], M = a.target_off[i + 1] - a.target_off[i];
    uint32_t work = 0;
    if (K >= 1 && K <= a.max_k && M >= 1 && M <= a.max_m) {
        const int mx = K > M ? K : M;
        int L = a.w < 0 ? mx : (a.w > abs(K - M) ? a.w : abs(K - M));
        L = L < mx ? L : mx;
        const int W = 2 * L + 1 < M ? 2 * L + 1 : M;
        work = ((uint32_t)K * (uint32_t)W) >> 4;  // <= 4096 * 4096 / 16 = 2^20
    }
    work = work < 0xFFFFFu ? work : 0xFFFFFu;
    return ((0xFFFFFu - work) << 11) | (uint32_t)i;  // 20 + 11 bits: unique for i < 2048
}

__global__ void __launch_bounds__(kOrderThreads) order_pairs(AlignArgs a, int32_t *order) {
    __shared__ __align__(16) uint32_t keys[kOrderMax];
    const int n = a.n_pairs;
    const int n16 = (n + 15) & ~15;
    for (int i = threadIdx.x; i < n16; i += kOrderThreads) keys[i] = i < n ? order_key(a, i) : ~0u;  // pad: never below a key
    __syncthreads();
    const uint4 *k4 = reinterpret_cast<const uint4 *>(keys);
    // four lanes per pair, each counting a quarter of the keys; partial counts meet by shuffles
    const int i = blockIdx.x * kOrderPairsPerGroup + (int)threadIdx.x / kOrderSplit;
    const int part = threadIdx.x % kOrderSplit;
    const uint32_t mine = i < n ? keys[i] : 0u;
    const int quads = n16 >> 2;  // a multiple of 4
    const int per = ((quads / kOrderSplit) + 3) & ~3;
    const int q0 = part * per;
    const int q1 = q0 + per < quads ? q0 + per : quads;
    int r = 0;
    for (int q = q0; q < q1; q += 4) {  // every lane of a quarter reads the same 16 keys
        uint4 k[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) k[u] = q + u < q1 ? k4[q + u] : make_uint4(~0u, ~0u, ~0u, ~0u);
#pragma unroll
        for (int u = 0; u < 4; ++u) r += (k[u].x < mine) + (k[u].y < mine) + (k[u].z < mine) + (k[u].w < mine);
    }
    r += __shfl_xor(r, 1);
    r += __shfl_xor(r, 2);
    if (i < n && part == 0) order[r] = i;
}

inline size_t order_offset(size_t code_words) { return (4 * code_words + 255) & ~size_t(255); }

template <int TB>
int launch_tb(const AlignArgs &a, void *workspace, size_t workspace_bytes, hipStream_t stream) {
    const LdsPlan lp = plan_lds(a.max_k, a.max_m, a.w, TB);
    if (lp.total > kLdsLimit) return TT_EUNSUPPORTED;
    const int rw = row_words_bound(a.max_k, a.max_m, a.w);
    const size_t stride = (size_t)a.max_k * (size_t)rw;  // code words per pair
    const bool sorted = a.n_pairs >= 2 && a.n_pairs <= kOrderMax;
    const size_t need = sorted ? order_offset(stride * (size_t)a.n_pairs) + 4 * (size_t)a.n_pairs
                               : 4 * stride * (size_t)a.n_pairs;
    if (workspace == nullptr || workspace_bytes < need) return TT_EWORKSPACE;
    int32_t *order = nullptr;
    if (sorted) {
        order = reinterpret_cast<int32_t *>(static_cast<uint8_t *>(workspace) + order_offset(stride * (size_t)a.n_pairs));
        hipLaunchKernelGGL(order_pairs, dim3((a.n_pairs + kOrderPairsPerGroup - 1) / kOrderPairsPerGroup),
                           dim3(kOrderThreads), 0, stream, a, order);
        if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
    }
    auto launch = [&](auto kernel) -> int {
        if (lp.total > 64 * 1024 &&
            hipFuncSetAttribute(reinterpret_cast<const void *>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)lp.total) != hipSuccess)
            return TT_ELAUNCH;
        hipLaunchKernelGGL(kernel, dim3(a.n_pairs), dim3(band_threads<TB>()), lp.total, stream, a, lp,
                           static_cast<uint32_t *>(workspace), stride, rw, order);
        return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
    };
    return lp.tstride == TB / 4 + 1 ? launch(&dtw_band<TB, TB / 4 + 1>) : launch(&dtw_band<TB, TB / 4>);
}

}  // namespace

int align_token_slot(int32_t max_token_bytes) {
    if (max_token_bytes < 1) return 0;
    if (max_token_bytes <= 8) return 8;
    if (max_token_bytes <= 16) return 16;
    if (max_token_bytes <= 32) return 32;
    if (max_token_bytes <= 64) return 64;
    return 0;
}

size_t align_lds_bytes(int32_t max_k, int32_t max_m, int32_t w, int tb) {
    const LdsPlan lp = plan_lds(max_k, max_m, w, tb);
    return lp.total > kLdsLimit ? 0 : lp.total;
}

size_t align_workspace_bytes(int32_t n_pairs, int32_t max_k, int32_t max_m, int32_t w) {
    if (TT_ALIGN_ROWS && align_rows_fits(max_k, max_m)) return 0;
    const size_t words = (size_t)n_pairs * (size_t)max_k * (size_t)row_words_bound(max_k, max_m, w);
    if (n_pairs >= 2 && n_pairs <= kOrderMax) return order_offset(words) + 4 * (size_t)n_pairs;
    return 4 * words;
}

int launch_align(const AlignArgs &a, void *workspace, size_t workspace_bytes, hipStream_t stream) {
    const int mt = a.vd.max_token_bytes > a.vt.max_token_bytes ? a.vd.max_token_bytes : a.vt.max_token_bytes;
    const int tb = align_token_slot(mt);
    if (TT_ALIGN_ROWS && align_rows_fits(a.max_k, a.max_m)) return launch_align_rows(a, tb, stream);
    switch (tb) {
        case 8: return launch_tb<8>(a, workspace, workspace_bytes, stream);
        case 16: return launch_tb<16>(a, workspace, workspace_bytes, stream);
        case 32: return launch_tb<32>(a, workspace, workspace_bytes, stream);
        case 64: return launch_tb<64>(a, workspace, workspace_bytes, stream);
        default: return TT_EUNSUPPORTED;
    }
}

}  // namespace tt
