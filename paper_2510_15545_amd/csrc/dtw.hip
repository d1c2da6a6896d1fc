// Dynamic Token Warping on gfx950 for pairs of any length: one 1024-thread workgroup
// per (draft, proxy-target) pair.
//
// Computes Alg. 1 of the paper (cumulative cost C over draft x target tokens with
// the Sakoe-Chiba band, Sec. 4.1) using the byte-level Levenshtein token distance
// of App. H, then the backtrack from (K, M) and the mapping of App. A.2.
//
// Work decomposition:
//   * Staging: every thread loads one token (draft or target) -- id, byte offsets,
//     bytes -- validates it and packs it into a fixed-width LDS slot.
//   * Draft rows are processed in strips of 64 with lane r of wave 0 owning row
//     i = i0 + r.  Wave 0 sweeps the strip's anti-diagonals: at step t lane r finishes
//     cell (i0 + r, jfirst + t - r).  C(i-1, j) arrives from lane r-1 through a DPP wave
//     shift (lane 0 takes the previous strip's last row from LDS through the shift's
//     fill operand), C(i-1, j-1) is the value received one step earlier and C(i, j-1)
//     is the lane's own previous value.  The step is branch-free.
//   * Token distances: for bands up to the planned width (512 cells per row when LDS
//     allows) the distances of a strip are evaluated cell-parallel into an LDS byte
//     matrix laid out by sweep step (one dword per lane holds four consecutive steps),
//     double-buffered: while wave 0 sweeps strip s, waves 1-15 fill the buffer of strip
//     s + 1.  The sweep runs four steps per dword with the next dword and lane 0's next
//     four row-above values prefetched.  Wider bands: wave 0 evaluates each distance in
//     place during the sweep.
//   * Token distance: the bit-parallel edit-distance recurrence (Myers 1999, in
//     Hyyro's 2001 global-distance form) with the longer token as the pattern (one
//     bit per byte, at most 64) and the shorter one as the text; per-byte match masks
//     come from SWAR byte comparison of the packed pattern.
//   * Each cell's predecessor choice is a 2-bit code, 16 per dword, row-major inside
//     the band.  The current strip's codes live in LDS; finished strips are parked in
//     the caller's workspace and brought back strip by strip during the backtrack.
//   * Backtrack (wave 0), one row per step: inside row i the path runs left from its
//     entry column to the highest column whose move is not a left move (a find-last-set
//     over the 2-bit codes, 16 per dword), then enters row i-1.  The codes of every row
//     are first gathered into the freed cost buffers when they fit (else the strips are
//     fetched back one by one).  Path cells and map entries are then written by all
//     threads with binary searches over the rows' runs.
//
// LDS layout (bytes, each region 16-byte aligned):
//   tslot [max_m][TB] / tlen [max_m]   target token bytes and lengths
//   dslot [max_k][TB] / dlen [max_k]   draft token bytes and lengths
//   row0, row1 [max_m+8] int32         C of the row above the strip (double-buffered,
//                                      padded so four-step groups may read past M)
//   cost  2 x [groups][64] u32        token distances of a strip, [step/4][lane], double-buffered
//   scode [64][WPR] u32                direction codes of the current strip
//   path  [max_k+max_m] u32            backtracked cells (i << 16 | j), reverse order
//   sink  [64] u32                     target of the stores a lane does not need
// with WPR = ceil(min(max_m, 2 L + 1) / 16) for the largest band half-width L the
// bounds allow.
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
constexpr int kThreads = 1024;                   // wave 0 sweeps, the other waves precompute distances
constexpr int kPrecomp = 512;                    // widest band whose distances are precomputed per strip
constexpr int kRowPad = 8;                       // INF entries past column M in the row buffers
constexpr size_t kLdsLimit = 160 * 1024 - 1024;  // gfx950 LDS per workgroup, less static use

__host__ __device__ inline size_t align16(size_t v) { return (v + 15) & ~size_t(15); }

struct LdsPlan {
    size_t tslot, tlen, dslot, dlen, row0, row1, cost, cost_bytes, scode, path, sink, total;
    int wpr_max;
    int cost_w;  // widest band (cells per row) the two cost buffers hold
};

// Four-step groups of a 64-row strip sweep over a band of width w: the band's columns
// shift by up to one per row, so a strip spans up to w + 126 steps (+1 group for the
// prefetch).
__host__ __device__ inline int cost_groups(int w) { return (w + 2 * (kWave - 1) + 3) / 4 + 1; }

__host__ __device__ inline int band_half_width_bound(int32_t max_k, int32_t max_m, int32_t w) {
    int mx = max_k > max_m ? max_k : max_m;
    if (w < 0) return mx;
    int widen = mx - 1;  // largest possible |K - M|
    int L = w > widen ? w : widen;
    return L < mx ? L : mx;
}

__host__ __device__ inline int words_per_row_bound(int32_t max_k, int32_t max_m, int32_t w) {
    const long long L = band_half_width_bound(max_k, max_m, w);
    long long W = 2 * L + 1;
    if (W > max_m) W = max_m;
    return (int)((W + 15) / 16);
}

__host__ __device__ inline LdsPlan plan_lds_with(int32_t max_k, int32_t max_m, int32_t w, int tb, int cost_w) {
    LdsPlan p;
    p.wpr_max = words_per_row_bound(max_k, max_m, w);
    const size_t strip_rows = max_k < kWave ? (size_t)max_k : kWave;
    size_t off = 0;
    p.tslot = off;
    off = align16(off + (size_t)max_m * tb);
    p.tlen = off;
    off = align16(off + (size_t)max_m);
    p.dslot = off;
    off = align16(off + (size_t)max_k * tb);
    p.dlen = off;
    off = align16(off + (size_t)max_k);
    p.row0 = off;
    off = align16(off + 4 * ((size_t)max_m + 1 + kRowPad));
    p.row1 = off;
    off = align16(off + 4 * ((size_t)max_m + 1 + kRowPad));
    // distances of a strip, by sweep step, double-buffered (bands up to cost_w cells per row)
    p.cost_w = cost_w;
    p.cost_bytes = cost_w > 0 ? align16(4 * (size_t)kWave * cost_groups(cost_w)) : 0;
    p.cost = off;
    off = align16(off + 2 * p.cost_bytes);
    p.scode = off;
    off = align16(off + 4 * strip_rows * (size_t)p.wpr_max);
    p.path = off;  // per row: run (first column << 16 | entry column), then path offset
    off = align16(off + 8 * (size_t)max_k);
    p.sink = off;
    off = align16(off + 4 * kWave);
    p.total = off;
    return p;
}

// The plan with the widest precomputed band (at most kPrecomp cells per row) that fits in
// LDS; bands wider than the chosen width are swept with distances evaluated in place.
__host__ __device__ inline LdsPlan plan_lds(int32_t max_k, int32_t max_m, int32_t w, int tb) {
    const long long lb = band_half_width_bound(max_k, max_m, w);
    const long long wband = (2 * lb + 1) < max_m ? (2 * lb + 1) : max_m;  // cells per row, at most
    int cost_w = (int)(wband < kPrecomp ? wband : kPrecomp);
    LdsPlan p = plan_lds_with(max_k, max_m, w, tb, cost_w);
    while (p.total > kLdsLimit && cost_w > 0) {
        cost_w = cost_w > 32 ? cost_w / 2 : 0;
        p = plan_lds_with(max_k, max_m, w, tb, cost_w);
    }
    return p;
}

// C(i-1, .) from the lane below: DPP wave shift right by one lane; lane 0 gets `fill`.
__device__ __forceinline__ int from_lane_below(int v, int fill) {
    return __builtin_amdgcn_update_dpp(fill, v, 0x138 /* wave_shr:1 */, 0xF, 0xF, false);
}

__device__ __forceinline__ int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

struct Band {
    int K, M, L, W, WPR;
    __device__ __forceinline__ int jlo(int i) const { return (i - L) > 1 ? (i - L) : 1; }
    __device__ __forceinline__ int jhi(int i) const { return (i + L) < M ? (i + L) : M; }
};

// One sweep step for lane = row: combine the three predecessors of the cell, record the
// 2-bit choice and the cell value.  `rv` is lane 0's C(i0-1, j) (the fill of the shift).
struct SweepState {
    int cur, above_prev, lastc;
    uint32_t cw;
    int o;  // band offset of this lane's cell at the current step
};

__device__ __forceinline__ void sweep_step(SweepState &st, int d, int rv, int width, int j, int M, bool last_row,
                                           uint32_t *mycode, uint32_t *sink, int *rowOut) {
    const int lane = threadIdx.x;
    const bool inb = (unsigned)st.o < (unsigned)width;
    const int above = from_lane_below(st.cur, rv);  // C(i-1, j)
    const int diagv = st.above_prev;                // C(i-1, j-1)
    st.above_prev = above;
    const int left = st.cur;                        // C(i, j-1)
    // ties: diagonal, then (i-1, j), then (i, j-1)
    const int m1 = above < diagv ? above : diagv;
    const int c1 = above < diagv ? 1 : 0;
    const int best = left < m1 ? left : m1;
    const int code = left < m1 ? 2 : c1;
    const int nc = d + best;
    st.cur = inb ? nc : kInf;
    st.lastc = inb ? nc : st.lastc;
    const uint32_t keep = ((st.o & 15) == 0) ? 0u : st.cw;
    st.cw = inb ? (keep | ((uint32_t)code << (2 * (st.o & 15)))) : st.cw;
    uint32_t *cdst = inb ? (mycode + (st.o >> 4)) : (sink + lane);
    *cdst = st.cw;
    int *rdst = (last_row && j >= 0 && j <= M) ? (rowOut + j) : reinterpret_cast<int *>(sink + lane);
    *rdst = st.cur;
    ++st.o;
}

// Narrow strip: distances precomputed in `cost` as [step/4][lane] dwords.
__device__ __forceinline__ void sweep_strip_narrow(const Band &g, int i0, int rows, const int *rowIn, int *rowOut,
                                                   const uint32_t *cost, uint32_t *scode, uint32_t *sink,
                                                   int &cost_km) {
    const int lane = threadIdx.x;
    const int i = i0 + lane;
    const bool act = lane < rows;
    const int myjlo = g.jlo(i);
    const int width = act ? g.jhi(i) - myjlo + 1 : 0;
    const int jfirst = g.jlo(i0);
    const int jlast = g.jhi(i0 + rows - 1);
    const int steps = (jlast - jfirst + 1) + rows - 1;
    const int groups = (steps + 3) >> 2;
    uint32_t *mycode = scode + lane * g.WPR;
    const bool last_row = act && lane == rows - 1;

    SweepState st;
    st.cur = kInf;
    st.lastc = kInf;
    st.above_prev = (lane == 0) ? rowIn[jfirst - 1] : kInf;  // only lane 0 sees a finite C(i-1, j-1)
    st.cw = 0;
    st.o = jfirst - lane - myjlo;
    uint32_t dw = cost[lane];
    // lane 0 runs past column M at the end of the strip: those reads hit the INF pad at M+1
    const int jcap = g.M + 1;
    int r0 = rowIn[min(jfirst, jcap)], r1 = rowIn[min(jfirst + 1, jcap)];
    int r2 = rowIn[min(jfirst + 2, jcap)], r3 = rowIn[min(jfirst + 3, jcap)];
    for (int q = 0; q < groups; ++q) {
        // prefetch the next group (the buffers are padded for the read past the end)
        const uint32_t dwn = cost[(q + 1) * kWave + lane];
        const int jn = jfirst + 4 * (q + 1);
        const int n0 = rowIn[min(jn, jcap)], n1 = rowIn[min(jn + 1, jcap)];
        const int n2 = rowIn[min(jn + 2, jcap)], n3 = rowIn[min(jn + 3, jcap)];
        const int jb = jfirst + 4 * q - lane;
        sweep_step(st, (int)(dw & 0xFFu), r0, width, jb, g.M, last_row, mycode, sink, rowOut);
        sweep_step(st, (int)((dw >> 8) & 0xFFu), r1, width, jb + 1, g.M, last_row, mycode, sink, rowOut);
        sweep_step(st, (int)((dw >> 16) & 0xFFu), r2, width, jb + 2, g.M, last_row, mycode, sink, rowOut);
        sweep_step(st, (int)(dw >> 24), r3, width, jb + 3, g.M, last_row, mycode, sink, rowOut);
        dw = dwn;
        r0 = n0;
        r1 = n1;
        r2 = n2;
        r3 = n3;
    }
    if (act && i == g.K) cost_km = st.lastc;
}

// Wide strip: each step evaluates the token distance of the lane's cell in place.
template <int TB>
__device__ __forceinline__ void sweep_strip_wide(const Band &g, int i0, int rows, const int *rowIn, int *rowOut,
                                                 const uint32_t *tslot, const uint8_t *tlen, const uint32_t *dslot,
                                                 const uint8_t *dlen, uint32_t *scode, uint32_t *sink, int &cost_km) {
    const int lane = threadIdx.x;
    const int i = i0 + lane;
    const bool act = lane < rows;
    const int myjlo = g.jlo(i);
    const int width = act ? g.jhi(i) - myjlo + 1 : 0;
    const int jfirst = g.jlo(i0);
    const int jlast = g.jhi(i0 + rows - 1);
    const int steps = (jlast - jfirst + 1) + rows - 1;
    uint32_t *mycode = scode + lane * g.WPR;
    const bool last_row = act && lane == rows - 1;

    uint32_t xw[TB / 4];
    read_slot<TB>(dslot + (act ? i - 1 : 0) * (TB / 4), xw);
    const int xm = act ? dlen[i - 1] : 0;

    SweepState st;
    st.cur = kInf;
    st.lastc = kInf;
    st.above_prev = (lane == 0) ? rowIn[jfirst - 1] : kInf;
    st.cw = 0;
    st.o = jfirst - lane - myjlo;
    uint32_t yw[TB / 4];
    int jc = clampi(jfirst - lane, 1, g.M);
    read_slot<TB>(tslot + (jc - 1) * (TB / 4), yw);
    int yn = tlen[jc - 1];
    const int jcap = g.M + 1;  // lane 0 runs past column M at the end: the INF pad
    int rv = rowIn[min(jfirst, jcap)];
    for (int t = 0; t < steps; ++t) {
        const int j = jfirst + t - lane;
        const int d = token_distance<TB>(xw, xm, yw, yn);
        const int rvn = rowIn[min(jfirst + t + 1, jcap)];
        jc = clampi(j + 1, 1, g.M);
        uint32_t ywn[TB / 4];
        read_slot<TB>(tslot + (jc - 1) * (TB / 4), ywn);
        const int ynn = tlen[jc - 1];
        sweep_step(st, d, rv, width, j, g.M, last_row, mycode, sink, rowOut);
        rv = rvn;
#pragma unroll
        for (int q = 0; q < TB / 4; ++q) yw[q] = ywn[q];
        yn = ynn;
    }
    if (act && i == g.K) cost_km = st.lastc;
}

// Token distances of the band cells of the strip starting at row i0 into `cost`, laid out by
// sweep step (cell (i0 + r, j) at step t = j - jlo(i0) + r, byte t & 3 of dword
// [t / 4][r]); threads tid, tid + nthr, ... each take one cell.
template <int TB>
__device__ __forceinline__ void strip_costs(const Band &g, int i0, int rows, uint8_t *cost, const uint32_t *tslot,
                                            const uint8_t *tlen, const uint32_t *dslot, const uint8_t *dlen, int tid,
                                            int nthr) {
    const int ncell = rows * g.W;
    const float invW = 1.0f / (float)g.W;
    const int jfirst = g.jlo(i0);
    for (int idx = tid; idx < ncell; idx += nthr) {
        int r = (int)((float)idx * invW);
        int c = idx - r * g.W;
        if (c < 0) {
            --r;
            c += g.W;
        } else if (c >= g.W) {
            ++r;
            c -= g.W;
        }
        const int i = i0 + r;
        const int j = g.jlo(i) + c;
        if (j <= g.jhi(i)) {
            uint32_t xw[TB / 4], yw[TB / 4];
            read_slot<TB>(dslot + (i - 1) * (TB / 4), xw);
            read_slot<TB>(tslot + (j - 1) * (TB / 4), yw);
            const int t = j - jfirst + r;
            cost[((t >> 2) * kWave + r) * 4 + (t & 3)] = (uint8_t)token_distance<TB>(xw, dlen[i - 1], yw, tlen[j - 1]);
        }
    }
}

template <int TB>
__global__ void __launch_bounds__(kThreads) dtw_band(AlignArgs a, LdsPlan lp, uint32_t *gcodes, size_t gcode_stride) {
    extern __shared__ __align__(16) uint8_t lds[];
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const int d0 = a.draft_off[b], K = a.draft_off[b + 1] - d0;
    const int t0 = a.target_off[b], M = a.target_off[b + 1] - t0;

    uint32_t *tslot = reinterpret_cast<uint32_t *>(lds + lp.tslot);
    uint8_t *tlen = lds + lp.tlen;
    uint32_t *dslot = reinterpret_cast<uint32_t *>(lds + lp.dslot);
    uint8_t *dlen = lds + lp.dlen;
    int *rowIn = reinterpret_cast<int *>(lds + lp.row0);
    int *rowOut = reinterpret_cast<int *>(lds + lp.row1);
    uint8_t *costbuf[2] = {lds + lp.cost, lds + lp.cost + lp.cost_bytes};
    uint32_t *scode = reinterpret_cast<uint32_t *>(lds + lp.scode);
    uint32_t *pathbuf = reinterpret_cast<uint32_t *>(lds + lp.path);
    uint32_t *sink = reinterpret_cast<uint32_t *>(lds + lp.sink);
    __shared__ int s_cost;
    __shared__ int votes[kThreads / kWave];

    // ---- staging + validation: one token (draft or target) per thread
    const bool shape_ok = K >= 1 && K <= a.max_k && M >= 1 && M <= a.max_m;
    int bad = shape_ok ? 0 : 1;
    if (shape_ok) {
        for (int e = tid; e < K + M; e += kThreads) {
            const bool ok = e < K ? stage_token<TB>(a.vd, a.draft_ids[d0 + e], dslot + e * (TB / 4), dlen + e)
                                  : stage_token<TB>(a.vt, a.target_ids[t0 + e - K], tslot + (e - K) * (TB / 4),
                                                    tlen + (e - K));
            bad |= ok ? 0 : 1;
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
    g.WPR = (g.W + 15) >> 4;
    const bool pre = g.W <= lp.cost_w;  // distances precomputed strip by strip
    const int nstrips = (K + kWave - 1) / kWave;
    uint32_t *parked = gcodes + (size_t)b * gcode_stride;  // codes of finished strips (K > 64 only)

    // ---- strips of 64 rows: wave 0 sweeps strip s while the other waves compute the
    // distances of strip s + 1 into the other buffer
    if (pre) strip_costs<TB>(g, 1, K < kWave ? K : kWave, costbuf[0], tslot, tlen, dslot, dlen, tid, kThreads);
    // the sweep is the critical path: its wave wins issue arbitration on its SIMD
    if (wave == 0) __builtin_amdgcn_s_setprio(3);
    for (int j = tid; j <= M + kRowPad; j += kThreads) rowIn[j] = (j == 0) ? 0 : kInf;  // C(0, j)
    __syncthreads();
    int cost_km = kInf;
    for (int s = 0; s < nstrips; ++s) {
        const int i0 = 1 + s * kWave;
        const int rows = (K - i0 + 1) < kWave ? (K - i0 + 1) : kWave;
        if (wave == 0) {
            for (int j = lane; j <= M + kRowPad; j += kWave) rowOut[j] = kInf;
            if (pre)
                sweep_strip_narrow(g, i0, rows, rowIn, rowOut, reinterpret_cast<const uint32_t *>(costbuf[s & 1]),
                                   scode, sink, cost_km);
            else
                sweep_strip_wide<TB>(g, i0, rows, rowIn, rowOut, tslot, tlen, dslot, dlen, scode, sink, cost_km);
            if (s + 1 < nstrips) {  // park this strip's codes; the last strip stays in LDS
                for (int e = lane; e < rows * g.WPR; e += kWave) parked[(size_t)(i0 - 1) * g.WPR + e] = scode[e];
            }
        } else if (pre && s + 1 < nstrips) {
            const int i1 = i0 + kWave;
            const int rows1 = (K - i1 + 1) < kWave ? (K - i1 + 1) : kWave;
            strip_costs<TB>(g, i1, rows1, costbuf[(s + 1) & 1], tslot, tlen, dslot, dlen, tid - kWave,
                            kThreads - kWave);
        }
        __syncthreads();
        int *tmp = rowIn;
        rowIn = rowOut;
        rowOut = tmp;
    }
    if (wave == 0 && lane == (K - 1) % kWave) s_cost = cost_km;
    // every row's codes in one LDS matrix when they fit in the (now free) cost buffers:
    // the parked strips come back in parallel, the last strip is still in scode
    const size_t code_words = (size_t)K * g.WPR;
    uint32_t *codes = reinterpret_cast<uint32_t *>(lds + lp.cost);
    const bool all_codes = 4 * code_words <= 2 * lp.cost_bytes;
    if (all_codes) {
        const size_t last0 = (size_t)(nstrips - 1) * kWave * g.WPR;  // first word of the last strip
        for (size_t e = tid; e < code_words; e += kThreads)
            codes[e] = e < last0 ? parked[e] : scode[e - last0];
    }
    __syncthreads();
    uint32_t *seg = pathbuf;              // [K]: first column << 16 | entry column (0: not on the path)
    uint32_t *poff = pathbuf + a.max_k;   // [K]: index of the row's first path cell
    __shared__ int s_imin, s_n;

    // ---- backtrack (wave 0): inside row i the path runs left from its entry column e to
    // the highest column x <= e whose move is not (i, j-1); it enters row i-1 at x - 1
    // after a diagonal move and at x after an (i-1, j) move
    if (wave == 0) {
        if (lane == 0) a.cost[b] = s_cost;
        int e = M, i = K;
        if (all_codes && g.WPR <= kWave) {
            // lane l holds code word l of a row; two rows are searched per iteration while
            // the next two are read, and the runs are buffered one per lane (row i in lane
            // (i - 1) % 64) and flushed to LDS every 64 rows, so the walk is branch-free
            auto row_words = [&](int r) {  // code word `lane` of row r (0 past the band or row 0)
                return (r >= 1 && lane < g.WPR) ? codes[(size_t)(r - 1) * g.WPR + lane] : 0u;
            };
            uint32_t segbuf = 0;
            bool live = true;
            auto walk_row = [&](int r, uint32_t cur) {
                const int jl = g.jlo(r);
                const int c = e - jl;  // band offset of the entry column
                const int we = c >> 4, p15 = c & 15;
                const uint32_t nl = 0x55555555u & ~((cur >> 1) & ~cur);  // low bit of codes other than 2
                const uint32_t pm = p15 == 15 ? 0xFFFFFFFFu : ((1u << (2 * p15 + 2)) - 1u);
                const uint32_t m = nl & (lane < we ? 0xFFFFFFFFu : (lane == we ? pm : 0u));
                const unsigned long long has = __ballot(m != 0u);
                const int lw = has ? 63 - __clzll(has) : 0;
                const uint32_t mw = __builtin_amdgcn_readlane(m, lw);
                const uint32_t ww = __builtin_amdgcn_readlane(cur, lw);
                const int hb = 31 - __clz(mw | 1u);
                const int x = jl + lw * 16 + (hb >> 1);
                segbuf = (lane == ((r - 1) & (kWave - 1))) ? (((uint32_t)x << 16) | (uint32_t)e) : segbuf;
                if (((r - 1) & (kWave - 1)) == 0 && r - 1 + lane < K) seg[r - 1 + lane] = segbuf;
                // has == 0 never happens: a run of (i, j-1) moves ends inside the band
                live = has != 0ull;
                e = ((ww >> hb) & 3u) == 0u ? x - 1 : x;
            };
            uint32_t c0 = row_words(K), c1 = row_words(K - 1);
            for (; i >= 1; i -= 2) {
                const uint32_t n0 = row_words(i - 2), n1 = row_words(i - 3);
                walk_row(i, c0);
                if (!live) break;  // row i is not on the path
                if (e < 1 || i == 1) {
                    --i;
                    break;
                }
                walk_row(i - 1, c1);
                if (!live) {
                    --i;
                    break;
                }
                if (e < 1) {
                    i -= 2;
                    break;
                }
                c0 = n0;
                c1 = n1;
            }
            // the partial block of rows the walk ended in
            const int rl = i + 1;  // last row written: rows rl.. are in seg or segbuf
            const int blk = (rl - 1) & ~(kWave - 1);
            if (rl >= 1 && ((rl - 1) & (kWave - 1)) != 0) {
                const int r = blk + lane;
                if (r >= rl - 1 && r < K && r < blk + kWave) seg[r] = segbuf;
            }
            if (i < 0) i = 0;
        } else {
            int strip = nstrips - 1;  // strip held in scode when the codes are not all in LDS
            for (; i >= 1; --i) {
                const uint32_t *rc;
                if (all_codes) {
                    rc = codes + (size_t)(i - 1) * g.WPR;
                } else {
                    if (i < 1 + strip * kWave) {  // fetch the strip above from the workspace
                        --strip;
                        for (int e2 = lane; e2 < kWave * g.WPR; e2 += kWave)
                            scode[e2] = parked[(size_t)strip * kWave * g.WPR + e2];
                    }
                    rc = scode + (size_t)(i - 1 - strip * kWave) * g.WPR;
                }
                const int jl = g.jlo(i);
                const int c = e - jl;
                int w = c >> 4;
                const int p15 = c & 15;
                uint32_t word = rc[w];
                uint32_t m = 0x55555555u & ~((word >> 1) & ~word) &
                             (p15 == 15 ? 0xFFFFFFFFu : ((1u << (2 * p15 + 2)) - 1u));
                while (m == 0 && w > 0) {
                    --w;
                    word = rc[w];
                    m = 0x55555555u & ~((word >> 1) & ~word);
                }
                if (m == 0) break;  // never taken
                const int hb = 31 - __clz(m);
                const int x = jl + w * 16 + (hb >> 1);
                if (lane == 0) seg[i - 1] = ((uint32_t)x << 16) | (uint32_t)e;
                e = ((word >> hb) & 3u) == 0u ? x - 1 : x;
                if (e < 1) {
                    --i;
                    break;
                }
            }
        }
        // rows 1..i are not on the path (only if the walk broke off); path offsets for the rest
        const int imin = i + 1;
        int carry = 0;
        for (int r0 = imin - 1; r0 < K; r0 += kWave) {
            const int r = r0 + lane;
            const uint32_t sv = r < K ? seg[r] : 0u;
            const int len = r < K ? (int)(sv & 0xFFFFu) - (int)(sv >> 16) + 1 : 0;
            const int incl = dtw::wave_prefix_sum(len) + carry;
            if (r < K) poff[r] = (uint32_t)(incl - len);
            carry = __builtin_amdgcn_readlane(incl, kWave - 1);
        }
        if (lane == 0) {
            s_imin = imin;
            s_n = carry;
            a.path_len[b] = carry;
        }
    }
    __syncthreads();
    const int imin = s_imin, n = s_n;
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

template <int TB>
int launch_tb(const AlignArgs &a, void *workspace, size_t workspace_bytes, hipStream_t stream) {
    const LdsPlan lp = plan_lds(a.max_k, a.max_m, a.w, TB);
    if (lp.total > kLdsLimit) return TT_EUNSUPPORTED;
    const size_t stride = (size_t)a.max_k * (size_t)lp.wpr_max;  // parked code words per pair
    uint32_t *gcodes = nullptr;
    if (a.max_k > kWave) {
        if (workspace == nullptr || workspace_bytes < 4 * stride * (size_t)a.n_pairs) return TT_EWORKSPACE;
        gcodes = static_cast<uint32_t *>(workspace);
    }
    if (lp.total > 64 * 1024) {
        if (hipFuncSetAttribute(reinterpret_cast<const void *>(&dtw_band<TB>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lp.total) != hipSuccess)
            return TT_ELAUNCH;
    }
    hipLaunchKernelGGL(dtw_band<TB>, dim3(a.n_pairs), dim3(kThreads), lp.total, stream, a, lp, gcodes, stride);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
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
    if (max_k <= kWave) return 0;
    return 4 * (size_t)n_pairs * (size_t)max_k * (size_t)words_per_row_bound(max_k, max_m, w);
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
