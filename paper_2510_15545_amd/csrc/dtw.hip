// Dynamic Token Warping on gfx950: one wave64 per (draft, proxy-target) pair.
//
// Computes Alg. 1 of the paper (cumulative cost C over draft x target tokens with
// the Sakoe-Chiba band, Sec. 4.1) using the byte-level Levenshtein token distance
// of App. H, then the backtrack from (K, M) and the mapping of App. A.2.
//
// Work decomposition (per workgroup = one wave = one pair):
//   * Staging: every lane loads one token (draft or target) -- id, byte offsets,
//     bytes -- validates it and packs it into a fixed-width LDS slot.
//   * Draft rows are processed in strips of 64 with lane r owning row i = i0 + r.
//     The wave sweeps the strip's anti-diagonals: at step t lane r finishes cell
//     (i0 + r, jfirst + t - r).  C(i-1, j) arrives from lane r-1 through a DPP wave
//     shift (lane 0 takes the previous strip's last row from LDS through the shift's
//     fill operand), C(i-1, j-1) is the value received one step earlier and C(i, j-1)
//     is the lane's own previous value.  The step is branch-free.
//   * Narrow bands (at most 128 cells per row): all 64 lanes first evaluate every
//     band cell's token distance into an LDS byte matrix laid out by sweep step (one
//     dword per lane holds four consecutive steps), then the sweep runs four steps per
//     dword with the next dword and lane 0's next four row-above values prefetched.
//     Wide bands: the sweep evaluates the distance in place (most lanes are in band).
//   * Token distance: the bit-parallel edit-distance recurrence (Myers 1999, in
//     Hyyro's 2001 global-distance form) with the longer token as the pattern (one
//     bit per byte, at most 64) and the shorter one as the text; per-byte match masks
//     come from SWAR byte comparison of the packed pattern.
//   * Each cell's predecessor choice is a 2-bit code, 16 per dword, row-major inside
//     the band.  The current strip's codes live in LDS; finished strips are parked in
//     the caller's workspace and brought back strip by strip during the backtrack.
//   * Backtrack: the wave loads an 8 x 8 window of codes ending at the current cell
//     (one code per lane) and walks it with scalar readlane steps, reloading when the
//     walk leaves the window; visited cells are buffered one per lane and flushed to
//     LDS every 64 steps.
//
// LDS layout (bytes, each region 16-byte aligned):
//   tslot [max_m][TB] / tlen [max_m]   target token bytes and lengths
//   dslot [max_k][TB] / dlen [max_k]   draft token bytes and lengths
//   row0, row1 [max_m+8] int32         C of the row above the strip (double-buffered,
//                                      padded so four-step groups may read past M)
//   cost  [49][64] u32                 token distances of a narrow strip, [step/4][lane]
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
constexpr int kNarrow = 128;                     // widest band precomputed into the cost matrix
constexpr int kCostGroups = (kNarrow + kWave - 1 + 3) / 4 + 1;  // four-step groups of a narrow strip, +1 prefetch
constexpr int kRowPad = 8;                       // INF entries past column M in the row buffers
constexpr size_t kLdsLimit = 160 * 1024 - 1024;  // gfx950 LDS per workgroup, less static use

__host__ __device__ inline size_t align16(size_t v) { return (v + 15) & ~size_t(15); }

struct LdsPlan {
    size_t tslot, tlen, dslot, dlen, row0, row1, cost, scode, path, sink, total;
    int wpr_max;
};

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

__host__ __device__ inline LdsPlan plan_lds(int32_t max_k, int32_t max_m, int32_t w, int tb) {
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
    p.cost = off;
    off = align16(off + 4 * (size_t)kWave * kCostGroups);
    p.scode = off;
    off = align16(off + 4 * strip_rows * (size_t)p.wpr_max);
    p.path = off;
    off = align16(off + 4 * ((size_t)max_k + (size_t)max_m));
    p.sink = off;
    off = align16(off + 4 * kWave);
    p.total = off;
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

template <int TB>
__global__ void __launch_bounds__(kWave) dtw_band_wave(AlignArgs a, LdsPlan lp, uint32_t *gcodes,
                                                       size_t gcode_stride) {
    extern __shared__ __align__(16) uint8_t lds[];
    const int b = blockIdx.x;
    const int lane = threadIdx.x;
    const int d0 = a.draft_off[b], K = a.draft_off[b + 1] - d0;
    const int t0 = a.target_off[b], M = a.target_off[b + 1] - t0;

    uint32_t *tslot = reinterpret_cast<uint32_t *>(lds + lp.tslot);
    uint8_t *tlen = lds + lp.tlen;
    uint32_t *dslot = reinterpret_cast<uint32_t *>(lds + lp.dslot);
    uint8_t *dlen = lds + lp.dlen;
    int *rowIn = reinterpret_cast<int *>(lds + lp.row0);
    int *rowOut = reinterpret_cast<int *>(lds + lp.row1);
    uint8_t *cost = lds + lp.cost;
    uint32_t *scode = reinterpret_cast<uint32_t *>(lds + lp.scode);
    uint32_t *pathbuf = reinterpret_cast<uint32_t *>(lds + lp.path);
    uint32_t *sink = reinterpret_cast<uint32_t *>(lds + lp.sink);
    __shared__ int s_cost;

    // ---- staging + validation: one token (draft or target) per lane
    bool ok = K >= 1 && K <= a.max_k && M >= 1 && M <= a.max_m;
    if (ok) {
        bool bad = false;
        for (int e = lane; e < K + M; e += kWave) {
            if (e < K)
                bad |= !stage_token<TB>(a.vd, a.draft_ids[d0 + e], dslot + e * (TB / 4), dlen + e);
            else
                bad |= !stage_token<TB>(a.vt, a.target_ids[t0 + e - K], tslot + (e - K) * (TB / 4),
                                        tlen + (e - K));
        }
        ok = !__any(bad);
    }
    if (!ok) {
        if (lane == 0) {
            a.cost[b] = -1;
            a.path_len[b] = 0;
        }
        for (int j = lane; j < M; j += kWave) a.map[t0 + j] = -1;
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
    const bool narrow = g.W <= kNarrow;
    const int nstrips = (K + kWave - 1) / kWave;
    uint32_t *parked = gcodes + (size_t)b * gcode_stride;  // codes of finished strips (K > 64 only)

    for (int j = lane; j <= M + kRowPad; j += kWave) rowIn[j] = (j == 0) ? 0 : kInf;  // C(0, j)
    __syncthreads();

    int cost_km = kInf;
    for (int s = 0; s < nstrips; ++s) {
        const int i0 = 1 + s * kWave;
        const int rows = (K - i0 + 1) < kWave ? (K - i0 + 1) : kWave;
        if (narrow) {
            // token distances of every band cell of the strip, cell-parallel
            const int ncell = rows * g.W;
            const float invW = 1.0f / (float)g.W;
            for (int idx = lane; idx < ncell; idx += kWave) {
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
                    const int t = j - g.jlo(i0) + r;  // sweep step at which lane r reaches (i, j)
                    cost[((t >> 2) * kWave + r) * 4 + (t & 3)] =
                        (uint8_t)token_distance<TB>(xw, dlen[i - 1], yw, tlen[j - 1]);
                }
            }
        }
        for (int j = lane; j <= M + kRowPad; j += kWave) rowOut[j] = kInf;
        __syncthreads();
        if (narrow)
            sweep_strip_narrow(g, i0, rows, rowIn, rowOut, reinterpret_cast<const uint32_t *>(cost), scode, sink,
                               cost_km);
        else
            sweep_strip_wide<TB>(g, i0, rows, rowIn, rowOut, tslot, tlen, dslot, dlen, scode, sink, cost_km);
        __syncthreads();
        if (s + 1 < nstrips) {  // park this strip's codes; the last strip stays in LDS
            for (int e = lane; e < rows * g.WPR; e += kWave) parked[(size_t)(i0 - 1) * g.WPR + e] = scode[e];
        }
        int *tmp = rowIn;
        rowIn = rowOut;
        rowOut = tmp;
    }
    if (lane == (K - 1) % kWave) s_cost = cost_km;
    __syncthreads();
    if (lane == 0) a.cost[b] = s_cost;

    // ---- backtrack from (K, M): walk 8 x 8 windows of codes held one per lane
    int ii = K, jj = M, n = 0;
    int strip = nstrips - 1;  // strip whose codes are in LDS
    int dr = 8, dc = 8;       // offset of (ii, jj) from the window's last cell; 8 forces a load
    int wcode = 3;
    uint32_t pbuf = 0;        // visited cells, cell n held by lane n % 64
    const int cap = K + M;
    while (ii >= 1 && jj >= 1 && n < cap) {
        if (ii < 1 + strip * kWave) {  // the walk left the strip held in LDS: fetch the one above
            --strip;
            const int i0 = 1 + strip * kWave;
            __threadfence_block();
            for (int e = lane; e < kWave * g.WPR; e += kWave) scode[e] = parked[(size_t)(i0 - 1) * g.WPR + e];
            __syncthreads();
            dr = 8;
        }
        if ((dr | dc) > 7) {
            const int ci = ii - (lane >> 3), cj = jj - (lane & 7);
            const int s0 = 1 + strip * kWave;
            const int c = cj - g.jlo(ci);
            const bool valid = ci >= s0 && cj >= 1 && c >= 0 && cj <= g.jhi(ci);
            const uint32_t word = scode[valid ? (ci - s0) * g.WPR + (c >> 4) : 0];
            wcode = valid ? (int)((word >> (2 * (c & 15))) & 3u) : 3;
            dr = 0;
            dc = 0;
        }
        const int code = __builtin_amdgcn_readlane(wcode, dr * 8 + dc);
        if (code == 3) break;  // never taken: every path cell lies inside the band
        pbuf = (lane == (n & (kWave - 1))) ? (((uint32_t)ii << 16) | (uint32_t)jj) : pbuf;
        ++n;
        if ((n & (kWave - 1)) == 0) pathbuf[n - kWave + lane] = pbuf;
        const int di = code != 2 ? 1 : 0, dj = code != 1 ? 1 : 0;
        ii -= di;
        jj -= dj;
        dr += di;
        dc += dj;
    }
    if (lane < (n & (kWave - 1))) pathbuf[(n & ~(kWave - 1)) + lane] = pbuf;
    if (lane == 0) a.path_len[b] = n;
    __syncthreads();
    int32_t *pp = a.path + 2 * ((size_t)d0 + (size_t)t0);
    for (int q = lane; q < n; q += kWave) {
        const uint32_t cell = pathbuf[n - 1 - q];
        const int ci = (int)(cell >> 16), cj = (int)(cell & 0xFFFFu);
        pp[2 * q] = ci - 1;
        pp[2 * q + 1] = cj - 1;
        const bool last_in_col = (q == n - 1) || ((int)(pathbuf[n - 2 - q] & 0xFFFFu) != cj);
        if (last_in_col) a.map[t0 + cj - 1] = ci - 1;
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
        if (hipFuncSetAttribute(reinterpret_cast<const void *>(&dtw_band_wave<TB>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lp.total) != hipSuccess)
            return TT_ELAUNCH;
    }
    hipLaunchKernelGGL(dtw_band_wave<TB>, dim3(a.n_pairs), dim3(kWave), lp.total, stream, a, lp, gcodes, stride);
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
