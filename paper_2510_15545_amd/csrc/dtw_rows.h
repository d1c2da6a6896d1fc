// Row-scan Dynamic Token Warping for short pairs (K <= 64 draft tokens, M <= 64 target
// tokens), as device functions shared by the alignment kernel and the fused step kernel.
//
// Same results as the strip kernel (Alg. 1 with the Sakoe-Chiba band of Sec. 4.1, the
// byte Levenshtein distance of App. H, backtrack from (K, M) with ties to the diagonal,
// then (i-1, j), then (i, j-1), and the mapping of App. A.2), computed row by row with
// lane = column instead of along anti-diagonals:
//
//   * Staging and token distances use every thread of the workgroup: each band cell's
//     distance is one thread's work, written to an LDS byte matrix [i][j].
//   * Row i of the cumulative cost follows from row i-1 with two wave scans.  With
//     U(j) = d(i, j) + min(C(i-1, j-1), C(i-1, j)) and S(j) the prefix sum of d(i, .)
//     over the band,  C(i, j) = S(j) + min over k <= j of (U(k) - S(k)): the left moves
//     inside a row are a (min, +) prefix scan.  Out-of-band cells are infinite.
//   * A cell's predecessor is (i, j-1) iff C(i, j-1) < min(C(i-1, j-1), C(i-1, j)), else
//     the diagonal iff C(i-1, j-1) <= C(i-1, j), else (i-1, j).  One wave runs the row
//     recurrence and leaves C in LDS.
//   * Inside row i the optimal path runs left from its entry column e to the highest
//     column x <= e whose move is not a left move, then enters row i-1 at x - 1
//     (diagonal) or x.  Every wave tabulates, for its rows and every possible e, that
//     x and the next entry column (two ballots per row give the move masks); the
//     backtrack is then one LDS lookup per row.
//   * Row i covers columns [x_i, e_i], x_i non-decreasing in i.  Path cell q lies in the
//     last row whose run starts at or before q, and column j maps to the last row whose
//     run starts at or before j (a column shared by two rows through an (i-1, j) move
//     belongs to the higher one: the map holds the largest draft index).  Both are
//     prefix maxima over LDS arrays filled with atomic max, written lane-parallel.
#pragma once

#include <climits>

#include "dtw_common.h"

namespace tt {
namespace rows {

using dtw::kInf;
using dtw::kWave;

constexpr int kMaxSide = 64;  // bound on K and M

constexpr int kCmLd = kMaxSide + 1;  // row stride of the cumulative cost matrix

template <int TB>
struct Lds {
    uint32_t tslot[kMaxSide * (TB / 4)];
    uint32_t dslot[kMaxSide * (TB / 4)];
    int cm[(kMaxSide + 1) * kCmLd];     // C(i, j) at [i * 65 + j], i, j = 0..64
    int rowmax[2 * kMaxSide];           // path index -> row starting there (scratch)
    int colmax[kMaxSide + 1];           // column -> last row whose segment starts there (scratch)
    uint8_t ftab[kMaxSide * kCmLd];     // row i, entry column e: entry column of row i - 1
    uint8_t xtab[kMaxSide * kCmLd];     // row i, entry column e: first column of row i's run
    uint8_t tlen[kMaxSide];
    uint8_t dlen[kMaxSide];
    uint8_t cost[kMaxSide * kMaxSide];  // d(i, j) at [(i-1) * 64 + j - 1]
};

template <unsigned CTRL, unsigned ROW_MASK>
__device__ __forceinline__ int dpp_from(int v, int identity) {
    return __builtin_amdgcn_update_dpp(identity, v, CTRL, ROW_MASK, 0xF, false);
}

// Inclusive scans over the 64 lanes: Hillis-Steele inside rows of 16 lanes, then the
// row broadcasts of lane 15 and lane 31.
__device__ __forceinline__ int scan_add(int v) {
    v += dpp_from<0x111, 0xF>(v, 0);
    v += dpp_from<0x112, 0xF>(v, 0);
    v += dpp_from<0x114, 0xF>(v, 0);
    v += dpp_from<0x118, 0xF>(v, 0);
    v += dpp_from<0x142, 0xA>(v, 0);
    v += dpp_from<0x143, 0xC>(v, 0);
    return v;
}

// (INT_MAX, the identity of v_min_i32, lets each step fuse into one DPP min.)
__device__ __forceinline__ int scan_min(int v) {
    v = min(v, dpp_from<0x111, 0xF>(v, INT_MAX));
    v = min(v, dpp_from<0x112, 0xF>(v, INT_MAX));
    v = min(v, dpp_from<0x114, 0xF>(v, INT_MAX));
    v = min(v, dpp_from<0x118, 0xF>(v, INT_MAX));
    v = min(v, dpp_from<0x142, 0xA>(v, INT_MAX));
    v = min(v, dpp_from<0x143, 0xC>(v, INT_MAX));
    return v;
}

// Value of the lane below (wave shift right by one); lane 0 gets `fill`.
__device__ __forceinline__ int from_lane_below(int v, int fill) {
    return __builtin_amdgcn_update_dpp(fill, v, 0x138 /* wave_shr:1 */, 0xF, 0xF, false);
}

__device__ __forceinline__ uint64_t lane_u64(uint64_t v, int lane) {
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, lane);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}

// Band half-width: |i - j| <= L with L = max(w, |K - M|), capped at max(K, M) (w < 0: no band).
__device__ __forceinline__ int band_half_width(int K, int M, int w) {
    const int mx = K > M ? K : M;
    int L = (w < 0) ? mx : (w > abs(K - M) ? w : abs(K - M));
    return L > mx ? mx : L;
}

// Loads and validates the pair's K + M tokens into LDS, threads tid, tid + nthr, ...;
// returns nonzero if this thread saw an invalid token.  Caller guarantees K, M <= 64.
template <int TB>
__device__ __forceinline__ int stage(const AlignArgs &a, Lds<TB> &s, int d0, int K, int t0, int M, int tid,
                                     int nthr) {
    int bad = 0;
    for (int e = tid; e < K + M; e += nthr) {
        const bool ok = e < K ? dtw::stage_token<TB>(a.vd, a.draft_ids[d0 + e], s.dslot + e * (TB / 4), s.dlen + e)
                              : dtw::stage_token<TB>(a.vt, a.target_ids[t0 + e - K], s.tslot + (e - K) * (TB / 4),
                                                     s.tlen + (e - K));
        bad |= ok ? 0 : 1;
    }
    return bad;
}

// Token distance of every band cell, one cell per thread.
template <int TB>
__device__ __forceinline__ void costs(Lds<TB> &s, int K, int M, int L, int tid, int nthr) {
    const float invM = 1.0f / (float)M;
    for (int idx = tid; idx < K * M; idx += nthr) {
        int r = (int)((float)idx * invM);
        int c = idx - r * M;
        if (c < 0) {
            --r;
            c += M;
        } else if (c >= M) {
            ++r;
            c -= M;
        }
        const int i = r + 1, j = c + 1;
        if (j >= i - L && j <= i + L) {
            uint32_t xw[TB / 4], yw[TB / 4];
            dtw::read_slot<TB>(s.dslot + r * (TB / 4), xw);
            dtw::read_slot<TB>(s.tslot + c * (TB / 4), yw);
            s.cost[r * kMaxSide + c] = (uint8_t)dtw::token_distance<TB>(xw, s.dlen[r], yw, s.tlen[c]);
        }
    }
}

// Border of C: C(0, 0) = 0, C(0, j) = C(i, 0) = infinity.
template <int TB>
__device__ __forceinline__ void init_border(Lds<TB> &s, int tid, int nthr) {
    for (int e = tid; e < 2 * kCmLd; e += nthr) {
        if (e < kCmLd) s.cm[e] = e == 0 ? 0 : kInf;
        else s.cm[(e - kCmLd) * kCmLd] = (e == kCmLd) ? 0 : kInf;
    }
}

// One wave: rows 1..K of C (lane = column j - 1), stored to LDS; returns C(K, M).
template <int TB>
__device__ __forceinline__ int recurrence(Lds<TB> &s, int K, int M, int L) {
    const int lane = threadIdx.x % kWave;
    const int j = lane + 1;
    int cprev = kInf;  // C(i-1, j); row 0 is infinite except C(0, 0) = 0
    // row i's distances and their band prefix sum are formed one row ahead, so that their
    // scan can fill the wait states of the current row's (min, +) scan
    int d = s.cost[lane];
    bool inb = j <= M && j >= 1 - L && j <= 1 + L;
    int sd = scan_add(inb ? d : 0);
    for (int i = 1; i <= K; ++i) {
        const int inext = i < K ? i + 1 : i;
        const int dn = s.cost[(inext - 1) * kMaxSide + lane];
        const bool inbn = j <= M && j >= inext - L && j <= inext + L;
        const int diag = from_lane_below(cprev, i == 1 ? 0 : kInf);
        const int m = min(diag, cprev);
        const int p = scan_min(inb ? m + d - sd : kInf);
        const int sdn = scan_add(inbn ? dn : 0);
        const int c = inb ? min(sd + p, kInf) : kInf;
        s.cm[i * kCmLd + j] = c;
        cprev = c;
        d = dn;
        inb = inbn;
        sd = sdn;
    }
    return __builtin_amdgcn_readlane(cprev, M - 1);
}

// Every wave: for rows wave + 1, wave + 1 + nwaves, ... and every entry column e, the
// first column x of the row's run and the entry column of the row below, from C in LDS.
template <int TB>
__device__ __forceinline__ void moves(Lds<TB> &s, int K, int M, int L, int wave, int nwaves) {
    const int lane = threadIdx.x % kWave;
    const int j = lane + 1;  // also the entry column e tabulated by this lane
    for (int i = 1 + wave; i <= K; i += nwaves) {
        const bool inb = j <= M && j >= i - L && j <= i + L;
        const int diag = s.cm[(i - 1) * kCmLd + j - 1];
        const int up = s.cm[(i - 1) * kCmLd + j];
        const int left = s.cm[i * kCmLd + j - 1];
        const bool not_left = !(left < min(diag, up));
        const uint64_t nl = __ballot(inb && not_left);
        const uint64_t dg = __ballot(inb && not_left && diag <= up);
        const uint64_t cand = nl & (j >= 64 ? ~0ull : ((1ull << j) - 1));
        const int x = cand ? 64 - __clzll(cand) : 0;  // highest not-left column <= e
        const int f = x > 0 ? (((dg >> (x - 1)) & 1ull) ? x - 1 : x) : 0;
        s.xtab[(i - 1) * kCmLd + j] = (uint8_t)x;
        s.ftab[(i - 1) * kCmLd + j] = (uint8_t)f;
        if (lane == 0) {  // entry column 0: the walk has ended
            s.xtab[(i - 1) * kCmLd] = 0;
            s.ftab[(i - 1) * kCmLd] = 0;
        }
    }
}

__device__ __forceinline__ int scan_max(int v) {
    v = max(v, dpp_from<0x111, 0xF>(v, INT_MIN));
    v = max(v, dpp_from<0x112, 0xF>(v, INT_MIN));
    v = max(v, dpp_from<0x114, 0xF>(v, INT_MIN));
    v = max(v, dpp_from<0x118, 0xF>(v, INT_MIN));
    v = max(v, dpp_from<0x142, 0xA>(v, INT_MIN));
    v = max(v, dpp_from<0x143, 0xC>(v, INT_MIN));
    return v;
}

// One wave: backtrack from (K, M) through the tables, then cost, path_len, path and map of
// pair b.  Returns i*(j) (0-based) in lane j - 1 for j <= M, -1 in the other lanes.
template <int TB>
__device__ __forceinline__ int backtrack(const AlignArgs &a, Lds<TB> &s, int b, int d0, int K, int t0, int M,
                                         int total) {
    const int lane = threadIdx.x % kWave;
    // entry column of every row, walking down from (K, M); 0 once the walk has ended
    int e = M, ent = 0;
    for (int i = K; i >= 1; --i) {
        ent = (lane == i - 1) ? e : ent;
        e = s.ftab[(i - 1) * kCmLd + e];
    }
    // row lane + 1 covers columns [x, ent]
    const int x = (lane < K && ent > 0) ? s.xtab[lane * kCmLd + ent] : 0;
    const int len = x > 0 ? ent - x + 1 : 0;
    const int incl = scan_add(len);
    const int off = incl - len;
    const int n = __builtin_amdgcn_readlane(incl, kWave - 1);
    if (lane == 0) {
        a.cost[b] = total;
        a.path_len[b] = n;
    }
    s.rowmax[lane] = -1;
    s.rowmax[lane + kWave] = -1;
    s.colmax[lane] = -1;
    if (len > 0) {
        atomicMax(&s.rowmax[off], lane);
        atomicMax(&s.colmax[x - 1], lane);
    }
    // path cell q: the last row starting at or before q (two passes of 64 cells)
    int2 *pp = reinterpret_cast<int2 *>(a.path + 2 * ((size_t)d0 + (size_t)t0));
    int carry = -1;
    for (int q0 = 0; q0 < n; q0 += kWave) {
        const int q = q0 + lane;
        const int row = max(scan_max(s.rowmax[q0 + lane]), carry);
        carry = __builtin_amdgcn_readlane(row, kWave - 1);
        const int r = row < 0 ? 0 : row;
        const int rx = __shfl(x, r);
        const int ro = __shfl(off, r);
        if (q < n) pp[q] = make_int2(r, rx - 1 + (q - ro));
    }
    // column j: the last row whose run starts at or before j
    const int mj = scan_max(s.colmax[lane]);
    if (lane < M) a.map[t0 + lane] = mj;
    return lane < M ? mj : -1;
}

}  // namespace rows
}  // namespace tt
