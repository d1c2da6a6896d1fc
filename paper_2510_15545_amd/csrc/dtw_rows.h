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
//     recurrence and leaves C in LDS; then every wave turns rows of C into two 64-bit
//     column masks per row ("not a left move", "diagonal move") with ballots.
//   * Backtrack: inside row i the path runs left from its entry column e to the highest
//     column x <= e whose move is not a left move, then enters row i-1 at x - 1
//     (diagonal) or x.  That is one find-last-set per row on the scalar unit.
//   * Row i covers columns [x_i, e_i]; each row's lane writes its path cells and the map
//     entries of its columns (a column shared with the row below by an (i-1, j) move
//     belongs to the higher row: the map holds the largest draft index).
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
    uint64_t nl[kMaxSide], dg[kMaxSide];  // move masks of row i at [i - 1]
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

// Every wave: the move masks of rows wave + 1, wave + 1 + nwaves, ... from C in LDS.
template <int TB>
__device__ __forceinline__ void moves(Lds<TB> &s, int K, int M, int L, int wave, int nwaves) {
    const int lane = threadIdx.x % kWave;
    const int j = lane + 1;
    for (int i = 1 + wave; i <= K; i += nwaves) {
        const bool inb = j <= M && j >= i - L && j <= i + L;
        const int diag = s.cm[(i - 1) * kCmLd + j - 1];
        const int up = s.cm[(i - 1) * kCmLd + j];
        const int left = s.cm[i * kCmLd + j - 1];
        const bool not_left = !(left < min(diag, up));
        const uint64_t nl = __ballot(inb && not_left);
        const uint64_t dg = __ballot(inb && not_left && diag <= up);
        if (lane == 0) {
            s.nl[i - 1] = nl;
            s.dg[i - 1] = dg;
        }
    }
}

// One wave: backtrack from (K, M) over the move masks, then cost, path_len, path and map
// of pair b.  When map_lds is given, map_lds[j - 1] also receives i*(j) (0-based).
template <int TB>
__device__ __forceinline__ void backtrack(const AlignArgs &a, const Lds<TB> &s, int b, int d0, int K, int t0,
                                          int M, int total, int *map_lds) {
    const int lane = threadIdx.x % kWave;
    const uint64_t nl_mask = lane < K ? s.nl[lane] : 0ull;  // row lane + 1
    const uint64_t dg_mask = lane < K ? s.dg[lane] : 0ull;
    int e = M, n = 0;
    int seg_x = 1, seg_e = 0;  // row lane + 1 covers columns [seg_x, seg_e] (empty if unvisited)
    for (int i = K; i >= 1; --i) {
        const uint64_t nl = lane_u64(nl_mask, i - 1);
        const uint64_t dg = lane_u64(dg_mask, i - 1);
        const uint64_t cand = nl & (e >= 64 ? ~0ull : ((1ull << e) - 1));  // e = 0: nothing left
        const int x = cand ? 64 - __clzll(cand) : 0;  // highest not-left column <= e; 0 if none
        seg_x = (lane == i - 1 && x > 0) ? x : seg_x;
        seg_e = (lane == i - 1 && x > 0) ? e : seg_e;
        n += x > 0 ? e - x + 1 : 0;
        e = x > 0 ? (((dg >> (x - 1)) & 1ull) ? x - 1 : x) : 0;
    }
    if (lane == 0) {
        a.cost[b] = total;
        a.path_len[b] = n;
    }
    // each row's lane writes its cells; the column it shares with the row below through an
    // (i-1, j) move is that row's map entry
    const int len = seg_e - seg_x + 1;  // 0 for rows the walk never reached
    const int off = scan_add(len) - len;
    const int x_up = __builtin_amdgcn_update_dpp(0, seg_x, 0x130 /* wave_shl:1 */, 0xF, 0xF, false);
    const int len_up = __builtin_amdgcn_update_dpp(0, len, 0x130 /* wave_shl:1 */, 0xF, 0xF, false);
    const int mlen = (lane + 1 < K && len > 0 && len_up > 0 && x_up == seg_e) ? len - 1 : len;
    int2 *pp = reinterpret_cast<int2 *>(a.path + 2 * ((size_t)d0 + (size_t)t0));
    for (int k = 0; __any(k < len); ++k) {
        if (k < len) pp[off + k] = make_int2(lane, seg_x - 1 + k);
        if (k < mlen) {
            a.map[t0 + seg_x - 1 + k] = lane;
            if (map_lds != nullptr) map_lds[seg_x - 1 + k] = lane;
        }
    }
}

}  // namespace rows
}  // namespace tt
