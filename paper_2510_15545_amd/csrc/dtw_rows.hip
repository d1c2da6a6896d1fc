// Dynamic Token Warping for short pairs (K <= 64 draft tokens, M <= 64 target tokens),
// one 256-thread workgroup per pair.
//
// Same outputs as the strip kernel (Alg. 1 with the Sakoe-Chiba band of Sec. 4.1, the
// byte Levenshtein distance of App. H, backtrack from (K, M) with ties to the diagonal,
// then (i-1, j), then (i, j-1), and the mapping of App. A.2), computed row by row with
// lane = column instead of along anti-diagonals:
//
//   * Staging and token distances use all four waves: every band cell's distance is one
//     thread's work, written to an LDS byte matrix [i][j].
//   * Row i of the cumulative cost follows from row i-1 with two wave scans.  With
//     U(j) = d(i, j) + min(C(i-1, j-1), C(i-1, j)) and S(j) the prefix sum of d(i, .)
//     over the band,  C(i, j) = S(j) + min over k <= j of (U(k) - S(k)): the left moves
//     inside a row are a (min, +) prefix scan.  Out-of-band cells are infinite.
//   * A cell's predecessor is (i, j-1) iff C(i, j-1) < min(C(i-1, j-1), C(i-1, j)), else
//     the diagonal iff C(i-1, j-1) <= C(i-1, j), else (i-1, j).  Two ballots per row keep
//     "not a left move" and "diagonal move" as 64-bit column masks; lane i-1 holds row i's.
//   * Backtrack: inside row i the path runs left from its entry column e to the highest
//     column x <= e whose move is not a left move, then enters row i-1 at x - 1
//     (diagonal) or x.  That is one find-last-set per row on the scalar unit.
//   * Row i covers columns [x_i, e_i]; the path and the mapping are written lane-parallel
//     from those segments (column j maps to the last row whose segment starts at or
//     before j: x_i is non-decreasing in i).
#include "dtw_common.h"

namespace tt {
namespace {

using dtw::kInf;
using dtw::kWave;

constexpr int kThreads = 256;
constexpr int kMaxSide = 64;  // bound on K and M for this kernel

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

__device__ __forceinline__ int scan_min(int v) {
    v = min(v, dpp_from<0x111, 0xF>(v, kInf));
    v = min(v, dpp_from<0x112, 0xF>(v, kInf));
    v = min(v, dpp_from<0x114, 0xF>(v, kInf));
    v = min(v, dpp_from<0x118, 0xF>(v, kInf));
    v = min(v, dpp_from<0x142, 0xA>(v, kInf));
    v = min(v, dpp_from<0x143, 0xC>(v, kInf));
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

template <int TB>
__global__ void __launch_bounds__(kThreads) dtw_rows(AlignArgs a) {
    __shared__ uint32_t tslot[kMaxSide * (TB / 4)];
    __shared__ uint32_t dslot[kMaxSide * (TB / 4)];
    __shared__ uint8_t tlen[kMaxSide];
    __shared__ uint8_t dlen[kMaxSide];
    __shared__ uint8_t cost[kMaxSide * kMaxSide];  // d(i, j) at [(i-1) * 64 + j - 1]

    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    const int d0 = a.draft_off[b], K = a.draft_off[b + 1] - d0;
    const int t0 = a.target_off[b], M = a.target_off[b + 1] - t0;

    // ---- staging + validation: one token (draft or target) per thread
    const bool shape_ok = K >= 1 && K <= a.max_k && M >= 1 && M <= a.max_m;
    int bad = shape_ok ? 0 : 1;
    if (shape_ok) {
        for (int e = tid; e < K + M; e += kThreads) {
            const bool ok = e < K ? dtw::stage_token<TB>(a.vd, a.draft_ids[d0 + e], dslot + e * (TB / 4), dlen + e)
                                  : dtw::stage_token<TB>(a.vt, a.target_ids[t0 + e - K],
                                                         tslot + (e - K) * (TB / 4), tlen + (e - K));
            bad |= ok ? 0 : 1;
        }
    }
    if (__syncthreads_or(bad)) {
        if (tid == 0) {
            a.cost[b] = -1;
            a.path_len[b] = 0;
        }
        for (int j = tid; j < M; j += kThreads) a.map[t0 + j] = -1;
        return;
    }

    // ---- band: |i - j| <= L with L = max(w, |K - M|) (w < 0: no band)
    const int mx = K > M ? K : M;
    int L = (a.w < 0) ? mx : (a.w > abs(K - M) ? a.w : abs(K - M));
    if (L > mx) L = mx;

    // ---- token distance of every band cell, one cell per thread
    const float invM = 1.0f / (float)M;
    for (int idx = tid; idx < K * M; idx += kThreads) {
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
            dtw::read_slot<TB>(dslot + r * (TB / 4), xw);
            dtw::read_slot<TB>(tslot + c * (TB / 4), yw);
            cost[r * kMaxSide + c] = (uint8_t)dtw::token_distance<TB>(xw, dlen[r], yw, tlen[c]);
        }
    }
    __syncthreads();
    if (tid >= kWave) return;  // one wave from here on

    // ---- cumulative cost, one row per iteration, lane = column j - 1
    const int j = lane + 1;
    int cprev = kInf;  // C(i-1, j); row 0 is infinite except C(0, 0) = 0
    uint64_t nl_mask = 0, dg_mask = 0;  // row lane + 1: not-left moves, diagonal moves
    int dnext = cost[lane];
    for (int i = 1; i <= K; ++i) {
        const int d = dnext;
        if (i < K) dnext = cost[i * kMaxSide + lane];
        const bool inb = j <= M && j >= i - L && j <= i + L;
        const int diag = from_lane_below(cprev, i == 1 ? 0 : kInf);
        const int up = cprev;
        const int m = min(diag, up);
        const int s = scan_add(inb ? d : 0);
        const int p = scan_min(inb ? m + d - s : kInf);
        const int c = inb ? min(s + p, kInf) : kInf;
        const int left = from_lane_below(c, kInf);  // C(i, j-1)
        const uint64_t nl = __ballot(inb && !(left < m));
        const uint64_t dg = __ballot(inb && !(left < m) && diag <= up);
        nl_mask = (lane == i - 1) ? nl : nl_mask;
        dg_mask = (lane == i - 1) ? dg : dg_mask;
        cprev = c;
    }
    const int total = __builtin_amdgcn_readlane(cprev, M - 1);

    // ---- backtrack from (K, M), one row per step
    int e = M, n = 0;
    int seg_x = 1, seg_e = 0;  // row lane + 1 covers columns [seg_x, seg_e] (empty if unvisited)
    for (int i = K; i >= 1 && e >= 1; --i) {
        const uint64_t nl = lane_u64(nl_mask, i - 1);
        const uint64_t cand = nl & (e >= 64 ? ~0ull : ((1ull << e) - 1));
        if (cand == 0) break;  // never taken: a left run always ends inside the band
        const int x = 64 - __clzll(cand);
        seg_x = (lane == i - 1) ? x : seg_x;
        seg_e = (lane == i - 1) ? e : seg_e;
        n += e - x + 1;
        const uint64_t dg = lane_u64(dg_mask, i - 1);
        e = ((dg >> (x - 1)) & 1ull) ? x - 1 : x;
    }
    if (lane == 0) {
        a.cost[b] = total;
        a.path_len[b] = n;
    }

    // ---- path (forward order) and mapping from the row segments
    const int len = seg_e - seg_x + 1;  // 0 for rows the walk never reached
    const int off = scan_add(len) - len;
    int32_t *pp = a.path + 2 * ((size_t)d0 + (size_t)t0);
    for (int q0 = 0; q0 < n; q0 += kWave) {  // uniform loop: the shuffles need every lane
        const int q = q0 + lane;
        int row = 0;  // last visited row whose segment starts at or before path index q
        for (int r = 0; r < K; ++r) {
            const int o = __builtin_amdgcn_readlane(off, r);
            const int l = __builtin_amdgcn_readlane(len, r);
            row = (l > 0 && o <= q) ? r : row;
        }
        const int rx = __shfl(seg_x, row);
        const int ro = __shfl(off, row);
        if (q < n) {
            pp[2 * q] = row;
            pp[2 * q + 1] = rx - 1 + (q - ro);
        }
    }
    if (j <= M) {
        int last = -1;  // last visited row whose segment starts at or before column j
        for (int r = 0; r < K; ++r) {
            const int x = __builtin_amdgcn_readlane(seg_x, r);
            const int l = __builtin_amdgcn_readlane(len, r);
            last = (l > 0 && x <= j) ? r : last;
        }
        a.map[t0 + lane] = last;
    }
}

template <int TB>
int launch_rows_tb(const AlignArgs &a, hipStream_t stream) {
    hipLaunchKernelGGL(dtw_rows<TB>, dim3(a.n_pairs), dim3(kThreads), 0, stream, a);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

}  // namespace

bool align_rows_fits(int32_t max_k, int32_t max_m) { return max_k <= kMaxSide && max_m <= kMaxSide; }

int launch_align_rows(const AlignArgs &a, int tb, hipStream_t stream) {
    switch (tb) {
        case 8: return launch_rows_tb<8>(a, stream);
        case 16: return launch_rows_tb<16>(a, stream);
        case 32: return launch_rows_tb<32>(a, stream);
        case 64: return launch_rows_tb<64>(a, stream);
        default: return TT_EUNSUPPORTED;
    }
}

}  // namespace tt
