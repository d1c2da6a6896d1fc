// Dynamic Token Warping on gfx950: one wave64 per (draft, proxy-target) pair.
//
// Computes Alg. 1 of the paper (cumulative cost C over draft x target tokens with
// the Sakoe-Chiba band, Sec. 4.1) using the byte-level Levenshtein token distance
// of App. H, then the backtrack from (K, M) and the mapping of App. A.2.
//
// Work decomposition (per workgroup = one wave = one pair):
//   * Staging: every lane loads one token (draft or target) -- id, byte offsets,
//     bytes -- validates it and packs it into a fixed-width LDS slot.
//   * Draft rows are processed in strips of 64.  For a strip, all 64 lanes first
//     evaluate the token distance of every band cell of the strip (cell-parallel)
//     into an LDS byte matrix.  Then the wave sweeps the strip's anti-diagonals with
//     lane r owning row i = i0 + r: at step t lane r finishes cell (i0 + r,
//     jfirst + t - r).  C(i-1, j) arrives from lane r-1 by a DPP wave shift,
//     C(i-1, j-1) is the value received one step earlier, C(i, j-1) is the lane's own
//     previous value; lane 0 reads the previous strip's last row from LDS.
//   * Token distance: the bit-parallel edit-distance recurrence (Myers 1999, in
//     Hyyro's 2001 global-distance form) with the longer token as the pattern (one
//     bit per byte, at most 64) and the shorter one as the text; per-byte match masks
//     come from SWAR byte comparison of the packed pattern.
//   * Each cell's predecessor choice is a 2-bit code packed 16 per dword, row-major
//     inside the band, kept in LDS; a single lane walks the codes back from (K, M),
//     re-reading a code word only when the walk leaves it.
//
// LDS layout (bytes, each region 16-byte aligned):
//   tslot [max_m][TB] / tlen [max_m]   target token bytes and lengths
//   dslot [max_k][TB] / dlen [max_k]   draft token bytes and lengths
//   row0, row1 [max_m+1] int32         C of the row above the strip (double-buffered)
//   cost  [min(64,max_k)][Wmax] u8     token distances of the current strip
//   path  [max_k+max_m] u32            backtracked cells (i << 16 | j), reverse order
//   codes [max_k][WPR] u32             direction codes, WPR = ceil(Wmax / 16)
// with Wmax = min(max_m, 2 L + 1) for the largest band half-width L the bounds allow.
#include "tt_internal.h"

namespace tt {
namespace {

constexpr int kInf = 0x3fffffff;
constexpr int kWave = 64;
constexpr size_t kLdsLimit = 160 * 1024;  // gfx950 LDS per workgroup

template <int TB>
struct MaskType {
    using type = uint32_t;
};
template <>
struct MaskType<64> {
    using type = uint64_t;
};

__host__ __device__ inline size_t align16(size_t v) { return (v + 15) & ~size_t(15); }

struct LdsPlan {
    size_t tslot, tlen, dslot, dlen, row0, row1, cost, path, codes, total;
};

__host__ __device__ inline int band_half_width_bound(int32_t max_k, int32_t max_m, int32_t w) {
    int mx = max_k > max_m ? max_k : max_m;
    if (w < 0) return mx;
    int widen = mx - 1;  // largest possible |K - M|
    int L = w > widen ? w : widen;
    return L < mx ? L : mx;
}

__host__ __device__ inline LdsPlan plan_lds(int32_t max_k, int32_t max_m, int32_t w, int tb) {
    LdsPlan p;
    int L = band_half_width_bound(max_k, max_m, w);
    long long W = 2LL * L + 1;
    if (W > max_m) W = max_m;
    const size_t wpr = (size_t)((W + 15) / 16);
    const size_t strip_rows = max_k < 64 ? (size_t)max_k : 64;
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
    off = align16(off + 4 * ((size_t)max_m + 1));
    p.row1 = off;
    off = align16(off + 4 * ((size_t)max_m + 1));
    p.cost = off;
    off = align16(off + strip_rows * (size_t)W);
    p.path = off;
    off = align16(off + 4 * ((size_t)max_k + (size_t)max_m));
    p.codes = off;
    off = align16(off + 4 * (size_t)max_k * wpr);
    p.total = off;
    return p;
}

// High bit of each byte of w that equals the byte broadcast in bc, compressed to 4 bits.
__device__ __forceinline__ uint32_t byte_match4(uint32_t w, uint32_t bc) {
    uint32_t t = w ^ bc;
    uint32_t z = ~(((t & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | t) & 0x80808080u;
    return (((z >> 7) * 0x00204081u) >> 21) & 0xFu;
}

// Edit distance between the packed pattern xw (m bytes) and the text bytes in yw (n bytes).
template <int TB>
__device__ __forceinline__ int bitparallel_distance(const uint32_t (&xw)[TB / 4], int m,
                                                    const uint32_t (&yw)[TB / 4], int n) {
    using M = typename MaskType<TB>::type;
    if (m == 0) return n;
    const M lim = (m >= (int)(8 * sizeof(M))) ? ~M(0) : ((M(1) << m) - 1);
    const M hib = M(1) << (m - 1);
    M vp = ~M(0), vn = 0;
    int score = m;
#pragma unroll
    for (int k = 0; k < TB; ++k) {
        if (k < n) {
            const uint32_t c = (yw[k >> 2] >> (8 * (k & 3))) & 0xFFu;
            const uint32_t bc = c * 0x01010101u;
            M eq = 0;
#pragma unroll
            for (int q = 0; q < TB / 4; ++q) eq |= M(byte_match4(xw[q], bc)) << (4 * q);
            eq &= lim;
            const M xv = eq | vn;
            const M xh = (((eq & vp) + vp) ^ vp) | eq;
            M hp = vn | ~(xh | vp);
            M hn = vp & xh;
            score += (hp & hib) ? 1 : 0;
            score -= (hn & hib) ? 1 : 0;
            hp = (hp << 1) | M(1);
            hn = hn << 1;
            vp = hn | ~(xv | hp);
            vn = hp & xv;
        }
    }
    return score;
}

// Edit distance is symmetric: iterate over the shorter token, the longer one is the pattern.
template <int TB>
__device__ __forceinline__ int token_distance(const uint32_t (&aw)[TB / 4], int m,
                                              const uint32_t (&bw)[TB / 4], int n) {
    const bool swap = n > m;
    uint32_t pw[TB / 4], tw[TB / 4];
#pragma unroll
    for (int q = 0; q < TB / 4; ++q) {
        pw[q] = swap ? bw[q] : aw[q];
        tw[q] = swap ? aw[q] : bw[q];
    }
    return bitparallel_distance<TB>(pw, swap ? n : m, tw, swap ? m : n);
}

// Loads, checks and packs token `id` of table v into an LDS slot; false if invalid.
template <int TB>
__device__ __forceinline__ bool stage_token(const tt_vocab &v, int32_t id, uint32_t *slot, uint8_t *len_out) {
    if (id < 0 || id >= v.n_tokens) return false;
    const int s = v.offsets[id];
    const int len = v.offsets[id + 1] - s;
    if (len < 0 || len > v.max_token_bytes || len > TB) return false;
    uint32_t w[TB / 4];
#pragma unroll
    for (int q = 0; q < TB / 4; ++q) w[q] = 0;
#pragma unroll
    for (int k = 0; k < TB; ++k)
        if (k < len) w[k >> 2] |= (uint32_t)v.bytes[s + k] << (8 * (k & 3));
#pragma unroll
    for (int q = 0; q < TB / 4; ++q) slot[q] = w[q];
    *len_out = (uint8_t)len;
    return true;
}

template <int TB>
__device__ __forceinline__ void read_slot(const uint32_t *slot, uint32_t (&w)[TB / 4]) {
#pragma unroll
    for (int q = 0; q < TB / 4; ++q) w[q] = slot[q];
}

// C(i-1, .) from the lane below: DPP wave shift right by one lane (lane 0 gets `fill`).
__device__ __forceinline__ int from_lane_below(int v, int fill) {
    return __builtin_amdgcn_update_dpp(fill, v, 0x138 /* wave_shr:1 */, 0xF, 0xF, false);
}

template <int TB>
__global__ void __launch_bounds__(kWave) dtw_band_wave(AlignArgs a, LdsPlan lp) {
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
    uint8_t *costbuf = lds + lp.cost;
    uint32_t *pathbuf = reinterpret_cast<uint32_t *>(lds + lp.path);
    uint32_t *codes = reinterpret_cast<uint32_t *>(lds + lp.codes);

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
    const int mx = K > M ? K : M;
    int L = (a.w < 0) ? mx : (a.w > abs(K - M) ? a.w : abs(K - M));
    if (L > mx) L = mx;
    const int W = (2 * L + 1 < M) ? 2 * L + 1 : M;
    const int WPR = (W + 15) >> 4;
    const float invW = 1.0f / (float)W;

    for (int j = lane; j <= M; j += kWave) rowIn[j] = (j == 0) ? 0 : kInf;  // C(0, j)
    __syncthreads();

    for (int i0 = 1; i0 <= K; i0 += kWave) {
        const int rows = (K - i0 + 1) < kWave ? (K - i0 + 1) : kWave;

        // ---- token distances of every band cell of the strip (cell-parallel)
        const int ncell = rows * W;
        for (int idx = lane; idx < ncell; idx += kWave) {
            int r = (int)((float)idx * invW);
            int c = idx - r * W;
            if (c < 0) {
                --r;
                c += W;
            } else if (c >= W) {
                ++r;
                c -= W;
            }
            const int i = i0 + r;
            const int jl = (i - L) > 1 ? (i - L) : 1;
            const int jh = (i + L) < M ? (i + L) : M;
            const int j = jl + c;
            if (j <= jh) {
                uint32_t xw[TB / 4], yw[TB / 4];
                read_slot<TB>(dslot + (i - 1) * (TB / 4), xw);
                read_slot<TB>(tslot + (j - 1) * (TB / 4), yw);
                costbuf[r * W + c] = (uint8_t)token_distance<TB>(xw, dlen[i - 1], yw, tlen[j - 1]);
            }
        }
        for (int j = lane; j <= M; j += kWave) rowOut[j] = kInf;
        __syncthreads();

        // ---- anti-diagonal sweep, lane = row
        const int i = i0 + lane;
        const bool act = lane < rows;
        const int myjlo = (i - L) > 1 ? (i - L) : 1;
        const int myjhi = (i + L) < M ? (i + L) : M;
        const int jfirst = (i0 - L) > 1 ? (i0 - L) : 1;
        const int jlast = (i0 + rows - 1 + L) < M ? (i0 + rows - 1 + L) : M;
        const int steps = (jlast - jfirst + 1) + rows - 1;
        const uint8_t *mycost = costbuf + lane * W;
        uint32_t *mycodes = codes + (size_t)(i - 1) * WPR;

        int cur = kInf, above_prev = kInf;
        uint32_t cw = 0;
        for (int t = 0; t < steps; ++t) {
            const int j = jfirst + t - lane;
            const bool inb = act && j >= myjlo && j <= myjhi;
            const int d = inb ? (int)mycost[j - myjlo] : 0;
            int above = from_lane_below(cur, kInf);  // C(i-1, j): lane-1 at step t-1
            int diagv = above_prev;                  // C(i-1, j-1): received at step t-1
            if (lane == 0) {
                above = (j >= 0 && j <= M) ? rowIn[j] : kInf;
                diagv = (j >= 1 && j - 1 <= M) ? rowIn[j - 1] : kInf;
            }
            above_prev = above;
            const int left = cur;  // C(i, j-1)
            if (inb) {
                int best = diagv, code = 0;  // ties: diagonal, then (i-1, j), then (i, j-1)
                if (above < best) {
                    best = above;
                    code = 1;
                }
                if (left < best) {
                    best = left;
                    code = 2;
                }
                cur = d + best;
                const int c = j - myjlo;
                cw |= (uint32_t)code << (2 * (c & 15));
                if ((c & 15) == 15 || j == myjhi) {
                    mycodes[c >> 4] = cw;
                    cw = 0;
                }
                if (i == K && j == M) a.cost[b] = cur;
            } else {
                cur = kInf;
            }
            if (act && lane == rows - 1 && j >= 0 && j <= M) rowOut[j] = cur;
        }
        __syncthreads();
        int *tmp = rowIn;
        rowIn = rowOut;
        rowOut = tmp;
    }

    // ---- backtrack from (K, M) following the stored predecessor codes
    __shared__ int s_n;
    if (lane == 0) {
        int ii = K, jj = M, n = 0;
        const int cap = K + M;
        int cached = -1;
        uint32_t word = 0;
        while (n < cap && ii >= 1 && jj >= 1) {
            pathbuf[n++] = ((uint32_t)ii << 16) | (uint32_t)jj;
            const int jl = (ii - L) > 1 ? (ii - L) : 1;
            const int c = jj - jl;
            if (c < 0 || c >= W) break;  // never taken: every path cell lies inside the band
            const int widx = (ii - 1) * WPR + (c >> 4);
            if (widx != cached) {
                word = codes[widx];
                cached = widx;
            }
            const int code = (word >> (2 * (c & 15))) & 3;
            if (code == 0) {
                --ii;
                --jj;
            } else if (code == 1) {
                --ii;
            } else {
                --jj;
            }
        }
        s_n = n;
        a.path_len[b] = n;
    }
    __syncthreads();
    const int n = s_n;
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
int launch_tb(const AlignArgs &a, hipStream_t stream) {
    const LdsPlan lp = plan_lds(a.max_k, a.max_m, a.w, TB);
    if (lp.total > kLdsLimit) return TT_EUNSUPPORTED;
    if (lp.total > 64 * 1024) {
        if (hipFuncSetAttribute(reinterpret_cast<const void *>(&dtw_band_wave<TB>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lp.total) != hipSuccess)
            return TT_ELAUNCH;
    }
    hipLaunchKernelGGL(dtw_band_wave<TB>, dim3(a.n_pairs), dim3(kWave), lp.total, stream, a, lp);
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

int launch_align(const AlignArgs &a, hipStream_t stream) {
    const int mt = a.vd.max_token_bytes > a.vt.max_token_bytes ? a.vd.max_token_bytes : a.vt.max_token_bytes;
    switch (align_token_slot(mt)) {
        case 8: return launch_tb<8>(a, stream);
        case 16: return launch_tb<16>(a, stream);
        case 32: return launch_tb<32>(a, stream);
        case 64: return launch_tb<64>(a, stream);
        default: return TT_EUNSUPPORTED;
    }
}

}  // namespace tt
