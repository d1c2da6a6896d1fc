// Dynamic Token Warping on gfx950: one wave64 per (draft, proxy-target) pair.
//
// Computes Alg. 1 of the paper (cumulative cost C over draft x target tokens with
// the Sakoe-Chiba band, Sec. 4.1) using the byte-level Levenshtein token distance
// of App. H, then the backtrack from (K, M) and the mapping of App. A.2.
//
// Work decomposition (per workgroup = one wave = one pair):
//   * Draft rows are processed in strips of 64; lane r owns row i = i0 + r.  Within
//     a strip the wave sweeps anti-diagonals: at step t lane r computes cell
//     (i0 + r, jfirst + t - r).  C(i-1, j) arrives from lane r-1 by a one-lane
//     shuffle, C(i-1, j-1) is the value received one step earlier, C(i, j-1) is the
//     lane's own previous value; lane 0 reads the previous strip's last row from LDS.
//   * The token distance is evaluated on the fly with the bit-parallel edit-distance
//     recurrence (Myers 1999, in Hyyro's 2001 global-distance form): the draft token
//     is the pattern (one bit per byte, at most 64), the target token's bytes are the
//     text, and the per-byte match masks come from SWAR byte comparison of the packed
//     pattern.
//   * Each cell's predecessor choice is a 2-bit code packed 16 per dword, row-major
//     inside the band, kept in LDS; a single lane walks the codes back from (K, M).
//   * Target token bytes are staged once per pair in LDS (fixed-width slots).
//
// LDS layout (bytes, each region 16-byte aligned):
//   slots  [max_m][TB]  target token bytes      tlen [max_m] u8 lengths
//   row0   [max_m+1]    int32 C of the row above the strip (double-buffered with row1)
//   path   [max_k+max_m] u32 backtracked cells (i << 16 | j), reverse order
//   codes  [max_k][WPR] u32 direction codes (WPR = ceil(min(max_m, 2 L_max + 1) / 16))
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
    size_t slots, tlen, row0, row1, path, codes, total;
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
    size_t wpr = (size_t)((W + 15) / 16);
    size_t off = 0;
    p.slots = off;
    off = align16(off + (size_t)max_m * tb);
    p.tlen = off;
    off = align16(off + (size_t)max_m);
    p.row0 = off;
    off = align16(off + 4 * ((size_t)max_m + 1));
    p.row1 = off;
    off = align16(off + 4 * ((size_t)max_m + 1));
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
__device__ __forceinline__ int token_distance(const uint32_t (&xw)[TB / 4], int m,
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

template <int TB>
__device__ __forceinline__ void load_token(const uint8_t *bytes, int start, int len, uint32_t (&w)[TB / 4]) {
#pragma unroll
    for (int q = 0; q < TB / 4; ++q) w[q] = 0;
#pragma unroll
    for (int k = 0; k < TB; ++k)
        if (k < len) w[k >> 2] |= (uint32_t)bytes[start + k] << (8 * (k & 3));
}

__device__ __forceinline__ bool token_ok(const tt_vocab &v, int32_t id) {
    if (id < 0 || id >= v.n_tokens) return false;
    const int32_t len = v.offsets[id + 1] - v.offsets[id];
    return len >= 0 && len <= v.max_token_bytes;
}

template <int TB>
__global__ void __launch_bounds__(kWave) dtw_band_wave(AlignArgs a, LdsPlan lp) {
    extern __shared__ __align__(16) uint8_t lds[];
    const int b = blockIdx.x;
    const int lane = threadIdx.x;
    const int d0 = a.draft_off[b], K = a.draft_off[b + 1] - d0;
    const int t0 = a.target_off[b], M = a.target_off[b + 1] - t0;

    // ---- validation: lengths within bounds, ids inside their tables, token lengths bounded
    bool ok = K >= 1 && K <= a.max_k && M >= 1 && M <= a.max_m;
    if (ok) {
        bool bad = false;
        for (int i = lane; i < K; i += kWave) bad |= !token_ok(a.vd, a.draft_ids[d0 + i]);
        for (int j = lane; j < M; j += kWave) bad |= !token_ok(a.vt, a.target_ids[t0 + j]);
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

    uint32_t *slots = reinterpret_cast<uint32_t *>(lds + lp.slots);
    uint8_t *tlen = lds + lp.tlen;
    int *rowIn = reinterpret_cast<int *>(lds + lp.row0);
    int *rowOut = reinterpret_cast<int *>(lds + lp.row1);
    uint32_t *pathbuf = reinterpret_cast<uint32_t *>(lds + lp.path);
    uint32_t *codes = reinterpret_cast<uint32_t *>(lds + lp.codes);

    // ---- stage the target tokens' bytes
    for (int j = lane; j < M; j += kWave) {
        const int id = a.target_ids[t0 + j];
        const int s = a.vt.offsets[id];
        const int n = a.vt.offsets[id + 1] - s;
        uint32_t w[TB / 4];
        load_token<TB>(a.vt.bytes, s, n, w);
#pragma unroll
        for (int q = 0; q < TB / 4; ++q) slots[j * (TB / 4) + q] = w[q];
        tlen[j] = (uint8_t)n;
    }

    // ---- band geometry for this pair
    const int mx = K > M ? K : M;
    int L = (a.w < 0) ? mx : (a.w > abs(K - M) ? a.w : abs(K - M));
    if (L > mx) L = mx;
    const int W = (2 * L + 1 < M) ? 2 * L + 1 : M;
    const int WPR = (W + 15) >> 4;

    for (int j = lane; j <= M; j += kWave) rowIn[j] = (j == 0) ? 0 : kInf;  // C(0, j)
    __syncthreads();

    for (int i0 = 1; i0 <= K; i0 += kWave) {
        const int rows = (K - i0 + 1) < kWave ? (K - i0 + 1) : kWave;
        const int i = i0 + lane;
        const bool act = lane < rows;
        uint32_t xw[TB / 4];
        int m = 0;
        if (act) {
            const int id = a.draft_ids[d0 + i - 1];
            const int s = a.vd.offsets[id];
            m = a.vd.offsets[id + 1] - s;
            load_token<TB>(a.vd.bytes, s, m, xw);
        } else {
#pragma unroll
            for (int q = 0; q < TB / 4; ++q) xw[q] = 0;
        }
        const int myjlo = (i - L) > 1 ? (i - L) : 1;
        const int myjhi = (i + L) < M ? (i + L) : M;
        const int jfirst = (i0 - L) > 1 ? (i0 - L) : 1;
        const int jlast = (i0 + rows - 1 + L) < M ? (i0 + rows - 1 + L) : M;
        const int steps = (jlast - jfirst + 1) + rows - 1;
        uint32_t *mycodes = codes + (size_t)(i - 1) * WPR;

        for (int j = lane; j <= M; j += kWave) rowOut[j] = kInf;
        __syncthreads();

        int cur = kInf, above_prev = kInf;
        uint32_t cw = 0;
        for (int t = 0; t < steps; ++t) {
            const int j = jfirst + t - lane;
            int above = __shfl_up(cur, 1);  // C(i-1, j) computed by lane-1 at step t-1
            int diagv = above_prev;          // C(i-1, j-1): received at step t-1
            if (lane == 0) {
                above = (j >= 0 && j <= M) ? rowIn[j] : kInf;
                diagv = (j - 1 >= 0 && j - 1 <= M) ? rowIn[j - 1] : kInf;
            }
            above_prev = above;
            const int left = cur;  // C(i, j-1)
            if (act && j >= myjlo && j <= myjhi) {
                uint32_t yw[TB / 4];
#pragma unroll
                for (int q = 0; q < TB / 4; ++q) yw[q] = slots[(j - 1) * (TB / 4) + q];
                const int n = tlen[j - 1];
                const int d = token_distance<TB>(xw, m, yw, n);
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
        while ((ii > 0 || jj > 0) && n < cap && ii >= 1 && jj >= 1) {
            pathbuf[n++] = ((uint32_t)ii << 16) | (uint32_t)jj;
            const int jl = (ii - L) > 1 ? (ii - L) : 1;
            const int c = jj - jl;
            if (c < 0 || c >= W) break;  // never taken: every path cell lies inside the band
            const uint32_t word = codes[(size_t)(ii - 1) * WPR + (c >> 4)];
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
