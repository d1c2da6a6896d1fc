// Device helpers shared by the two alignment kernels: token staging and the byte-level
// Levenshtein distance of App. H.  Internal to the library.
#pragma once

#include "tt_internal.h"

namespace tt {
namespace dtw {

constexpr int kInf = 0x3fffffff;  // cost of an unreachable cell
constexpr int kWave = 64;

// Bit vector holding one bit per pattern byte for a token slot of TB bytes.
template <int TB>
struct MaskType {
    using type = uint32_t;
};
template <>
struct MaskType<64> {
    using type = uint64_t;
};

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
            const uint32_t bc = __builtin_amdgcn_perm(0u, c, 0u);  // c in all four bytes
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
// The token's bytes come from the aligned dwords that overlap them, all loads issued
// together (a dword holding one of the token's bytes lies in the same page as that byte).
template <int TB>
__device__ __forceinline__ bool stage_token(const tt_vocab &v, int32_t id, uint32_t *slot, uint8_t *len_out) {
    if (id < 0 || id >= v.n_tokens) return false;
    const int s = v.offsets[id];
    const int len = v.offsets[id + 1] - s;
    if (len < 0 || len > v.max_token_bytes || len > TB) return false;
    const uint8_t *bp = v.bytes + s;
    const int mis = (int)(reinterpret_cast<uintptr_t>(bp) & 3u);
    const uint32_t sh = (uint32_t)mis * 8;
    const int nd = len > 0 ? ((mis + len - 1) >> 2) + 1 : 0;  // dwords touched, <= TB / 4 + 1
    const uint32_t *d = reinterpret_cast<const uint32_t *>(bp - mis);
    uint32_t raw[TB / 4 + 1];
#pragma unroll
    for (int q = 0; q < TB / 4 + 1; ++q) raw[q] = q < nd ? d[q] : 0u;
#pragma unroll
    for (int q = 0; q < TB / 4; ++q) {
        const uint32_t word = __builtin_amdgcn_alignbit(raw[q + 1], raw[q], sh);
        const int keep = len - 4 * q;  // bytes of the token in this word
        const uint32_t mask = keep >= 4 ? ~0u : (keep <= 0 ? 0u : ((1u << (8 * keep)) - 1u));
        slot[q] = word & mask;
    }
    *len_out = (uint8_t)len;
    return true;
}

template <int TB>
__device__ __forceinline__ void read_slot(const uint32_t *slot, uint32_t (&w)[TB / 4]) {
#pragma unroll
    for (int q = 0; q < TB / 4; ++q) w[q] = slot[q];
}

// Workgroup-wide OR of per-thread flag bits through one barrier: every wave leaves its
// votes in LDS (votes[nwaves]).
__device__ __forceinline__ int block_or(int flags, int *votes, int nwaves) {
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    int v = 0;
    for (int bit = 1; bit <= 2; bit <<= 1) v |= __any(flags & bit) ? bit : 0;
    if (lane == 0) votes[wave] = v;
    __syncthreads();
    int all = 0;
    for (int w = 0; w < nwaves; ++w) all |= votes[w];
    return all;
}

// Inclusive prefix sum over the 64 lanes (DPP: rows of 16 lanes, then row broadcasts).
__device__ __forceinline__ int wave_prefix_sum(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
    v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);  // row_bcast:15
    v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);  // row_bcast:31
    return v;
}

}  // namespace dtw
}  // namespace tt
