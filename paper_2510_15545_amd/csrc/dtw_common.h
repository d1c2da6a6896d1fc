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

// Bit k set where byte k of the packed pattern xw equals the byte broadcast in bc.  Equal
// bytes are found exactly by SWAR (0x80 in each byte of w ^ bc that is zero); v_dot4 then
// gathers the four flags of a dword into four mask bits (byte weights 1, 2, 4, 8 times 0x80).
template <int TB>
__device__ __forceinline__ typename MaskType<TB>::type match_mask(const uint32_t (&xw)[TB / 4], uint32_t bc) {
    using M = typename MaskType<TB>::type;
    M eq = 0;
#pragma unroll
    for (int p = 0; p < TB / 8; ++p) {
        uint32_t acc = 0;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const uint32_t t = xw[2 * p + h] ^ bc;
            const uint32_t z = ~(((t & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | t) & 0x80808080u;
            acc = __builtin_amdgcn_udot4(z, h ? 0x80402010u : 0x08040201u, acc, false);
        }
        eq |= M(acc >> 7) << (8 * p);
    }
    return eq;
}

__device__ __forceinline__ int popcount(uint32_t v) { return __popc(v); }
__device__ __forceinline__ int popcount(uint64_t v) { return __popcll(v); }

// Edit distance between the packed pattern xw (m bytes) and the text bytes in yw (n bytes):
// Myers' bit-parallel recurrence over the text with the top row D(0, j) = j.  The distance
// is read at the end from the last column's vertical deltas: D(m, n) = n + #(+1) - #(-1).
template <int TB>
__device__ __forceinline__ int bitparallel_distance(const uint32_t (&xw)[TB / 4], int m,
                                                    const uint32_t (&yw)[TB / 4], int n) {
    using M = typename MaskType<TB>::type;
    if (m == 0) return n;
    const M lim = (m >= (int)(8 * sizeof(M))) ? ~M(0) : ((M(1) << m) - 1);
    M vp = ~M(0), vn = 0;
#pragma unroll
    for (int k = 0; k < TB; ++k) {
        if (k < n) {
            const uint32_t bc = __builtin_amdgcn_perm(0u, yw[k >> 2], (uint32_t)(k & 3) * 0x01010101u);
            const M eq = match_mask<TB>(xw, bc) & lim;
            const M xv = eq | vn;
            const M xh = (((eq & vp) + vp) ^ vp) | eq;
            M hp = vn | ~(xh | vp);
            M hn = vp & xh;
            hp = (hp << 1) | M(1);
            hn = hn << 1;
            vp = hn | ~(xv | hp);
            vn = hp & xv;
        }
    }
    return n + popcount(vp & lim) - popcount(vn & lim);
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
