// Re-tokenisation of the draft tokens into proxy target tokens (Sec. 4.2.1 "Draft Token
// Calculation", Alg. 2 lines S = Tokenizer_d.encode(D), T = Tokenizer_t.decode(S); App. A.1
// string consistency) with a greedy longest-match target tokenizer over byte strings: the
// draft tokens' bytes form S, and from the start of S the longest target token that is a
// prefix of the rest is emitted (the lowest id among tokens with the same bytes).
//
// Target token index (built once per vocabulary): open addressing with linear probing,
// capacity a power of two >= 4 x the token count (load <= 1/4, so a miss probes ~1.4
// slots).  A slot is 16 bytes {first 8 bytes of the token, length, id} and is read with
// one 16-byte load; tokens longer than 8 bytes compare their tail against the table.  The
// slot of a token whose bytes equal those of a lower id is marked dead by a second pass.
// Hash: 32-bit FNV-1a over the token bytes (Fowler, Noll, Vo).  After the slots, a filter of
// 2 bits per slot (one bit set per token, at the top bits of the hash times an odd constant)
// tells a lookup that a byte string is certainly not a token without touching the 16 MB of
// slots: with at most one token per 8 bits about 12% of the non-tokens pass it.
//
// tt_retokenize, one 256-thread workgroup per stream:
//   1. the draft ids' lengths and a block prefix sum give each token's offset in S; the
//      bytes of S are staged into LDS (at most 4096);
//   2. every byte position p computes L(p), the longest target token starting at p: the
//      FNV-1a hashes of all prefixes come from one pass over the bytes; eight candidate
//      lengths at a time (longest first) test the filter, and the first slots of those that
//      pass are loaded together;
//   3. one wave walks p -> p + L(p) from 0 with the L and token values of 64 positions
//      held in its lanes (a readlane per step, the emitted positions kept in a scalar
//      mask), then writes the window's emitted ids to LDS;
//   4. the ids go to a padded per-stream area of the workspace with their count.
// The same index serves the vocabulary intersection of the Token-Level Intersection proposal
// (App. D Alg. 3): a token is in it when it is the lowest id holding its bytes and the other
// vocabulary's index finds those bytes.
// Then the ids are packed into CSR order: up to 2,048 streams one kernel in which every
// workgroup sums the counts before its stream; beyond, one workgroup scans the counts and a
// copy kernel packs.
#include "tt_internal.h"

namespace tt {
namespace {

constexpr uint32_t kFnvBasis = 2166136261u;
constexpr uint32_t kFnvPrime = 16777619u;
constexpr int kThreads = 256;
constexpr int kWave = 64;
constexpr int kBatch = 8;  // candidate lengths probed together
constexpr int kScanThreads = 1024;
constexpr int kFoldStreams = 2048;  // up to this many streams the offsets are summed inside the pack kernel

struct Slot {
    uint64_t key;  // first min(len, 8) bytes, little-endian, zero-padded
    int32_t len;   // token length; -1: dead (a lower id has the same bytes)
    int32_t id;    // -1: empty
};
static_assert(sizeof(Slot) == 16, "one 16-byte load per slot");

__device__ __forceinline__ uint32_t fnv_step(uint32_t h, uint32_t c) { return (h ^ c) * kFnvPrime; }

__device__ __forceinline__ Slot load_slot(const Slot *tab, uint32_t s) {
    const int4 v = *reinterpret_cast<const int4 *>(tab + s);
    Slot e;
    e.key = (uint64_t)(uint32_t)v.x | ((uint64_t)(uint32_t)v.y << 32);
    e.len = v.z;
    e.id = v.w;
    return e;
}

// Filter bit of hash h (fshift = 32 - log2 of the filter's bits): the top bits of h times the
// golden-ratio constant, so they do not repeat the slot index's low bits.
__device__ __forceinline__ uint32_t filter_bit(uint32_t h, int fshift) { return (h * 0x9E3779B1u) >> fshift; }

// bytes of token t equal bytes[0 .. len) beyond the first 8 (the key covers those)
__device__ __forceinline__ bool tail_equal(const tt_vocab &v, int t, const uint8_t *s, int len) {
    const uint8_t *tb = v.bytes + v.offsets[t];
    for (int k = 8; k < len; ++k)
        if (tb[k] != s[k]) return false;
    return true;
}

__global__ void __launch_bounds__(kThreads) index_clear(Slot *tab, uint32_t cap, uint32_t *filter, uint32_t fwords) {
    for (uint32_t s = blockIdx.x * kThreads + threadIdx.x; s < cap; s += gridDim.x * kThreads) {
        tab[s].key = 0;
        tab[s].len = 0;
        tab[s].id = -1;
    }
    for (uint32_t w = blockIdx.x * kThreads + threadIdx.x; w < fwords; w += gridDim.x * kThreads) filter[w] = 0u;
}

// hash, key and length of token t; false if its length is outside [1, max_token_bytes]
__device__ __forceinline__ bool token_sig(const tt_vocab &v, int t, uint32_t &h, uint64_t &key, int &len) {
    const int o = v.offsets[t];
    len = v.offsets[t + 1] - o;
    if (len < 1 || len > v.max_token_bytes) return false;
    h = kFnvBasis;
    key = 0;
    for (int k = 0; k < len; ++k) {
        const uint32_t c = v.bytes[o + k];
        h = fnv_step(h, c);
        if (k < 8) key |= (uint64_t)c << (8 * k);
    }
    return true;
}

__global__ void __launch_bounds__(kThreads) index_insert(tt_vocab v, Slot *tab, uint32_t mask, uint32_t *filter,
                                                         int fshift) {
    const int t = blockIdx.x * kThreads + threadIdx.x;
    if (t >= v.n_tokens) return;
    uint32_t h;
    uint64_t key;
    int len;
    if (!token_sig(v, t, h, key, len)) return;
    const uint32_t f = filter_bit(h, fshift);
    atomicOr(&filter[f >> 5], 1u << (f & 31u));
    uint32_t s = h & mask;
    for (uint32_t probe = 0; probe <= mask; ++probe) {  // at most 1/4 of the slots are taken
        if (atomicCAS(&tab[s].id, -1, t) == -1) {
            tab[s].key = key;
            tab[s].len = len;
            return;
        }
        s = (s + 1) & mask;
    }
}

// A token whose bytes equal those of a lower id marks its own slot dead.  The lowest id of a
// group is never marked and lies on every member's probe chain (linear probing leaves no
// empty slot between a hash's home slot and any entry inserted from it), so the outcome
// does not depend on the order in which members run.
__global__ void __launch_bounds__(kThreads) index_dedup(tt_vocab v, Slot *tab, uint32_t mask) {
    const int t = blockIdx.x * kThreads + threadIdx.x;
    if (t >= v.n_tokens) return;
    uint32_t h;
    uint64_t key;
    int len;
    if (!token_sig(v, t, h, key, len)) return;
    const uint8_t *tb = v.bytes + v.offsets[t];
    uint32_t s = h & mask;
    int own = -1;
    bool dup = false;
    for (uint32_t probe = 0; probe <= mask; ++probe) {
        const int id = tab[s].id;
        if (id < 0) break;
        if (id == t) own = (int)s;
        else if (id < t && tab[s].key == key && __hip_atomic_load(&tab[s].len, __ATOMIC_RELAXED,
                                                                   __HIP_MEMORY_SCOPE_AGENT) == len &&
                 tail_equal(v, id, tb, len))
            dup = true;
        s = (s + 1) & mask;
    }
    if (dup && own >= 0) __hip_atomic_store(&tab[own].len, -1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Block-wide exclusive prefix sum of one int per thread (256 threads); *total gets the sum.
__device__ __forceinline__ int block_exclusive_scan(int v, int *sh_w, int *total) {
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    int x = v;
    for (int d = 1; d < kWave; d <<= 1) {
        const int y = __shfl_up(x, d);
        if (lane >= d) x += y;
    }
    if (lane == kWave - 1) sh_w[wave] = x;
    __syncthreads();
    int before = 0, all = 0;
    for (int w = 0; w < kThreads / kWave; ++w) {
        before += w < wave ? sh_w[w] : 0;
        all += sh_w[w];
    }
    __syncthreads();
    *total = all;
    return before + x - v;
}

struct RetokParams {
    tt_vocab vd, vt;
    const Slot *tab;
    uint32_t mask;
    const uint32_t *filter;
    int32_t fshift;
    int32_t n_streams;
    const int32_t *draft_ids, *draft_off;
    int32_t max_bytes, max_m;
    int32_t *counts, *ids;  // workspace: per-stream count, padded ids [n_streams x max_m]
    int32_t *target_ids, *target_off;
};

__global__ void __launch_bounds__(kThreads) retok_stream(RetokParams p) {
    extern __shared__ int32_t sh[];
    // LDS: pos/out [max_bytes] | src [max_bytes] | tok [max_bytes] | L (u8) | S (u8)
    int32_t *sh_pos = sh;                     // token offsets in S, later the emitted ids
    int32_t *sh_src = sh + p.max_bytes;       // byte offset of each draft token in vd.bytes
    int32_t *sh_tok = sh + 2 * p.max_bytes;   // longest-match token at each position
    uint8_t *sh_L = reinterpret_cast<uint8_t *>(sh + 3 * p.max_bytes);
    uint8_t *sh_S = sh_L + p.max_bytes;
    __shared__ int sh_w[kThreads / kWave];
    __shared__ int sh_bad, sh_m;

    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int d0 = p.draft_off[b];
    const int K = p.draft_off[b + 1] - d0;
    if (tid == 0) sh_bad = (K < 0 || K > p.max_bytes) ? 1 : 0;
    __syncthreads();
    // 1. offsets of the draft tokens in S, then the bytes of S
    int n = 0;
    if (!sh_bad) {
        int carry = 0;
        for (int base = 0; base < K; base += kThreads) {
            const int i = base + tid;
            int len = 0;
            if (i < K) {
                const int id = p.draft_ids[d0 + i];
                if (id < 0 || id >= p.vd.n_tokens) {
                    sh_bad = 1;
                } else {
                    const int o = p.vd.offsets[id];
                    len = p.vd.offsets[id + 1] - o;
                    if (len < 0) sh_bad = 1;
                    sh_src[i] = o;
                }
            }
            int tot;
            const int ex = block_exclusive_scan(len < 0 ? 0 : len, sh_w, &tot);
            if (i < K) sh_pos[i] = carry + ex;
            carry += tot;
            if (carry > p.max_bytes) break;  // uniform: every thread sees the same carry
        }
        n = carry;
    }
    __syncthreads();
    if (n > p.max_bytes) sh_bad = 1;
    __syncthreads();
    if (!sh_bad) {
        for (int x = tid; x < n; x += kThreads) {
            int lo = 0, hi = K - 1;  // last token with pos <= x (zero-length tokens are skipped over)
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (sh_pos[mid] <= x) lo = mid;
                else hi = mid - 1;
            }
            sh_S[x] = p.vd.bytes[sh_src[lo] + (x - sh_pos[lo])];
        }
    }
    __syncthreads();
    // 2. longest target token starting at every position
    if (!sh_bad) {
        const int lmax_v = p.vt.max_token_bytes;
        for (int x = tid; x < n; x += kThreads) {
            const int lmax = lmax_v < n - x ? lmax_v : n - x;
            int best_len = 0, best_tok = 0;
            for (int hi = lmax; hi >= 1 && best_len == 0; hi -= kBatch) {
                const int lo = hi - kBatch + 1;  // candidates lo..hi (lo may be < 1)
                uint32_t h = kFnvBasis;
                uint64_t key = 0;
                const int pre = lo - 1 > 0 ? lo - 1 : 0;
                for (int k = 0; k < pre; ++k) {
                    const uint32_t c = sh_S[x + k];
                    h = fnv_step(h, c);
                    if (k < 8) key |= (uint64_t)c << (8 * k);
                }
                uint32_t hs[kBatch];
                uint64_t ks[kBatch];
#pragma unroll
                for (int k = 0; k < kBatch; ++k) {
                    const int l = lo + k;  // candidate length
                    if (l >= 1) {
                        const uint32_t c = sh_S[x + l - 1];
                        h = fnv_step(h, c);
                        if (l <= 8) key |= (uint64_t)c << (8 * (l - 1));
                    }
                    hs[k] = h;
                    ks[k] = key;
                }
                uint32_t fw[kBatch];
#pragma unroll
                for (int k = 0; k < kBatch; ++k) fw[k] = lo + k >= 1 ? p.filter[filter_bit(hs[k], p.fshift) >> 5] : 0u;
                uint32_t maybe = 0;  // bit k: length lo + k passes the filter
#pragma unroll
                for (int k = 0; k < kBatch; ++k)
                    maybe |= ((fw[k] >> (filter_bit(hs[k], p.fshift) & 31u)) & 1u) << k;
                Slot e[kBatch];
#pragma unroll
                for (int k = 0; k < kBatch; ++k) {
                    e[k].id = -1;
                    if ((maybe >> k) & 1u) e[k] = load_slot(p.tab, hs[k] & p.mask);
                }
#pragma unroll
                for (int k = kBatch - 1; k >= 0; --k) {
                    const int l = lo + k;
                    if (!((maybe >> k) & 1u) || best_len != 0) continue;
                    uint32_t s = hs[k] & p.mask;
                    Slot c = e[k];
                    for (uint32_t probe = 0; probe <= p.mask && c.id >= 0; ++probe) {
                        if (c.len == l && c.key == ks[k] && (l <= 8 || tail_equal(p.vt, c.id, sh_S + x, l))) {
                            best_len = l;
                            best_tok = c.id;
                            break;
                        }
                        s = (s + 1) & p.mask;
                        c = load_slot(p.tab, s);
                    }
                }
            }
            sh_L[x] = (uint8_t)best_len;
            sh_tok[x] = best_tok;
        }
    }
    __syncthreads();
    // 3. the greedy walk, one wave, 64 positions per window held in lanes.  Inside a window the
    // dependent loop is a bound check, a readlane and a mask update: a position where no target
    // token starts sends the walk past the window (a ballot then reports the failure), the
    // emitted positions go to a scalar mask, and their count and ids are formed after it
    if (wave == 0) {
        int pos = 0, m = 0;
        bool fail = sh_bad != 0;
        while (!fail && pos < n) {
            const int p0 = pos, m0 = m;
            const int lim = (n - p0 < kWave ? n - p0 : kWave);  // window length
            const bool inside = lane < lim;
            const int lv = inside ? (int)sh_L[p0 + lane] : 0;
            const int tv = inside ? sh_tok[p0 + lane] : 0;
            const uint64_t dead = __ballot(inside && lv == 0);  // no target token starts here
            const int step = lv == 0 ? kWave : lv;
            uint64_t emitted = 0;  // bit k: a token starts at p0 + k
            int rel = 0;
            while (rel < lim) {
                emitted |= 1ull << rel;
                rel += __builtin_amdgcn_readlane(step, rel);
            }
            m = m0 + __popcll(emitted);
            fail = (emitted & dead) != 0 || m > p.max_m;
            pos = p0 + rel;
            // sh_pos is free again: it takes the output, the k-th emitted position giving id m0 + k
            if ((emitted >> lane) & 1ull) sh_pos[m0 + __popcll(emitted & ((1ull << lane) - 1ull))] = tv;
        }
        if (lane == 0) sh_m = fail ? 0 : m;
    }
    __syncthreads();
    // 4. padded output and count
    const int m = sh_m;
    for (int j = tid; j < m; j += kThreads) p.ids[(int64_t)b * p.max_m + j] = sh_pos[j];
    if (tid == 0) p.counts[b] = m;
}

// CSR offsets from the counts (one workgroup, running total over chunks of 1024 streams).
__global__ void __launch_bounds__(kScanThreads) retok_offsets(RetokParams p) {
    __shared__ int sh_w[kScanThreads / kWave];
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    int carry = 0;
    if (tid == 0) p.target_off[0] = 0;
    for (int base = 0; base < p.n_streams; base += kScanThreads) {
        const int b = base + tid;
        const int v = b < p.n_streams ? p.counts[b] : 0;
        int x = v;
        for (int d = 1; d < kWave; d <<= 1) {
            const int y = __shfl_up(x, d);
            if (lane >= d) x += y;
        }
        if (lane == kWave - 1) sh_w[wave] = x;
        __syncthreads();
        int before = 0, all = 0;
        for (int w = 0; w < kScanThreads / kWave; ++w) {
            before += w < wave ? sh_w[w] : 0;
            all += sh_w[w];
        }
        __syncthreads();
        if (b < p.n_streams) p.target_off[b + 1] = carry + before + x;
        carry += all;
    }
}

__global__ void __launch_bounds__(kThreads) retok_pack(RetokParams p) {
    const int b = blockIdx.x;
    const int o = p.target_off[b];
    const int m = p.target_off[b + 1] - o;
    for (int j = threadIdx.x; j < m; j += kThreads) p.target_ids[o + j] = p.ids[(int64_t)b * p.max_m + j];
}

// For batches up to kFoldStreams: stream b sums the counts before it itself (at most
// kFoldStreams loads per workgroup), writes target_off[b] (and the total) and packs its ids,
// so no separate offsets kernel runs.
__global__ void __launch_bounds__(kThreads) retok_pack_fold(RetokParams p) {
    __shared__ int sh_w[kThreads / kWave];
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    int part = 0;
    for (int c = tid; c < b; c += kThreads) part += p.counts[c];
    for (int d = kWave / 2; d > 0; d >>= 1) part += __shfl_xor(part, d);
    if (lane == 0) sh_w[wave] = part;
    __syncthreads();
    int o = 0;
    for (int w = 0; w < kThreads / kWave; ++w) o += sh_w[w];
    const int m = p.counts[b];
    if (tid == 0) {
        p.target_off[b] = o;
        if (b == p.n_streams - 1) p.target_off[b + 1] = o + m;
    }
    for (int j = tid; j < m; j += kThreads) p.target_ids[o + j] = p.ids[(int64_t)b * p.max_m + j];
}

inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// Id in the index's table of the token with these bytes (the lowest id of several), or -1.
__device__ __forceinline__ int find_token(const Slot *tab, uint32_t mask, const tt_vocab &v, uint32_t h, uint64_t key,
                                          int len, const uint8_t *bytes) {
    uint32_t s = h & mask;
    for (uint32_t probe = 0; probe <= mask; ++probe) {
        const Slot c = load_slot(tab, s);
        if (c.id < 0) return -1;  // dead slots keep their id, so a chain never ends early
        if (c.len == len && c.key == key && (len <= 8 || tail_equal(v, c.id, bytes, len))) return c.id;
        s = (s + 1) & mask;
    }
    return -1;
}

// Vocabulary intersection (App. D Alg. 3), one thread per token t of vocabulary A: out[t] is
// the id in B of t's bytes when t is the lowest id in A holding them, else -1.
__global__ void __launch_bounds__(kThreads) vocab_isect(tt_vocab va, const Slot *ta, uint32_t ma, tt_vocab vb,
                                                        const Slot *tb, uint32_t mb, int32_t *out) {
    const int t = blockIdx.x * kThreads + threadIdx.x;
    if (t >= va.n_tokens) return;
    uint32_t h;
    uint64_t key;
    int len;
    int res = -1;
    if (token_sig(va, t, h, key, len)) {
        const uint8_t *bytes = va.bytes + va.offsets[t];
        if (find_token(ta, ma, va, h, key, len, bytes) == t) res = find_token(tb, mb, vb, h, key, len, bytes);
    }
    out[t] = res;
}

}  // namespace

uint32_t token_index_capacity(int32_t n_tokens) {
    uint32_t cap = 64;
    while (cap < 4u * (uint32_t)n_tokens) cap <<= 1;
    return cap;
}

// The filter: 2 bits per slot, in 32-bit words after the slots.
static uint32_t token_filter_words(uint32_t cap) { return cap / 16u; }

static int token_filter_shift(uint32_t cap) {
    int lg = 0;
    while ((1u << lg) < cap) ++lg;
    return 32 - (lg + 1);
}

size_t token_index_bytes(int32_t n_tokens) {
    const uint32_t cap = token_index_capacity(n_tokens);
    return sizeof(Slot) * (size_t)cap + 4 * (size_t)token_filter_words(cap);
}

int launch_token_index_build(const tt_vocab &v, void *index, hipStream_t stream) {
    const uint32_t cap = token_index_capacity(v.n_tokens);
    Slot *tab = static_cast<Slot *>(index);
    uint32_t *filter = reinterpret_cast<uint32_t *>(tab + cap);
    hipLaunchKernelGGL(index_clear, dim3((cap + kThreads - 1) / kThreads < 2048 ? (cap + kThreads - 1) / kThreads : 2048),
                       dim3(kThreads), 0, stream, tab, cap, filter, token_filter_words(cap));
    if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
    const dim3 grid((v.n_tokens + kThreads - 1) / kThreads);
    hipLaunchKernelGGL(index_insert, grid, dim3(kThreads), 0, stream, v, tab, cap - 1, filter, token_filter_shift(cap));
    if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
    hipLaunchKernelGGL(index_dedup, grid, dim3(kThreads), 0, stream, v, tab, cap - 1);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

int launch_vocab_intersection(const tt_vocab &vd, const void *vd_index, const tt_vocab &vt, const void *vt_index,
                              int32_t *d2t, int32_t *t2d, hipStream_t stream) {
    const Slot *td = static_cast<const Slot *>(vd_index);
    const Slot *tt_ = static_cast<const Slot *>(vt_index);
    const uint32_t md = token_index_capacity(vd.n_tokens) - 1, mt = token_index_capacity(vt.n_tokens) - 1;
    hipLaunchKernelGGL(vocab_isect, dim3((vd.n_tokens + kThreads - 1) / kThreads), dim3(kThreads), 0, stream, vd, td,
                       md, vt, tt_, mt, d2t);
    if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
    hipLaunchKernelGGL(vocab_isect, dim3((vt.n_tokens + kThreads - 1) / kThreads), dim3(kThreads), 0, stream, vt, tt_,
                       mt, vd, td, md, t2d);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

size_t retok_workspace_bytes(int32_t n_streams, int32_t max_m) {
    return align256(4 * (size_t)n_streams) + 4 * (size_t)n_streams * (size_t)max_m;
}

size_t retok_lds_bytes(int32_t max_bytes) { return 14 * (size_t)max_bytes; }

int launch_retokenize(const RetokArgs &a, hipStream_t stream) {
    RetokParams p;
    p.vd = a.vd;
    p.vt = a.vt;
    p.tab = static_cast<const Slot *>(a.index);
    p.mask = token_index_capacity(a.vt.n_tokens) - 1;
    p.filter = reinterpret_cast<const uint32_t *>(p.tab + p.mask + 1);
    p.fshift = token_filter_shift(p.mask + 1);
    p.n_streams = a.n_streams;
    p.draft_ids = a.draft_ids;
    p.draft_off = a.draft_off;
    p.max_bytes = a.max_bytes;
    p.max_m = a.max_m;
    uint8_t *ws = static_cast<uint8_t *>(a.workspace);
    p.counts = reinterpret_cast<int32_t *>(ws);
    p.ids = reinterpret_cast<int32_t *>(ws + align256(4 * (size_t)a.n_streams));
    p.target_ids = a.target_ids;
    p.target_off = a.target_off;
    if (a.n_streams > 0) {
        hipLaunchKernelGGL(retok_stream, dim3(a.n_streams), dim3(kThreads), retok_lds_bytes(a.max_bytes), stream, p);
        if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
    }
    if (a.n_streams > 0 && a.n_streams <= kFoldStreams) {
        hipLaunchKernelGGL(retok_pack_fold, dim3(a.n_streams), dim3(kThreads), 0, stream, p);
        return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
    }
    hipLaunchKernelGGL(retok_offsets, dim3(1), dim3(kScanThreads), 0, stream, p);  // target_off[0] = 0 at least
    if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
    if (a.n_streams == 0) return TT_OK;
    hipLaunchKernelGGL(retok_pack, dim3(a.n_streams), dim3(kThreads), 0, stream, p);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

}  // namespace tt
