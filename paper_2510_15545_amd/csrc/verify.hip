// Vocabulary-wide lossless speculative sampling on gfx950.
//
// Per stream b (Sec. 3 "Standard Speculative Sampling", Sec. 4.2.2-4.2.3, App. D Alg. 4):
//   gamma  = number of leading proposals with u_j < P_t(t_j) / q_j (fp32), first rejection stops
//   r      = gamma; R(x) = max(0, P_t[r](x) - q_r [x == t_r]) if r < M, else P_t[M](x)
//   token  = inverse-CDF sample of R with the uniform u_sample[b]
//
// The row of stream b is read once from HBM.  It is cut into chunks of 1024 floats
// (one wave, 16 floats per lane, 16-byte loads).  Each chunk's residual mass is
// accumulated in exact Q62 fixed point (R quantised by truncation), so chunk sums and
// their prefix are independent of summation order and the sampled token is
// bit-identical to a sequential scan.  Sampling forms Z and T = floor(u * Z) exactly,
// scans the chunk sums to the crossing chunk, re-reads that one chunk (4 KiB) and
// scans it to the crossing index.  Row loads carry the non-temporal hint: every row
// is read once, and for 256 rows of 151,936 floats that cut the kernel from 34.6 to
// 30.6 us against ordinary loads.
//
// Two launch shapes:
//   row path    (at least one stream per CU): one workgroup per stream runs the
//               acceptance scan once, streams its whole row (about eight chunks per
//               wave: 64 to 1024 threads), keeps the chunk sums in LDS and one wave
//               samples.  One kernel.
//   split path  (fewer streams): verify_stream over B x S workgroups (every workgroup
//               of a stream recomputes gamma, streams its share of the row and stores
//               chunk sums), then verify_sample with one wave per stream.  The kernel
//               boundary publishes the chunk sums: an in-kernel hand-off between
//               workgroups needs an agent-scope release, which on gfx950 writes back
//               the XCD's whole L2 (one per workgroup made the kernel 5-10x slower).
// Sampling runs in one wave with DPP prefix sums and no LDS or barriers.
// In the split path workgroup id -> (stream, split) is XCD-aware: the hardware deals
// workgroup ids round-robin over the 8 XCDs, so XCD x receives the contiguous work range
// [x * G/8, (x+1) * G/8) and a stream's splits share one XCD.
#include "stamps.h"
#include "verify_core.h"

#ifndef TT_VERIFY_TARGET_WG
#define TT_VERIFY_TARGET_WG 2048  // split path: workgroups to aim for
#endif
#ifndef TT_VERIFY_ROW_MIN_STREAMS
#define TT_VERIFY_ROW_MIN_STREAMS 256  // row path from this many streams up
#endif

TT_STAMPS_TABLE(verify)

namespace tt {
namespace {

using namespace vcore;

constexpr int kSplitThreads = 256;
constexpr int kRowThreads = 1024;
constexpr int kXcds = 8;
constexpr int kRowMaxChunks = 2048;  // row path: rows up to 2M floats (LDS holds their chunk sums)

struct VParams {
    VerifyArgs a;
    uint64_t *zsum;
    int32_t *rsel;
    uint64_t *partials;
    int32_t nc, splits, cpw, work_items, vec4;
};

// Acceptance scan by one wave: gamma (first rejection, else M) and the rejected
// position's t, q and P_t(t) (rtok = -1 after full acceptance); false if the stream is invalid (M
// outside [0, max_m] or an id outside [0, v_t)).  The proposal's mass at t_j is q_j
// (one-hot) or q_rows[t0 + j][t_j] (DENSE).  t_j, q_j and u_j are loaded together; only
// P_t(t_j) (and the dense q(t_j)) wait for t_j.
struct Rejection {
    int rtok;  // t_gamma (-1 after full acceptance)
    float rq;  // one-hot q_gamma
    float rp;  // P_t(t_gamma)
};

template <bool DENSE>
__device__ __forceinline__ bool accept_scan(const VerifyArgs &a, int b, int t0, int M, int lane, int &gamma,
                                            Rejection &rj) {
    gamma = M;
    rj = Rejection{-1, 0.0f, 0.0f};
    if (M < 0 || M > a.max_m) return false;
    for (int base = 0; base < M; base += kWave) {
        const int j = base + lane;
        bool bad = false, rej = false;
        float pt = 0.0f, q1 = 0.0f;
        int tok = -1;
        if (j < M) {
            tok = a.target_ids[t0 + j];
            q1 = DENSE ? 0.0f : a.q[t0 + j];
            const float uj = a.u_accept[t0 + j];
            bad = tok < 0 || tok >= a.v_t;
            if (!bad) {
                pt = a.target_probs[(int64_t)(t0 + b + j) * a.target_ld + tok];
                const float qj = DENSE ? a.q_rows[(int64_t)(t0 + j) * a.q_ld + tok] : q1;
                const float ratio = pt / qj;
                rej = !((qj <= 0.0f) || (uj < ratio));
            }
        }
        if (__any(bad)) return false;
        const unsigned long long rm = __ballot(rej);
        if (rm != 0ull && gamma == M) {
            const int l = __ffsll(rm) - 1;
            gamma = base + l;
            rj.rtok = __shfl(tok, l);
            rj.rq = __shfl(q1, l);
            rj.rp = __shfl(pt, l);
        }
    }
    return true;
}

// The proposal taken off row r: the dense draft row (DENSE, r < M), else the one-hot
// mass rq at token rtok (rtok = -1 after full acceptance: the bonus row is sampled as is).
struct Proposal {
    const float *qrow;
    int rtok;
    float rq;
};

template <bool DENSE>
__device__ __forceinline__ Proposal proposal(const VerifyArgs &a, int t0, int M, int r) {
    Proposal pr{nullptr, -1, 0.0f};
    if (r < M) {
        if (DENSE) pr.qrow = a.q_rows + (int64_t)(t0 + r) * a.q_ld;
        else {
            pr.rtok = a.target_ids[t0 + r];
            pr.rq = a.q[t0 + r];
        }
    }
    return pr;
}

// Q62 chunk sums of row's chunks [c0, c1) by the calling workgroup's waves; rp is the
// row's entry at the one-hot proposal's token (from the acceptance scan), next the LDS chunk
// counter (or null).
template <class Store>
__device__ __forceinline__ void stream_row(const float *row, const Proposal &pr, int vt, bool vec, int c0, int c1,
                                           int stride, float rp, Store store, int *next) {
    if (pr.qrow != nullptr) stream_chunks_dense(row, pr.qrow, vt, vec, c0, c1, stride, store, next);
    else stream_chunks(row, vt, vec, c0, c1, stride, pr.rtok, pr.rq, rp, store, next);
}

// ------------------------------------------------------------------ row path
template <bool DENSE, int THREADS>
__global__ void __launch_bounds__(THREADS) verify_row(VParams p) {
    constexpr int kWaves = THREADS / kWave;
    const VerifyArgs &a = p.a;
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);  // uniform: wave-level branches stay scalar
    extern __shared__ uint64_t sh_part[];  // nc chunk sums
    __shared__ int sh_gamma, sh_ok, sh_next;
    __shared__ Rejection sh_rj;

    TT_STAMP(0);
    const int t0 = a.target_off[b];
    const int M = a.target_off[b + 1] - t0;
    const float us = a.u_sample[b];
    if (wave == 0) {
        int gamma;
        Rejection rj;
        const bool ok = accept_scan<DENSE>(a, b, t0, M, lane, gamma, rj);
        if (lane == 0) {
            sh_gamma = gamma;
            sh_ok = ok ? 1 : 0;
            sh_rj = rj;
            sh_next = kWaves;
        }
        TT_STAMP(1);
    }
    __syncthreads();
    TT_STAMP(2);
    if (!sh_ok) {
        if (tid == 0) {
            a.n_accepted[b] = -1;
            a.out_token[b] = -1;
            p.rsel[b] = -1;
        }
        return;
    }
    const int r = sh_gamma;
    const Rejection rj = sh_rj;
    const int vt = a.v_t;
    const bool vec = p.vec4 != 0;
    const float *row = a.target_probs + (int64_t)(t0 + b + r) * a.target_ld;
    const Proposal pr{DENSE && r < M ? a.q_rows + (int64_t)(t0 + r) * a.q_ld : nullptr, rj.rtok, rj.rq};
    stream_row(row, pr, vt, vec, 0, p.nc, kWaves, rj.rp, [&](int c, uint64_t s) { sh_part[c] = s; }, &sh_next);
    TT_STAMP(3);
    __syncthreads();
    TT_STAMP(4);
    if (wave != 0) return;
    uint64_t Z;
    const int token =
        wave_sample(row, pr.qrow, vt, p.nc, vec, [&](int c) { return sh_part[c]; }, us, pr.rtok, pr.rq, &Z);
    if (tid == 0) {
        a.n_accepted[b] = r;
        a.out_token[b] = token;
        p.zsum[b] = Z;
        p.rsel[b] = r;
    }
    TT_STAMP(5);
}

// ------------------------------------------------------------------ split path
// GIVEN: gamma was found by an earlier kernel of the same call (the fused step's front) and
// is read from rsel (-1: a sentinel stream whose outputs are already written).
template <bool DENSE, bool GIVEN>
__global__ void __launch_bounds__(kSplitThreads) verify_stream(VParams p) {
    const VerifyArgs &a = p.a;
    const int G = gridDim.x;
    const int g = blockIdx.x;
    const int work = (g % kXcds) * (G / kXcds) + g / kXcds;
    if (work >= p.work_items) return;
    const int b = work / p.splits, s = work % p.splits;
    const int tid = threadIdx.x, lane = tid % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);  // uniform: wave-level branches stay scalar
    __shared__ int sh_gamma, sh_ok, sh_next;
    __shared__ float sh_rp;

    const int t0 = a.target_off[b];
    const int M = a.target_off[b + 1] - t0;
    const int c0 = s * p.cpw;
    const int c1 = (c0 + p.cpw) < p.nc ? (c0 + p.cpw) : p.nc;
    if (tid == 0) sh_next = c0 + kSplitThreads / kWave;
    if (GIVEN) {
        const int r = p.rsel[b];
        if (tid == 0) {
            sh_gamma = r;
            sh_ok = r >= 0 ? 1 : 0;
            // the rejected proposal's entry, if this workgroup's share of the row holds it
            const int rtok = r >= 0 && r < M ? a.target_ids[t0 + r] : -1;
            const int x0 = s * p.cpw * kChunk;
            sh_rp = rtok >= x0 && rtok < x0 + p.cpw * kChunk && rtok < a.v_t
                        ? a.target_probs[(int64_t)(t0 + b + r) * a.target_ld + rtok]
                        : 0.0f;
        }
    } else if (wave == 0) {  // every workgroup of the stream recomputes gamma
        int gamma;
        Rejection rj;
        const bool ok = accept_scan<DENSE>(a, b, t0, M, lane, gamma, rj);
        if (lane == 0) {
            sh_gamma = gamma;
            sh_ok = ok ? 1 : 0;
            sh_rp = rj.rp;
        }
    }
    __syncthreads();
    if (!sh_ok) {
        if (!GIVEN && s == 0 && tid == 0) {
            a.n_accepted[b] = -1;
            a.out_token[b] = -1;
            p.rsel[b] = -1;
        }
        return;
    }
    const int r = sh_gamma;
    if (!GIVEN && s == 0 && tid == 0) p.rsel[b] = r;
    const float *row = a.target_probs + (int64_t)(t0 + b + r) * a.target_ld;
    const Proposal pr = proposal<DENSE>(a, t0, M, r);
    uint64_t *out = p.partials + (int64_t)b * p.nc;
    stream_row(row, pr, a.v_t, p.vec4 != 0, c0, c1, kSplitThreads / kWave, sh_rp,
               [&](int c, uint64_t sum) { out[c] = sum; }, &sh_next);
}

// One wave per stream: exact threshold, crossing chunk, crossing index.
template <bool DENSE>
__global__ void __launch_bounds__(kWave) verify_sample(VParams p) {
    const VerifyArgs &a = p.a;
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const uint64_t *part = p.partials + (int64_t)b * p.nc;
    const int r = p.rsel[b];
    const int t0 = a.target_off[b];
    const int M = a.target_off[b + 1] - t0;
    const float us = a.u_sample[b];
    if (r < 0) return;  // sentinel stream, outputs already written (uniform per workgroup)
    const float *row = a.target_probs + (int64_t)(t0 + b + r) * a.target_ld;
    const Proposal pr = proposal<DENSE>(a, t0, M, r);
    uint64_t Z;
    const int token =
        wave_sample(row, pr.qrow, a.v_t, p.nc, p.vec4 != 0, [&](int c) { return part[c]; }, us, pr.rtok, pr.rq, &Z);
    if (tid == 0) {
        a.n_accepted[b] = r;
        a.out_token[b] = token;
        p.zsum[b] = Z;
    }
}

// Optional normalised residual row: res[x] = R(x) / fp32(Z * 2^-62), one-hot when Z = 0.
template <bool DENSE>
__global__ void __launch_bounds__(kSplitThreads) residual_write(VParams p, int rsplit) {
    const VerifyArgs &a = p.a;
    const int b = blockIdx.x / rsplit, sidx = blockIdx.x % rsplit;
    if (a.n_accepted[b] < 0) return;
    const int r = p.rsel[b];
    const uint64_t Z = p.zsum[b];
    const int tok = a.out_token[b];
    const int t0 = a.target_off[b];
    const int M = a.target_off[b + 1] - t0;
    const float *row = a.target_probs + (int64_t)(t0 + b + r) * a.target_ld;
    const Proposal pr = proposal<DENSE>(a, t0, M, r);
    float *res = a.residual + (int64_t)b * a.target_ld;
    const int vt = a.v_t;
    const int per = (vt + rsplit - 1) / rsplit;
    const int x0 = sidx * per;
    const int x1 = (x0 + per) < vt ? (x0 + per) : vt;
    if (Z == 0) {
        for (int x = x0 + (int)threadIdx.x; x < x1; x += kSplitThreads) res[x] = (x == tok) ? 1.0f : 0.0f;
        return;
    }
    const float zf = (float)Z * 0x1p-62f;
    for (int x = x0 + (int)threadIdx.x; x < x1; x += kSplitThreads)
        res[x] = clamp01(row[x] - (pr.qrow != nullptr ? pr.qrow[x] : (x == pr.rtok ? pr.rq : 0.0f))) / zf;
}

inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

}  // namespace

VerifyLayout verify_layout(int32_t n_streams, int32_t v_t) {
    VerifyLayout L;
    const size_t n = n_streams > 0 ? (size_t)n_streams : 0;
    L.n_chunks = v_t > 0 ? (int32_t)((v_t + kChunk - 1) / kChunk) : 0;
    size_t off = 0;
    L.zsum = off;
    off = align256(off + 8 * n);
    L.rsel = off;
    off = align256(off + 4 * n);
    L.partials = off;
    off = align256(off + 8 * n * (size_t)L.n_chunks);
    L.total = off;
    return L;
}

bool verify_row_path(int32_t n_streams, int32_t v_t) {
    const VerifyLayout L = verify_layout(n_streams, v_t);
    return n_streams >= TT_VERIFY_ROW_MIN_STREAMS && L.n_chunks <= kRowMaxChunks;
}

namespace {

VParams make_params(const VerifyArgs &a) {
    const VerifyLayout L = verify_layout(a.n_streams, a.v_t);
    uint8_t *ws = static_cast<uint8_t *>(a.workspace);
    VParams p;
    p.a = a;
    p.zsum = reinterpret_cast<uint64_t *>(ws + L.zsum);
    p.rsel = reinterpret_cast<int32_t *>(ws + L.rsel);
    p.partials = reinterpret_cast<uint64_t *>(ws + L.partials);
    p.nc = L.n_chunks;
    p.vec4 = ((reinterpret_cast<uintptr_t>(a.target_probs) & 15u) == 0 && (a.target_ld % 4) == 0) ? 1 : 0;
    if (a.q_rows != nullptr && ((reinterpret_cast<uintptr_t>(a.q_rows) & 15u) != 0 || (a.q_ld % 4) != 0)) p.vec4 = 0;
    p.splits = 1;
    p.cpw = p.nc;
    p.work_items = a.n_streams;
    return p;
}

int launch_residual(const VParams &p, hipStream_t stream) {
    int rsplit = (p.a.v_t + 8191) / 8192;
    if (rsplit < 1) rsplit = 1;
    if (p.a.q_rows != nullptr)
        hipLaunchKernelGGL(residual_write<true>, dim3(p.a.n_streams * rsplit), dim3(kSplitThreads), 0, stream, p,
                           rsplit);
    else
        hipLaunchKernelGGL(residual_write<false>, dim3(p.a.n_streams * rsplit), dim3(kSplitThreads), 0, stream, p,
                           rsplit);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

// Split path: the streaming kernel over B x S workgroups, then one sampling wave per stream.
template <bool DENSE, bool GIVEN>
int launch_split(VParams &p, hipStream_t stream) {
    const VerifyArgs &a = p.a;
    // splits per stream: aim for TT_VERIFY_TARGET_WG workgroups, at least one chunk per wave
    constexpr int kWaves = kSplitThreads / kWave;
    int max_splits = (p.nc + kWaves - 1) / kWaves;
    int splits = (TT_VERIFY_TARGET_WG + a.n_streams - 1) / a.n_streams;
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    p.cpw = (p.nc + splits - 1) / splits;
    p.splits = (p.nc + p.cpw - 1) / p.cpw;
    p.work_items = a.n_streams * p.splits;
    const int grid = ((p.work_items + kXcds - 1) / kXcds) * kXcds;
    hipLaunchKernelGGL((verify_stream<DENSE, GIVEN>), dim3(grid), dim3(kSplitThreads), 0, stream, p);
    if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
    hipLaunchKernelGGL(verify_sample<DENSE>, dim3(a.n_streams), dim3(kWave), 0, stream, p);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

// One workgroup of THREADS per stream.  The chunk sums in dynamic LDS can pass the 64 KiB a
// launch gets by default; the kernel is then allowed the size it asks for.
template <bool DENSE, int THREADS>
int launch_row(const VParams &p, hipStream_t stream) {
    const size_t lds = 8 * (size_t)p.nc;
    if (lds > 64 * 1024 &&
        hipFuncSetAttribute(reinterpret_cast<const void *>(&verify_row<DENSE, THREADS>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
        return TT_ELAUNCH;
    hipLaunchKernelGGL((verify_row<DENSE, THREADS>), dim3(p.a.n_streams), dim3(THREADS), lds, stream, p);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

template <bool DENSE>
int launch_verify_kernels(VParams &p, hipStream_t stream) {
    const VerifyArgs &a = p.a;
    if (verify_row_path(a.n_streams, a.v_t)) {
        // about eight chunks per wave: short rows take small workgroups, so that several
        // streams share a compute unit and their acceptance scans and samples overlap
        const int waves = (p.nc + 7) / 8;
        if (waves <= 1) return launch_row<DENSE, 64>(p, stream);
        if (waves <= 2) return launch_row<DENSE, 128>(p, stream);
        if (waves <= 4) return launch_row<DENSE, 256>(p, stream);
        if (waves <= 8) return launch_row<DENSE, 512>(p, stream);
        return launch_row<DENSE, kRowThreads>(p, stream);
    }
    return launch_split<DENSE, false>(p, stream);
}

}  // namespace

int launch_verify_residual(const VerifyArgs &a, hipStream_t stream) {
    if (a.workspace == nullptr || a.workspace_bytes < verify_layout(a.n_streams, a.v_t).total) return TT_EWORKSPACE;
    return launch_residual(make_params(a), stream);
}


int launch_verify_after_gamma(const VerifyArgs &a, hipStream_t stream) {
    if (a.workspace == nullptr || a.workspace_bytes < verify_layout(a.n_streams, a.v_t).total) return TT_EWORKSPACE;
    VParams p = make_params(a);
    const int st = launch_split<false, true>(p, stream);
    if (st != TT_OK) return st;
    return a.residual != nullptr ? launch_residual(p, stream) : TT_OK;
}

int launch_verify(const VerifyArgs &a, hipStream_t stream) {
    if (a.workspace == nullptr || a.workspace_bytes < verify_layout(a.n_streams, a.v_t).total) return TT_EWORKSPACE;
    VParams p = make_params(a);
    const int st = a.q_rows != nullptr ? launch_verify_kernels<true>(p, stream) : launch_verify_kernels<false>(p, stream);
    if (st != TT_OK) return st;
    return a.residual != nullptr ? launch_residual(p, stream) : TT_OK;
}

}  // namespace tt
