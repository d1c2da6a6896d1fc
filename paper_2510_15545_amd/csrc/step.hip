// The whole verification path of one decode step in one launch: Dynamic Token Warping
// (Sec. 4.1, Alg. 1, App. H), the mapping and probability transfer (Alg. 2, App. A.2),
// the acceptance scan and the vocabulary-wide sample (Sec. 3, Sec. 4.2.2-4.2.3, App. D
// Alg. 4).  One 1024-thread workgroup per stream; results are identical to tt_align,
// tt_transfer and tt_verify called in sequence.
//
//   1. All threads: the pair's tokens are staged into LDS (four waves) while other threads
//      prefetch what does not depend on the alignment: the draft probability of every
//      emitted draft token P_d(d_i), and P_t(t_j), u_j and t_j for every proxy position.
//   2. All threads: token distances of the band cells.
//   3. Wave 0: row-scan DTW, backtrack, path and map (dtw_rows.h); q_j = P_d(d_{i*(j)})
//      is a lookup in the prefetched values; the acceptance ballot gives gamma.
//   4. All waves stream the row gamma once (Q62 chunk sums into LDS); wave 0 samples.
//
// Compared with three launches this removes two kernel boundaries and the global round
// trips of map and q, and every global load of steps 1-3 is issued at the start.
#include "dtw_rows.h"
#include "stamps.h"
#include "verify_core.h"

TT_STAMPS_TABLE(step)

namespace tt {
namespace {

using vcore::kChunk;
using vcore::kWave;

constexpr int kThreads = 1024;
constexpr int kStageThreads = 256;                // waves 0-3 stage tokens
constexpr int kDraftPrefetch = 256;               // threads 256..319 gather P_d(d_i)
constexpr int kTargetPrefetch = 320;              // threads 320..383 gather P_t(t_j), u_j, t_j
// dynamic LDS of the streaming part (chunk sums): at most what gfx950's 160 KiB per workgroup
// leaves beside the largest static use (40 KiB at 32-byte token slots)
constexpr size_t kDynLdsMax = 160 * 1024 - 40 * 1024;

struct SParams {
    StepArgs s;
    uint64_t *zsum;
    int32_t *rsel;
    int32_t nc, vec4;
};

// STREAM = false: the kernel stops once gamma is known and leaves it in rsel for the split
// verification kernels (batches of long rows too small to fill the chip one stream per CU).
template <int TB, bool STREAM>
__global__ void __launch_bounds__(kThreads) step_fused(SParams p) {
    const AlignArgs &al = p.s.al;
    const TransferArgs &tr = p.s.tr;
    const VerifyArgs &ve = p.s.ve;
    __shared__ rows::Lds<TB> s;
    __shared__ float pd[rows::kMaxSide];   // P_d of the emitted draft tokens
    __shared__ float pt[rows::kMaxSide];   // P_t(t_j) on target row j
    __shared__ float ua[rows::kMaxSide];   // acceptance uniforms
    __shared__ int tid_t[rows::kMaxSide];  // target ids
    __shared__ int sh_votes[kThreads / kWave];
    __shared__ int sh_gamma, sh_ok, sh_rtok, sh_next;
    __shared__ float sh_rq, sh_rp;
    extern __shared__ uint64_t sh_part[];  // Q62 chunk sums of the selected row

    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);  // uniform: wave-level branches stay scalar
    TT_STAMP(0);
    const int d0 = al.draft_off[b], K = al.draft_off[b + 1] - d0;
    const int t0 = al.target_off[b], M = al.target_off[b + 1] - t0;
    const float us = ve.u_sample[b];  // needed only by the sampler, loaded while the rest runs


    // ---- 1. staging and prefetch
    const bool shape_ok = K >= 1 && K <= al.max_k && M >= 1 && M <= al.max_m;
    const bool vshape_ok = M >= 0 && M <= ve.max_m;  // max_m <= 64 here
    int bad = shape_ok ? 0 : 1, vbad = vshape_ok ? 0 : 1;
    if (shape_ok && tid < kStageThreads) bad = rows::stage<TB>(al, s, d0, K, t0, M, tid, kStageThreads);
    // the probability gathers stay in registers until just before step 3, so the barriers
    // of step 2 do not wait for them
    const bool pd_thread = shape_ok && tid >= kDraftPrefetch && tid < kDraftPrefetch + K;
    const bool pt_thread = vshape_ok && tid >= kTargetPrefetch && tid < kTargetPrefetch + M;
    float pv = __builtin_nanf(""), uv = 0.0f;
    int tok = 0;
    if (pd_thread) {
        const int i = tid - kDraftPrefetch;
        const int id = al.draft_ids[d0 + i];
        if (id >= 0 && id < tr.v_d) pv = tr.draft_probs[(int64_t)(d0 + i) * tr.draft_ld + id];
    }
    if (pt_thread) {
        const int j = tid - kTargetPrefetch;
        tok = al.target_ids[t0 + j];
        if (tok < 0 || tok >= ve.v_t) {
            vbad = 1;
        } else {
            pv = ve.target_probs[(int64_t)(t0 + b + j) * ve.target_ld + tok];
            uv = ve.u_accept[t0 + j];
        }
    }
    const int all_votes = dtw::block_or((bad ? 1 : 0) | (vbad ? 2 : 0), sh_votes, kThreads / kWave);
    const bool align_ok = (all_votes & 1) == 0;
    const bool verify_ok = (all_votes & 2) == 0;
    TT_STAMP(1);

    // ---- 2. token distances, cumulative cost, move masks
    const int L = rows::band_half_width(K, M, al.w);
    int total = 0;
    if (align_ok) {  // uniform over the workgroup
        rows::init_border<TB>(s, tid, kThreads);
        rows::costs<TB>(s, K, M, L, tid, kThreads);
        __syncthreads();
        if (wave == 0) total = rows::recurrence<TB>(s, K, M, L);
        __syncthreads();
        TT_STAMP(2);
        rows::moves<TB>(s, K, M, L, wave, kThreads / kWave);
    }
    if (pd_thread) pd[tid - kDraftPrefetch] = pv;
    if (pt_thread) {
        tid_t[tid - kTargetPrefetch] = tok;
        pt[tid - kTargetPrefetch] = pv;
        ua[tid - kTargetPrefetch] = uv;
    }
    __syncthreads();

    // ---- 3. backtrack, transfer and acceptance (one wave)
    if (wave == 0) {
        float qj = __builtin_nanf("");  // q of position lane (lanes < M)
        if (align_ok) {
            const int mi = rows::backtrack<TB>(al, s, b, d0, K, t0, M, total);
            if (mi >= 0 && mi < K) qj = pd[mi];
        } else {
            if (lane == 0) {
                al.cost[b] = -1;
                al.path_len[b] = 0;
            }
            for (int j = lane; j < M; j += kWave) al.map[t0 + j] = -1;
        }
        for (int j = lane; j < M; j += kWave) tr.q[t0 + j] = j < rows::kMaxSide ? qj : __builtin_nanf("");
        if (verify_ok) {
            const bool rej = lane < M && !((qj <= 0.0f) || (ua[lane] < pt[lane] / qj));
            const unsigned long long rm = __ballot(rej);
            const int gamma = rm ? __ffsll(rm) - 1 : M;
            const float rq = __shfl(qj, gamma < M ? gamma : 0);
            if (lane == 0) {
                sh_gamma = gamma;
                sh_rtok = gamma < M ? tid_t[gamma] : -1;
                sh_rq = gamma < M ? rq : 0.0f;
                sh_rp = gamma < M ? pt[gamma] : 0.0f;  // the row's entry at t_gamma, already gathered
                sh_next = kThreads / kWave;
            }
        }
        if (lane == 0) sh_ok = verify_ok ? 1 : 0;
    }
    __syncthreads();
    TT_STAMP(3);
    if (!sh_ok) {
        if (tid == 0) {
            ve.n_accepted[b] = -1;
            ve.out_token[b] = -1;
            p.rsel[b] = -1;
        }
        return;
    }

    if (!STREAM) {
        if (tid == 0) p.rsel[b] = sh_gamma;
        return;
    }

    // ---- 4. stream the selected row once, then sample
    const int r = sh_gamma, rtok = sh_rtok;
    const float rq = sh_rq;
    const int vt = ve.v_t;
    const float *row = ve.target_probs + (int64_t)(t0 + b + r) * ve.target_ld;
    const bool vec = p.vec4 != 0;
    const float rp = sh_rp;
    vcore::stream_chunks(row, vt, vec, 0, p.nc, kThreads / kWave, rtok, rq, rp,
                         [&](int c, uint64_t sum) { sh_part[c] = sum; }, &sh_next);
    TT_STAMP(4);
    __syncthreads();
    TT_STAMP(5);
    if (wave != 0) return;
    uint64_t Z;
    const int token =
        vcore::wave_sample(row, nullptr, vt, p.nc, vec, [&](int c) { return sh_part[c]; }, us, rtok, rq, &Z);
    if (lane == 0) {
        ve.n_accepted[b] = r;
        ve.out_token[b] = token;
        p.zsum[b] = Z;
        p.rsel[b] = r;
    }
    TT_STAMP_WAVE(6);
}

template <int TB, bool STREAM>
int launch_tb(const SParams &p, size_t lds, hipStream_t stream) {
    if (lds > 64 * 1024 &&
        hipFuncSetAttribute(reinterpret_cast<const void *>(&step_fused<TB, STREAM>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
        return TT_ELAUNCH;
    hipLaunchKernelGGL((step_fused<TB, STREAM>), dim3(p.s.ve.n_streams), dim3(kThreads), lds, stream, p);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

template <bool STREAM>
int launch_any_tb(const SParams &p, int tb, size_t lds, hipStream_t stream) {
    switch (tb) {
        case 8: return launch_tb<8, STREAM>(p, lds, stream);
        case 16: return launch_tb<16, STREAM>(p, lds, stream);
        case 32: return launch_tb<32, STREAM>(p, lds, stream);
        default: return launch_tb<64, STREAM>(p, lds, stream);
    }
}

SParams make_sparams(const StepArgs &s, const VerifyLayout &L) {
    uint8_t *ws = static_cast<uint8_t *>(s.ve.workspace);
    SParams p;
    p.s = s;
    p.zsum = reinterpret_cast<uint64_t *>(ws + L.zsum);
    p.rsel = reinterpret_cast<int32_t *>(ws + L.rsel);
    p.nc = L.n_chunks;
    p.vec4 = ((reinterpret_cast<uintptr_t>(s.ve.target_probs) & 15u) == 0 && (s.ve.target_ld % 4) == 0) ? 1 : 0;
    return p;
}

}  // namespace

// The fused kernel gives each stream one workgroup: the right shape once the streams fill the
// chip, and for short rows at any batch size (a row of <= 16K floats is a few chunks, so the
// launches saved outweigh the one compute unit per stream: 1 stream at V_t = 640 takes 8.6 us
// fused against 12.8 us as three calls; 32 streams at V_t = 151,936 take 22 us fused against 17).
constexpr int32_t kFusedShortRow = 16384;

bool step_fused_fits(const StepArgs &s, int tb) {
    return (tb == 8 || tb == 16 || tb == 32 || tb == 64) && align_rows_fits(s.al.max_k, s.al.max_m) &&
           s.ve.max_m <= rows::kMaxSide &&
           (verify_row_path(s.ve.n_streams, s.ve.v_t) || s.ve.v_t <= kFusedShortRow) &&
           8 * (size_t)verify_layout(s.ve.n_streams, s.ve.v_t).n_chunks <= kDynLdsMax;
}

int launch_step_fused(const StepArgs &s, int tb, hipStream_t stream) {
    if (!step_fused_fits(s, tb)) return TT_EUNSUPPORTED;
    const VerifyLayout L = verify_layout(s.ve.n_streams, s.ve.v_t);
    if (s.ve.workspace == nullptr || s.ve.workspace_bytes < L.total) return TT_EWORKSPACE;
    const SParams p = make_sparams(s, L);
    const int st = launch_any_tb<true>(p, tb, 8 * (size_t)p.nc, stream);
    if (st != TT_OK) return st;
    return s.ve.residual != nullptr ? launch_verify_residual(s.ve, stream) : TT_OK;
}

bool step_front_fits(const StepArgs &s, int tb) {
    return (tb == 8 || tb == 16 || tb == 32 || tb == 64) && align_rows_fits(s.al.max_k, s.al.max_m) &&
           s.ve.max_m <= rows::kMaxSide;
}

int launch_step_front(const StepArgs &s, int tb, hipStream_t stream) {
    if (!step_front_fits(s, tb)) return TT_EUNSUPPORTED;
    const VerifyLayout L = verify_layout(s.ve.n_streams, s.ve.v_t);
    if (s.ve.workspace == nullptr || s.ve.workspace_bytes < L.total) return TT_EWORKSPACE;
    const SParams p = make_sparams(s, L);
    const int st = launch_any_tb<false>(p, tb, 0, stream);
    if (st != TT_OK) return st;
    return launch_verify_after_gamma(s.ve, stream);
}

}  // namespace tt
