// Alignment kernel for short pairs (K, M <= 64): one 256-thread workgroup per pair, the
// row-scan formulation of the device functions in dtw_rows.h.
#include "dtw_rows.h"

namespace tt {
namespace {

constexpr int kThreads = 256;

template <int TB>
__global__ void __launch_bounds__(kThreads) dtw_rows(AlignArgs a) {
    __shared__ rows::Lds<TB> s;
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const int d0 = a.draft_off[b], K = a.draft_off[b + 1] - d0;
    const int t0 = a.target_off[b], M = a.target_off[b + 1] - t0;

    const bool shape_ok = K >= 1 && K <= a.max_k && M >= 1 && M <= a.max_m;
    __shared__ int votes[kThreads / rows::kWave];
    const int bad = shape_ok ? rows::stage<TB>(a, s, d0, K, t0, M, tid, kThreads) : 1;
    if (dtw::block_or(bad, votes, kThreads / rows::kWave)) {
        if (tid == 0) {
            a.cost[b] = -1;
            a.path_len[b] = 0;
        }
        for (int j = tid; j < M; j += kThreads) a.map[t0 + j] = -1;
        return;
    }
    const int L = rows::band_half_width(K, M, a.w);
    const int wave = __builtin_amdgcn_readfirstlane(tid / rows::kWave);  // uniform per wave
    rows::init_border<TB>(s, tid, kThreads);
    rows::costs<TB>(s, K, M, L, tid, kThreads);
    __syncthreads();
    int total = 0;
    if (wave == 0) total = rows::recurrence<TB>(s, K, M, L);
    __syncthreads();
    rows::moves<TB>(s, K, M, L, wave, kThreads / rows::kWave);
    __syncthreads();
    if (wave == 0) rows::backtrack<TB>(a, s, b, d0, K, t0, M, total);
}

template <int TB>
int launch_rows_tb(const AlignArgs &a, hipStream_t stream) {
    hipLaunchKernelGGL(dtw_rows<TB>, dim3(a.n_pairs), dim3(kThreads), 0, stream, a);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

}  // namespace

bool align_rows_fits(int32_t max_k, int32_t max_m) { return max_k <= rows::kMaxSide && max_m <= rows::kMaxSide; }

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
