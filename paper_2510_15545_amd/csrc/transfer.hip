// Probability transfer (Alg. 2 "MapProbabilities", App. A.2): for every target
// position j of pair b, q_j = P_d[row draft_off[b] + i][d_i] with i = map(j).
//
// The work is ΣM_b scattered 4-byte gathers, so the kernel is latency-bound; one
// wave per pair keeps the CSR bookkeeping trivial and issues all of a pair's
// gathers at once (map -> draft id -> probability: three dependent loads).
#include <cmath>

#include "tt_internal.h"

namespace tt {
namespace {

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;

__global__ void __launch_bounds__(kWave * kWavesPerBlock) transfer_gather(TransferArgs a) {
    const int b = blockIdx.x * kWavesPerBlock + (int)(threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    if (b >= a.n_pairs) return;
    const int d0 = a.draft_off[b];
    const int K = a.draft_off[b + 1] - d0;
    const int t0 = a.target_off[b], t1 = a.target_off[b + 1];
    for (int t = t0 + lane; t < t1; t += kWave) {
        const int i = a.map[t];
        float v = __builtin_nanf("");
        if (i >= 0 && i < K) {
            const int tok = a.draft_ids[d0 + i];
            if (tok >= 0 && tok < a.v_d) v = a.draft_probs[(int64_t)(d0 + i) * a.draft_ld + tok];
        }
        a.q[t] = v;
    }
}

}  // namespace

int launch_transfer(const TransferArgs &a, hipStream_t stream) {
    const int blocks = (a.n_pairs + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL(transfer_gather, dim3(blocks), dim3(kWave * kWavesPerBlock), 0, stream, a);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

}  // namespace tt
