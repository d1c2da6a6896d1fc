// Position deviation of matched tokens (Sec. 5 "DTW Bridges the Gap", Fig. CDF; App. K
// "Settings of w"): a draft / proxy target pair (i, j) on an optimal warping path deviates
// by |i - j| positions.  The histogram over a batch of aligned pairs is what App. K's
// procedure reads to place the band half-width w (the offset where the CDF reaches 0.9,
// collected with w = infinity); delta_quantile reads that offset off the histogram.
//
// Two launches: a fill kernel clears the histogram (no memset node, so the call can be
// captured in a HIP graph), then up to 256 workgroups of 256 threads count their pairs into
// LDS histograms (one atomic per run of equal deviation in a thread's eight consecutive
// cells) and add their non-zero bins to the global one with device-scope atomics.
// The result does not depend on the order of the additions.
#include "tt_internal.h"

namespace tt {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxGroups = 256;  // one per compute unit: fewer global atomics on the shared bins
constexpr int kRun = 8;           // consecutive path cells per thread

__global__ void __launch_bounds__(kThreads) hist_clear(int32_t *hist, int n_bins) {
    for (int d = threadIdx.x; d < n_bins; d += kThreads) hist[d] = 0;
}

__global__ void __launch_bounds__(kThreads) delta_hist(int32_t n_pairs, const int32_t *draft_off,
                                                       const int32_t *target_off, const int32_t *path_len,
                                                       const int32_t *path, int n_bins, int32_t *hist) {
    extern __shared__ int32_t sh_hist[];
    for (int d = threadIdx.x; d < n_bins; d += kThreads) sh_hist[d] = 0;
    __syncthreads();
    const int last = n_bins - 1;
    for (int b = blockIdx.x; b < n_pairs; b += gridDim.x) {
        const int K = draft_off[b + 1] - draft_off[b], M = target_off[b + 1] - target_off[b];
        const int n = path_len[b];
        if (n <= 0 || n > K + M) continue;  // sentinel pair, or a length the path area cannot hold
        const int32_t *cells = path + 2 * (int64_t)(draft_off[b] + target_off[b]);
        // kRun consecutive cells per thread: along a path i - j changes by at most one per
        // step, so a thread's cells form few runs of equal deviation and it adds once per run
        for (int c0 = threadIdx.x * kRun; c0 < n; c0 += kThreads * kRun) {
            const int c1 = c0 + kRun < n ? c0 + kRun : n;
            int cur = -1, cnt = 0;
            for (int c = c0; c < c1; ++c) {
                int dev = abs(cells[2 * c] - cells[2 * c + 1]);
                dev = dev < last ? dev : last;
                if (dev != cur) {
                    if (cnt) atomicAdd(&sh_hist[cur], cnt);
                    cur = dev;
                    cnt = 0;
                }
                ++cnt;
            }
            if (cnt) atomicAdd(&sh_hist[cur], cnt);
        }
    }
    __syncthreads();
    for (int d = threadIdx.x; d < n_bins; d += kThreads)
        if (sh_hist[d] != 0) atomicAdd(&hist[d], sh_hist[d]);
}

// App. K: the smallest d with (hist[0] + ... + hist[d]) * den >= num * total, exact in int64
// (|hist| < 2^31 and n_bins <= 8192 keep the prefixes below 2^44, den <= 65536 the products
// below 2^60); 0 when the total is 0.  One workgroup: 32 bins per thread, a scan of the
// thread sums in LDS, the first bin reaching the quantile by an LDS minimum.
constexpr int kQuantBins = 32;

__global__ void __launch_bounds__(kThreads) delta_quantile(const int32_t *hist, int n_bins, int32_t num, int32_t den,
                                                           int32_t *out) {
    __shared__ int64_t sums[kThreads];
    __shared__ int first;
    const int t = threadIdx.x;
    const int b0 = t * kQuantBins;
    int64_t own = 0;
    for (int k = 0; k < kQuantBins && b0 + k < n_bins; ++k) own += hist[b0 + k];
    sums[t] = own;
    if (t == 0) first = n_bins - 1;
    __syncthreads();
    for (int off = 1; off < kThreads; off <<= 1) {  // inclusive scan of the thread sums
        const int64_t v = t >= off ? sums[t - off] : 0;
        __syncthreads();
        sums[t] += v;
        __syncthreads();
    }
    const int64_t total = sums[kThreads - 1];
    if (total == 0) {
        if (t == 0) *out = 0;
        return;
    }
    const int64_t need = (int64_t)num * total;
    int64_t cum = sums[t] - own;
    for (int k = 0; k < kQuantBins && b0 + k < n_bins; ++k) {
        cum += hist[b0 + k];
        if (cum * (int64_t)den >= need) {
            atomicMin(&first, b0 + k);
            break;
        }
    }
    __syncthreads();
    if (t == 0) *out = first;
}

}  // namespace

int launch_delta_quantile(const int32_t *hist, int32_t n_bins, int32_t num, int32_t den, int32_t *d_out,
                          hipStream_t stream) {
    hipLaunchKernelGGL(delta_quantile, dim3(1), dim3(kThreads), 0, stream, hist, n_bins, num, den, d_out);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

int launch_delta_histogram(int32_t n_pairs, const int32_t *draft_off, const int32_t *target_off,
                           const int32_t *path_len, const int32_t *path, int32_t n_bins, int32_t *hist,
                           hipStream_t stream) {
    hipLaunchKernelGGL(hist_clear, dim3(1), dim3(kThreads), 0, stream, hist, n_bins);
    if (hipGetLastError() != hipSuccess) return TT_ELAUNCH;
    if (n_pairs == 0) return TT_OK;
    const int groups = n_pairs < kMaxGroups ? n_pairs : kMaxGroups;
    hipLaunchKernelGGL(delta_hist, dim3(groups), dim3(kThreads), sizeof(int32_t) * (size_t)n_bins, stream, n_pairs,
                       draft_off, target_off, path_len, path, n_bins, hist);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ELAUNCH;
}

}  // namespace tt
