// The speedup-bin forecast head: per forecast row p_i, weighted sums over the bins.
// Column 0 of the weight table holds the bin representatives m_b, so out_0 is the
// expected speedup S_hat_i = sum_b p_{i,b} m_b (Section 3.1, Table 3); column 1 + c holds
// each bin's share of mass at or above cutoff c, so out_{1+c} is the discovery score
// Pr[g >= x_c] (Section 3.6).  The host builds the table once per call in float64.
//
// Bound: HBM at n * (4 n_bins + 4 (1 + n_cutoffs)) bytes, i.e. a few MB for the largest
// batches; in practice one launch of latency.  One lane per forecast row; a wave reads
// 64 consecutive rows, so the loads of a wave cover one contiguous span.
#include "common.h"
#include "kernels.h"

namespace surr {
namespace {

__global__ __launch_bounds__(256) void forecast_head_kernel(const float* __restrict__ p,
                                                            int64_t n, int nb, BinWeights w,
                                                            int nc, float* __restrict__ speedup,
                                                            float* __restrict__ disc) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    float pr[kMaxBins];
#pragma unroll
    for (int b = 0; b < kMaxBins; ++b) pr[b] = b < nb ? p[i * nb + b] : 0.f;
    if (speedup) {
        float acc = 0.f;
#pragma unroll
        for (int b = 0; b < kMaxBins; ++b)
            if (b < nb) acc = fmaf(pr[b], w.w[b][0], acc);
        speedup[i] = acc;
    }
    if (disc) {
#pragma unroll
        for (int c = 0; c < kMaxCutoffs; ++c) {
            if (c >= nc) break;
            float acc = 0.f;
#pragma unroll
            for (int b = 0; b < kMaxBins; ++b)
                if (b < nb) acc = fmaf(pr[b], w.w[b][1 + c], acc);
            disc[i * nc + c] = acc;
        }
    }
}

}  // namespace

hipError_t launch_forecast_head(const float* probs, int64_t n, int n_bins, const BinWeights& w,
                                int n_cutoffs, float* speedup, float* disc, hipStream_t s) {
    if (n == 0 || (!speedup && !disc)) return hipSuccess;
    const unsigned blocks = (unsigned)((n + 255) / 256);
    forecast_head_kernel<<<blocks, 256, 0, s>>>(probs, n, n_bins, w, n_cutoffs, speedup, disc);
    return hipGetLastError();
}

}  // namespace surr
