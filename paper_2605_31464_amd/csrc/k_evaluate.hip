// Forecast quality against measured speedups, for scoring batches of rollouts or
// evaluation sets: per candidate the measured bin (Table 3), the correctness reward, the
// Brier score and the CRPS (Section 2.2); over the batch their means, the rewards, the
// expected calibration error over ten confidence buckets and the forecast error
// (Section 3.1); speedup recovered (Section 3.1) from the top-score selections the host
// enqueues per budget.
//
// Up to 256 workgroups of 256 threads stride over the candidates (a wave reads 64
// consecutive rows).  Each keeps its sums in float64 per thread, reduces them in a fixed
// order (wave butterfly, then its four waves in order) and writes one partial row; the
// maxima needed by speedup recovered are partial rows too.  eval_finalize_kernel combines
// the rows in block order, so every result is independent of timing.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace surr {
namespace {

constexpr int kEvThreads = 256, kBuckets = 10;
// per-thread sums: correct, brier, crps, |m_yhat - S|, then per bucket count, confidence
// and correct count
constexpr int kSums = 4 + 3 * kBuckets;

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// partial row of workgroup blk: kSums float64 sums, then the max speedup (as float64)
constexpr int kPart = kSums + 1;

__global__ __launch_bounds__(kEvThreads) void eval_metrics_kernel(
    const float* __restrict__ p, const float* __restrict__ S, int n, int nb, EvalBins bins,
    int32_t* __restrict__ bin_out, float* __restrict__ brier_out, float* __restrict__ crps_out,
    double* __restrict__ partial) {
    __shared__ double part[kEvThreads / 64][kPart];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    double acc[kSums];
#pragma unroll
    for (int j = 0; j < kSums; ++j) acc[j] = 0.0;
    float smax = -INFINITY;
    for (int i = blockIdx.x * kEvThreads + tid; i < n; i += gridDim.x * kEvThreads) {
        float pr[kMaxBins];
#pragma unroll
        for (int b = 0; b < kMaxBins; ++b) pr[b] = b < nb ? p[(int64_t)i * nb + b] : 0.f;
        const float s = S[i];
        smax = fmaxf(smax, s);
        int y = 0;  // edges strictly below the speedup
#pragma unroll
        for (int j = 0; j < kMaxBins - 1; ++j) y += (j < nb - 1 && (double)s > bins.edge[j]);
        int yh = 0;  // first argmax
#pragma unroll
        for (int b = 1; b < kMaxBins; ++b)
            if (b < nb && pr[b] > pr[yh]) yh = b;
        float q = 0.f, br = 0.f, cr = 0.f, F = 0.f, myh = 0.f;
#pragma unroll
        for (int b = 0; b < kMaxBins; ++b) {
            if (b < nb) {
                if (b == yh) { q = pr[b]; myh = bins.value[b]; }
                const float d = pr[b] - (b == y ? 1.f : 0.f);
                br = fmaf(d, d, br);
                if (b < nb - 1) {
                    F += pr[b];
                    const float c = F - (y <= b ? 1.f : 0.f);
                    cr = fmaf(c, c, cr);
                }
            }
        }
        br *= 0.5f;
        cr /= (float)(nb - 1);
        const double correct = yh == y ? 1.0 : 0.0;
        acc[0] += correct;
        acc[1] += br;
        acc[2] += cr;
        acc[3] += fabs((double)myh - (double)s);
        const int m = min(max((int)floorf(q * 10.f), 0), kBuckets - 1);
#pragma unroll
        for (int k = 0; k < kBuckets; ++k) {
            if (k == m) {
                acc[4 + k] += 1.0;
                acc[4 + kBuckets + k] += q;
                acc[4 + 2 * kBuckets + k] += correct;
            }
        }
        if (bin_out) bin_out[i] = y;
        if (brier_out) brier_out[i] = br;
        if (crps_out) crps_out[i] = cr;
    }
#pragma unroll
    for (int j = 0; j < kSums; ++j) {
        const double v = wave_sum_f64(acc[j]);
        if (lane == 0) part[wave][j] = v;
    }
    smax = wave_max(smax);
    if (lane == 0) part[wave][kSums] = smax;
    __syncthreads();
    if (tid < kPart) {
        double t = tid == kSums ? -INFINITY : 0.0;
        for (int w = 0; w < kEvThreads / 64; ++w)
            t = tid == kSums ? fmax(t, part[w][tid]) : t + part[w][tid];
        partial[(int64_t)blockIdx.x * kPart + tid] = t;
    }
}

// Partial maxima of speedup over each budget's selected list: block (c, b) covers list
// entries b, b + nb_blk, ... of budget c (lists + 2 n c, counts[2 c] entries).
__global__ __launch_bounds__(kEvThreads) void recovered_part_kernel(
    const float* __restrict__ S, int n, const int32_t* __restrict__ lists,
    const int32_t* __restrict__ counts, float* __restrict__ partial) {
    __shared__ float wmax[kEvThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int c = blockIdx.y;
    const int32_t* list = lists + (int64_t)c * 2 * n;
    const int cnt = counts[2 * c];
    float u = -INFINITY;
    for (int j = blockIdx.x * kEvThreads + tid; j < cnt; j += gridDim.x * kEvThreads)
        u = fmaxf(u, S[list[j]]);
    u = wave_max(u);
    if (lane == 0) wmax[wave] = u;
    __syncthreads();
    if (tid == 0) {
        float r = wmax[0];
        for (int w = 1; w < kEvThreads / 64; ++w) r = fmaxf(r, wmax[w]);
        partial[(int64_t)c * gridDim.x + blockIdx.x] = r;
    }
}

// Combine the partial rows in block order and write the summary.
__global__ __launch_bounds__(64) void eval_finalize_kernel(const double* __restrict__ part,
                                                           int n_blk, const float* __restrict__ rec,
                                                           int rec_blk, int n_budgets, int n,
                                                           double* __restrict__ summary) {
    __shared__ double t[kPart];
    const int tid = threadIdx.x;
    if (tid < kPart) {
        double v = tid == kSums ? -INFINITY : 0.0;
        for (int b = 0; b < n_blk; ++b)
            v = tid == kSums ? fmax(v, part[(int64_t)b * kPart + tid]) : v + part[(int64_t)b * kPart + tid];
        t[tid] = v;
    }
    __syncthreads();
    if (tid != 0) return;
    const double inv = 1.0 / n;
    summary[0] = t[0] * inv;               // accuracy (mean correctness reward)
    summary[1] = t[1] * inv;               // mean Brier
    summary[2] = t[2] * inv;               // mean CRPS
    summary[3] = (t[0] + n - t[1]) * inv;  // mean of r_corr + 1 - Brier
    summary[4] = (t[0] + n - t[2]) * inv;  // mean of r_corr + 1 - CRPS
    double e = 0.0;                        // sum_m |B_m|/n |acc_m - conf_m|
    for (int k = 0; k < kBuckets; ++k) e += fabs(t[4 + 2 * kBuckets + k] - t[4 + kBuckets + k]);
    summary[5] = e * inv;
    summary[6] = t[3] * inv;               // forecast error
    const double best = t[kSums];
    double mean = 0.0;
    for (int c = 0; c < n_budgets; ++c) {
        float r = -INFINITY;
        for (int b = 0; b < rec_blk; ++b) r = fmaxf(r, rec[(int64_t)c * rec_blk + b]);
        const double v = 100.0 * (double)r / best;
        summary[8 + c] = v;
        mean += v;
    }
    summary[7] = mean / n_budgets;
}

}  // namespace

static int eval_blocks(int n) { return std::min(256, (n + kEvThreads - 1) / kEvThreads); }

size_t eval_partial_bytes(int n, int n_budgets) {
    return (size_t)eval_blocks(n) * (kPart * sizeof(double) + (size_t)n_budgets * sizeof(float));
}

hipError_t launch_eval_metrics(const float* probs, const float* speedup, int n, int n_bins,
                               const EvalBins& bins, int32_t* bin_out, float* brier_out,
                               float* crps_out, double* partial, hipStream_t s) {
    eval_metrics_kernel<<<eval_blocks(n), kEvThreads, 0, s>>>(probs, speedup, n, n_bins, bins,
                                                              bin_out, brier_out, crps_out, partial);
    return hipGetLastError();
}

hipError_t launch_eval_finalize(const float* speedup, int n, const int32_t* lists,
                                const int32_t* counts, int n_budgets, double* partial,
                                double* summary, hipStream_t s) {
    const int nb = eval_blocks(n);
    float* rec = reinterpret_cast<float*>(partial + (size_t)nb * kPart);
    recovered_part_kernel<<<dim3(nb, n_budgets), kEvThreads, 0, s>>>(speedup, n, lists, counts, rec);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    eval_finalize_kernel<<<1, 64, 0, s>>>(partial, nb, rec, nb, n_budgets, n, summary);
    return hipGetLastError();
}

}  // namespace surr
