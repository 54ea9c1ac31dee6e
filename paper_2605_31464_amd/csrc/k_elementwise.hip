// Bandwidth-bound kernels: embedding gather, RMSNorm, RoPE, fp32 SwiGLU, row gather,
// full-vocab log-softmax + verdict read-out, and selective deferral.
#include <climits>

#include "common.h"
#include "kernels.h"

namespace surr {
namespace {

// ---------------------------------------------------------------- embedding gather
// One wavefront per packed token t: find its prompt b (cu[b] <= t < cu[b+1]) by binary
// search, read the token id, and widen the embedding row to the fp32 residual.
template <bool BF16>
__global__ __launch_bounds__(256) void embed_kernel(const int32_t* __restrict__ tokens,
                                                    int64_t row_stride,
                                                    const int32_t* __restrict__ cu, int B,
                                                    int64_t T, const void* __restrict__ embed,
                                                    int d, int vocab, float* __restrict__ x,
                                                    int32_t* __restrict__ pos,
                                                    const int32_t* __restrict__ pos_off,
                                                    const int32_t* __restrict__ vt_off,
                                                    int32_t* __restrict__ vcol,
                                                    int32_t* __restrict__ err_flag) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= T) return;
    int lo = 0, hi = B;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (cu[mid] <= t) lo = mid; else hi = mid;
    }
    const int j = (int)(t - cu[lo]);
    int tok = tokens[(int64_t)lo * row_stride + j];
    if (tok < 0 || tok >= vocab) {
        if (lane == 0) err_flag[0] = 1;
        tok = 0;
    }
    if (lane == 0) {
        pos[t] = pos_off ? pos_off[lo] + j : j;
        if (vcol) vcol[t] = vt_off[lo] + vt_key_order(j);
    }
    float4* xr = reinterpret_cast<float4*>(x + t * d);
    if constexpr (BF16) {
        const uint4* er = reinterpret_cast<const uint4*>(
            static_cast<const uint16_t*>(embed) + (int64_t)tok * d);
        for (int c = lane; c < d / 8; c += 64) {
            const uint4 v = er[c];
            xr[2 * c] = make_float4(bf16_to_f32(v.x & 0xffffu), bf16_to_f32(v.x >> 16),
                                    bf16_to_f32(v.y & 0xffffu), bf16_to_f32(v.y >> 16));
            xr[2 * c + 1] = make_float4(bf16_to_f32(v.z & 0xffffu), bf16_to_f32(v.z >> 16),
                                        bf16_to_f32(v.w & 0xffffu), bf16_to_f32(v.w >> 16));
        }
    } else {
        const float4* er = reinterpret_cast<const float4*>(
            static_cast<const float*>(embed) + (int64_t)tok * d);
        for (int c = lane; c < d / 4; c += 64) xr[c] = er[c];
    }
}

// ---------------------------------------------------------------- V^T padding
// Prompt b owns columns [vt_off[b], vt_off[b + 1]) of the transposed V copy; stored
// column c holds key vt_key_order(c), so the columns whose key is >= L_b are padding.
// They start inside the last 16-key group at the earliest.
__global__ __launch_bounds__(256) void vt_pad_zero_kernel(uint16_t* __restrict__ vt, int64_t ld_vt,
                                                          int rows, const int32_t* __restrict__ cu,
                                                          const int32_t* __restrict__ vt_off) {
    const int b = blockIdx.x;
    const int L = cu[b + 1] - cu[b], base = vt_off[b];
    const int c0 = L & ~15, nc = vt_off[b + 1] - base - c0;
    const int64_t n = (int64_t)rows * nc;
    for (int64_t e = (int64_t)blockIdx.y * 256 + threadIdx.x; e < n; e += (int64_t)gridDim.y * 256) {
        const int r = (int)(e / nc), c = c0 + (int)(e - (int64_t)r * nc);
        if (vt_key_order(c) >= L) vt[(int64_t)r * ld_vt + base + c] = 0;
    }
}

// ---------------------------------------------------------------- RMSNorm
// One wavefront per row; fp32 sum of squares reduced in a fixed butterfly order.
// Two passes over the row (the second mostly from L2); used for rows longer than the
// single-pass kernel below holds in registers.
template <bool OUT_BF16>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* __restrict__ x, int64_t ldx,
                                                      const int32_t* __restrict__ rows,
                                                      int64_t n_rows, const float* __restrict__ g,
                                                      int d, float eps, void* __restrict__ y,
                                                      int64_t ldy) {
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= n_rows) return;
    const int64_t src = rows ? (int64_t)rows[r] : r;
    const float4* xr = reinterpret_cast<const float4*>(x + src * ldx);
    const float4* g4 = reinterpret_cast<const float4*>(g);
    float ss = 0.f;
    for (int c = lane; c < d / 4; c += 64) {
        const float4 v = xr[c];
        ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    }
    ss = wave_sum(ss);
    const float sc = rsqrtf(ss / (float)d + eps);
    for (int c = lane; c < d / 4; c += 64) {
        const float4 v = xr[c];
        const float4 w = g4[c];
        const float a = v.x * sc * w.x, b = v.y * sc * w.y, e = v.z * sc * w.z, f = v.w * sc * w.w;
        if constexpr (OUT_BF16) {
            uint2 o;
            o.x = pack_bf16x2(a, b);
            o.y = pack_bf16x2(e, f);
            reinterpret_cast<uint2*>(static_cast<uint16_t*>(y) + r * ldy)[c] = o;
        } else {
            reinterpret_cast<float4*>(static_cast<float*>(y) + r * ldy)[c] = make_float4(a, b, e, f);
        }
    }
}

// Single-pass form for rows of at most 256 * NC values: lane l keeps the float4 chunks
// l, l + 64, ... of its row in registers, so x is read from HBM exactly once.  Same
// arithmetic and reduction order as the two-pass kernel above.  With PRE_G the gains are
// loaded together with x (one memory round trip instead of two; used for the few-row
// calls of decode steps, where latency, not bandwidth, sets the time).
template <bool OUT_BF16, int NC, bool PRE_G = false>
__global__ __launch_bounds__(256) void rmsnorm_reg_kernel(const float* __restrict__ x,
                                                          int64_t ldx,
                                                          const int32_t* __restrict__ rows,
                                                          int64_t n_rows,
                                                          const float* __restrict__ g, int d,
                                                          float eps, void* __restrict__ y,
                                                          int64_t ldy) {
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= n_rows) return;
    const int64_t src = rows ? (int64_t)rows[r] : r;
    const float4* xr = reinterpret_cast<const float4*>(x + src * ldx);
    const float4* g4 = reinterpret_cast<const float4*>(g);
    const int n4 = d / 4;
    float4 v[NC];
    float4 gw[PRE_G ? NC : 1];
#pragma unroll
    for (int k = 0; k < NC; ++k) {
        const int c = lane + 64 * k;
        v[k] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (c < n4) v[k] = xr[c];
        if constexpr (PRE_G) {
            gw[k] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (c < n4) gw[k] = g4[c];
        }
    }
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < NC; ++k)
        if (lane + 64 * k < n4) ss += v[k].x * v[k].x + v[k].y * v[k].y + v[k].z * v[k].z + v[k].w * v[k].w;
    ss = wave_sum(ss);
    const float sc = rsqrtf(ss / (float)d + eps);
#pragma unroll
    for (int k = 0; k < NC; ++k) {
        const int c = lane + 64 * k;
        if (c >= n4) continue;
        float4 w;
        if constexpr (PRE_G) w = gw[k];
        else w = g4[c];
        const float a = v[k].x * sc * w.x, b = v[k].y * sc * w.y, e = v[k].z * sc * w.z,
                    f = v[k].w * sc * w.w;
        if constexpr (OUT_BF16) {
            uint2 o;
            o.x = pack_bf16x2(a, b);
            o.y = pack_bf16x2(e, f);
            reinterpret_cast<uint2*>(static_cast<uint16_t*>(y) + r * ldy)[c] = o;
        } else {
            reinterpret_cast<float4*>(static_cast<float*>(y) + r * ldy)[c] = make_float4(a, b, e, f);
        }
    }
}

template <bool OUT_BF16>
hipError_t rmsnorm_dispatch(const float* x, int64_t ldx, const int32_t* rows, int64_t n_rows,
                            const float* g, int d, float eps, void* y, int64_t ldy,
                            hipStream_t s) {
    const unsigned grid = (unsigned)((n_rows + 3) / 4);
    const int nc = (d / 4 + 63) / 64;
#define SURR_RMS_REG(NC_)                                                                        \
    do {                                                                                         \
        if (n_rows <= 256)                                                                       \
            rmsnorm_reg_kernel<OUT_BF16, NC_, true><<<grid, 256, 0, s>>>(x, ldx, rows, n_rows, g, d, eps, y, ldy); \
        else                                                                                     \
            rmsnorm_reg_kernel<OUT_BF16, NC_><<<grid, 256, 0, s>>>(x, ldx, rows, n_rows, g, d, eps, y, ldy); \
    } while (0)
    if (nc <= 2) SURR_RMS_REG(2);
    else if (nc <= 4) SURR_RMS_REG(4);
    else if (nc <= 8) SURR_RMS_REG(8);
    else if (nc <= 16) SURR_RMS_REG(16);
    else if (nc <= 24) SURR_RMS_REG(24);
    else
        rmsnorm_kernel<OUT_BF16><<<grid, 256, 0, s>>>(x, ldx, rows, n_rows, g, d, eps, y, ldy);
#undef SURR_RMS_REG
    return hipGetLastError();
}

// ---------------------------------------------------------------- RoPE
// One thread per rotated pair (token, head, i < hd/2): dims i and i + hd/2 rotate by
// theta = pos * base^(-2i/hd), whose cos/sin come from the float32 table cs[pos][i].
template <bool BF16>
__global__ __launch_bounds__(256) void rope_kernel(void* __restrict__ qkv, int64_t ld, int64_t T,
                                                   const int32_t* __restrict__ pos, int n_heads,
                                                   int hd, const float2* __restrict__ cs) {
    const int half = hd >> 1;
    const int64_t per_tok = (int64_t)n_heads * half;
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= T * per_tok) return;
    const int64_t t = idx / per_tok;
    const int rem = (int)(idx - t * per_tok);
    const int h = rem / half, i = rem - (rem / half) * half;
    const float2 c = cs[(int64_t)pos[t] * half + i];
    const int64_t e1 = t * ld + (int64_t)h * hd + i, e2 = e1 + half;
    if constexpr (BF16) {
        uint16_t* p = static_cast<uint16_t*>(qkv);
        const float x1 = bf16_to_f32(p[e1]), x2 = bf16_to_f32(p[e2]);
        p[e1] = (uint16_t)f32_to_bf16(x1 * c.x - x2 * c.y);
        p[e2] = (uint16_t)f32_to_bf16(x2 * c.x + x1 * c.y);
    } else {
        float* p = static_cast<float*>(qkv);
        const float x1 = p[e1], x2 = p[e2];
        p[e1] = x1 * c.x - x2 * c.y;
        p[e2] = x2 * c.x + x1 * c.y;
    }
}

// ---------------------------------------------------------------- fp32 SwiGLU
__global__ __launch_bounds__(256) void swiglu_f32_kernel(const float* __restrict__ gu,
                                                         float* __restrict__ u, int64_t T,
                                                         int d_ff) {
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= T * d_ff) return;
    const int64_t t = idx / d_ff;
    const int j = (int)(idx - t * d_ff);
    const float* row = gu + t * 2 * (int64_t)d_ff + (j >> 5) * 64 + (j & 31);
    const float gv = row[0], uv = row[32];
    u[idx] = gv / (1.f + expf(-gv)) * uv;
}

// ---------------------------------------------------------------- row gather
__global__ __launch_bounds__(256) void gather_rows_kernel(const uint32_t* __restrict__ src,
                                                          int64_t ld_src,
                                                          const int32_t* __restrict__ rows,
                                                          int words,
                                                          uint32_t* __restrict__ dst,
                                                          int64_t ld_dst) {
    const int64_t r = blockIdx.x;
    const uint32_t* s = src + (int64_t)rows[r] * ld_src;
    uint32_t* o = dst + r * ld_dst;
    for (int c = threadIdx.x; c < words; c += 256) o[c] = s[c];
}

// Inverse of gather_rows: row r of src goes to row rows[r] of dst.
__global__ __launch_bounds__(256) void scatter_rows_kernel(const uint32_t* __restrict__ src,
                                                           int64_t ld_src,
                                                           const int32_t* __restrict__ rows,
                                                           int words,
                                                           uint32_t* __restrict__ dst,
                                                           int64_t ld_dst) {
    const int64_t r = blockIdx.x;
    const uint32_t* s = src + r * ld_src;
    uint32_t* o = dst + (int64_t)rows[r] * ld_dst;
    for (int c = threadIdx.x; c < words; c += 256) o[c] = s[c];
}

// Row r of a 64-row-aligned cache: prompt b = the last with po[b] <= r, j = r - po[b];
// copies columns [col0, col0 + words) of packed row cu[b] + j when j < L_b, else zeros.
__global__ __launch_bounds__(256) void capture_rows_kernel(const uint32_t* __restrict__ src,
                                                           int64_t ld_src, int col0, int words,
                                                           const int32_t* __restrict__ cu,
                                                           const int32_t* __restrict__ po, int B,
                                                           uint32_t* __restrict__ dst,
                                                           int64_t ld_dst) {
    const int64_t r = blockIdx.x;
    int lo = 0, hi = B;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (po[mid] <= r) lo = mid; else hi = mid;
    }
    const int j = (int)(r - po[lo]);
    uint32_t* o = dst + r * ld_dst;
    if (j < cu[lo + 1] - cu[lo]) {
        const uint32_t* sr = src + (int64_t)(cu[lo] + j) * ld_src + col0;
        for (int c = threadIdx.x; c < words; c += 256) o[c] = sr[c];
    } else {
        for (int c = threadIdx.x; c < words; c += 256) o[c] = 0u;
    }
}

// ---------------------------------------------------------------- sequence caches
// Token j of prompt b (packed row t = cu[b] + j) continues its sequence at position
// len[b] + j: columns [col0, col0 + words) of row t go to cache row off[b] + len[b] + j.
__device__ __forceinline__ void append_row(int64_t t, const uint32_t* __restrict__ src,
                                           int64_t ld_src, int col0, int words,
                                           const int32_t* __restrict__ cu, int B,
                                           const int32_t* __restrict__ off,
                                           const int32_t* __restrict__ len,
                                           uint32_t* __restrict__ dst, int64_t ld_dst) {
    int lo = 0, hi = B;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (cu[mid] <= t) lo = mid; else hi = mid;
    }
    const int64_t r = (int64_t)off[lo] + len[lo] + (t - cu[lo]);
    const uint32_t* sr = src + t * ld_src + col0;
    uint32_t* o = dst + r * ld_dst;
    for (int c = threadIdx.x; c < words; c += 256) o[c] = sr[c];
}

__global__ __launch_bounds__(256) void append_rows_kernel(const uint32_t* __restrict__ src,
                                                          int64_t ld_src, int col0, int words,
                                                          const int32_t* __restrict__ cu, int B,
                                                          const int32_t* __restrict__ off,
                                                          const int32_t* __restrict__ len,
                                                          uint32_t* __restrict__ dst,
                                                          int64_t ld_dst) {
    append_row(blockIdx.x, src, ld_src, col0, words, cu, B, off, len, dst, ld_dst);
}

// Transposed V of the same tokens: column vt_off[b] + pi(j) of vt goes to column
// off[b] + pi(len[b] + j) of the cache's V^T (pi = vt_key_order, applied to the index
// inside the 64-aligned block of each side).  Block (b, 64-token chunk), threads over rows.
__device__ __forceinline__ void append_vt_chunk(int b, int j0, const uint16_t* __restrict__ vt,
                                                int64_t ld_vt, const int32_t* __restrict__ vt_off,
                                                const int32_t* __restrict__ cu,
                                                const int32_t* __restrict__ off,
                                                const int32_t* __restrict__ len, int rows,
                                                uint16_t* __restrict__ cvt, int64_t ld_c) {
    const int L = cu[b + 1] - cu[b];
    if (j0 >= L) return;
    const int jn = min(64, L - j0), base = len[b];
    for (int d = threadIdx.x; d < rows; d += 256) {
        const uint16_t* sr = vt + (int64_t)d * ld_vt + vt_off[b];
        uint16_t* o = cvt + (int64_t)d * ld_c + off[b];
        for (int j = j0; j < j0 + jn; ++j) o[vt_key_order(base + j)] = sr[vt_key_order(j)];
    }
}

__global__ __launch_bounds__(256) void append_vt_kernel(const uint16_t* __restrict__ vt,
                                                        int64_t ld_vt,
                                                        const int32_t* __restrict__ vt_off,
                                                        const int32_t* __restrict__ cu,
                                                        const int32_t* __restrict__ off,
                                                        const int32_t* __restrict__ len,
                                                        int rows, uint16_t* __restrict__ cvt,
                                                        int64_t ld_c) {
    append_vt_chunk(blockIdx.x, blockIdx.y * 64, vt, ld_vt, vt_off, cu, off, len, rows, cvt, ld_c);
}

// Both appends of a bf16 layer in one launch (a decode step's appends are a few rows, so
// the launch, not the copy, is the cost): blocks [0, T) copy the K row of token t, the
// rest copy 64-token chunks of V^T, chunks blocks per prompt.
__global__ __launch_bounds__(256) void append_kv_kernel(const uint32_t* __restrict__ src,
                                                        int64_t ld_src, int col0, int words,
                                                        int64_t T, const uint16_t* __restrict__ vt,
                                                        int64_t ld_vt,
                                                        const int32_t* __restrict__ vt_off,
                                                        const int32_t* __restrict__ cu, int B,
                                                        const int32_t* __restrict__ off,
                                                        const int32_t* __restrict__ len,
                                                        uint32_t* __restrict__ ck, int64_t ld_ck,
                                                        int rows, uint16_t* __restrict__ cvt,
                                                        int64_t ld_c, int chunks) {
    const int64_t i = blockIdx.x;
    if (i < T) {
        append_row(i, src, ld_src, col0, words, cu, B, off, len, ck, ld_ck);
    } else {
        const int64_t v = i - T;
        append_vt_chunk((int)(v / chunks), (int)(v % chunks) * 64, vt, ld_vt, vt_off, cu, off, len,
                        rows, cvt, ld_c);
    }
}

// Full-vocabulary LSE of one row of logits by a workgroup of kLseThreads threads, and
// optionally its first argmax.  Thread t reads the 16-byte chunks t, t + kLseThreads, ...
// (each wavefront step covers 1 KB contiguous), so a row streams at full width instead of
// one value per thread.  Every reduction runs in a fixed order (a thread's values in index
// order, a butterfly across lanes, then the waves in order), so the result depends on the
// row alone.  max ignores NaN (fmaxf); the argmax takes the larger value, the lower index
// on ties.
constexpr int kLseThreads = 1024, kLseWaves = kLseThreads / 64;

template <bool ARGMAX>
__device__ __forceinline__ void row_lse(const float* __restrict__ z, int V, float* red, int* redi,
                                        float& lse, int& argmax) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int V4 = (V % 4 == 0 && (reinterpret_cast<uintptr_t>(z) & 15) == 0) ? V / 4 : 0;
    const float4* z4 = reinterpret_cast<const float4*>(z);
    float mx = -INFINITY;
    int am = V;
    auto take = [&](float v, int i) {
        if constexpr (ARGMAX) {
            if (v > mx) { mx = v; am = i; }
        } else {
            mx = fmaxf(mx, v);
        }
    };
    for (int i = tid; i < V4; i += kLseThreads) {
        const float4 v = z4[i];
        take(v.x, 4 * i);
        take(v.y, 4 * i + 1);
        take(v.z, 4 * i + 2);
        take(v.w, 4 * i + 3);
    }
    for (int i = 4 * V4 + tid; i < V; i += kLseThreads) take(z[i], i);
    if constexpr (ARGMAX) {
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const float ov = __shfl_xor(mx, o, 64);
            const int oi = __shfl_xor(am, o, 64);
            if (ov > mx || (ov == mx && oi < am)) { mx = ov; am = oi; }
        }
    } else {
        mx = wave_max(mx);
    }
    if (lane == 0) { red[wave] = mx; redi[wave] = am; }
    __syncthreads();
    mx = red[0];
    am = redi[0];
    for (int w = 1; w < kLseWaves; ++w) {
        if constexpr (ARGMAX) {
            if (red[w] > mx || (red[w] == mx && redi[w] < am)) { mx = red[w]; am = redi[w]; }
        } else {
            mx = fmaxf(mx, red[w]);
        }
    }
    __syncthreads();
    float sum = 0.f;
    for (int i = tid; i < V4; i += kLseThreads) {
        const float4 v = z4[i];
        sum += expf(v.x - mx);
        sum += expf(v.y - mx);
        sum += expf(v.z - mx);
        sum += expf(v.w - mx);
    }
    for (int i = 4 * V4 + tid; i < V; i += kLseThreads) sum += expf(z[i] - mx);
    sum = wave_sum(sum);
    if (lane == 0) red[wave] = sum;
    __syncthreads();
    float tot = red[0];
    for (int w = 1; w < kLseWaves; ++w) tot += red[w];
    lse = mx + logf(tot);
    argmax = am;
}

// Next-token read-out per row of logits: the full-vocabulary LSE (as in
// lse_verdict_kernel), the first argmax, and optionally the log-prob of a given target id.
__global__ __launch_bounds__(kLseThreads) void lse_next_kernel(const float* __restrict__ logits, int64_t ld,
                                                               int V, const int32_t* __restrict__ target,
                                                               int32_t* __restrict__ next_token,
                                                               float* __restrict__ target_lp) {
    __shared__ float red[kLseWaves];
    __shared__ int redi[kLseWaves];
    const int b = blockIdx.x;
    const float* z = logits + (int64_t)b * ld;
    float lse;
    int am;
    row_lse<true>(z, V, red, redi, lse, am);
    if (threadIdx.x == 0) {
        if (next_token) next_token[b] = am;
        if (target_lp) target_lp[b] = z[target[b]] - lse;
    }
}

// Verdict read-out of row b from its verdict logits zv[0 .. nv) and the full-vocabulary
// log-sum-exp: lp_v = zv[v] - lse, p = softmax(lp), q = max p and the first argmax.
__device__ void verdict_readout(const float* zv, int nv, float lse, int b, float* lp,
                                float* probs, float* conf, int32_t* verdict) {
    float l[16];
    float m2 = -INFINITY;
    for (int v = 0; v < nv; ++v) {
        l[v] = zv[v] - lse;
        lp[b * nv + v] = l[v];
        m2 = fmaxf(m2, l[v]);
    }
    float se = 0.f;
    for (int v = 0; v < nv; ++v) {
        l[v] = expf(l[v] - m2);
        se += l[v];
    }
    int best = 0;
    float q = -1.f;
    for (int v = 0; v < nv; ++v) {
        const float p = l[v] / se;
        if (probs) probs[b * nv + v] = p;
        if (p > q) {
            q = p;
            best = v;
        }
    }
    conf[b] = q;
    if (verdict) verdict[b] = best;
}

// ---------------------------------------------------------------- LSE + verdicts
// One workgroup per prompt.  LSE = max + log(sum exp(z - max)) over the full vocabulary
// (fixed-order reductions), lp_v = z[vid_v] - LSE, then p = softmax(lp), q = max p and
// the first argmax.
__global__ __launch_bounds__(kLseThreads) void lse_verdict_kernel(const float* __restrict__ logits,
                                                                  int64_t ld, int V,
                                                                  const int32_t* __restrict__ vid, int nv,
                                                                  float* __restrict__ lp,
                                                                  float* __restrict__ probs,
                                                                  float* __restrict__ conf,
                                                                  int32_t* __restrict__ verdict) {
    __shared__ float red[kLseWaves];
    __shared__ int redi[kLseWaves];
    const int b = blockIdx.x;
    const float* z = logits + (int64_t)b * ld;
    float lse;
    int am;
    row_lse<false>(z, V, red, redi, lse, am);
    if (threadIdx.x == 0) {
        float zv[16];
        for (int v = 0; v < nv; ++v) zv[v] = z[vid[v]];
        verdict_readout(zv, nv, lse, b, lp, probs, conf, verdict);
    }
}

// ---------------------------------------------------------------- LSE from tile records
// One workgroup per row merges the row's n_tiles records (max m_t, sum s_t of exp(z - m_t),
// first argmax a_t) written by the LM head's Epi::LseTile epilogue: thread t folds tiles
// t, t + 256, ... in order, then the partials merge by a fixed butterfly inside each wave
// and in wave order, so the result does not depend on timing.  The merge of (m1, s1, a1)
// and (m2, s2, a2) is (max, s1 e^(m1 - max) + s2 e^(m2 - max), the argmax of the larger
// maximum, the lower index on a tie).
constexpr int kCombThreads = 256, kCombWaves = kCombThreads / 64;

struct LseRec {
    float m, s;
    int a;
};

__device__ __forceinline__ LseRec lse_merge(LseRec x, LseRec y) {
    const float nm = fmaxf(x.m, y.m);
    const float sx = x.m > -INFINITY ? x.s * expf(x.m - nm) : 0.f;
    const float sy = y.m > -INFINITY ? y.s * expf(y.m - nm) : 0.f;
    LseRec r;
    r.a = y.m > x.m ? y.a : (x.m > y.m ? x.a : min(x.a, y.a));
    r.s = sx + sy;
    r.m = nm;
    return r;
}

__global__ __launch_bounds__(kCombThreads) void lse_combine_kernel(
    const float4* __restrict__ part, int n_tiles, const float* __restrict__ picked, int nv,
    float* __restrict__ lp, float* __restrict__ probs, float* __restrict__ conf,
    int32_t* __restrict__ verdict, int32_t* __restrict__ next_token, float* __restrict__ target_lp) {
    __shared__ LseRec red[kCombWaves];
    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float4* rp = part + (int64_t)b * n_tiles;
    LseRec acc{-INFINITY, 0.f, INT_MAX};
    for (int t = tid; t < n_tiles; t += kCombThreads) {
        const float4 r = rp[t];
        acc = lse_merge(acc, LseRec{r.x, r.y, __float_as_int(r.z)});
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        LseRec other{__shfl_xor(acc.m, o, 64), __shfl_xor(acc.s, o, 64), __shfl_xor(acc.a, o, 64)};
        acc = lse_merge(acc, other);
    }
    if (lane == 0) red[wave] = acc;
    __syncthreads();
    if (tid != 0) return;
    LseRec tot = red[0];
    for (int w = 1; w < kCombWaves; ++w) tot = lse_merge(tot, red[w]);
    const float lse = tot.m + logf(tot.s);
    const float* pk = picked + (int64_t)b * kPicked;
    if (nv > 0) {
        float zv[kMaxVerdicts];
        for (int v = 0; v < nv; ++v) zv[v] = pk[v];
        verdict_readout(zv, nv, lse, b, lp, probs, conf, verdict);
    }
    if (next_token) next_token[b] = tot.a;
    if (target_lp) target_lp[b] = pk[kMaxVerdicts] - lse;
}

// ---------------------------------------------------------------- selection
// One workgroup of 1024 threads selects and compacts n <= 65536 candidates.  With
// P = ceil(n / 1024) <= 64, wave w owns the contiguous segment [64 P w, 64 P (w + 1)) and
// holds it in registers as P chunks of 64 consecutive candidates (lane l of chunk c is
// candidate 64 P w + 64 c + l), so every load and every compacted store of a wave is
// contiguous.  A candidate is deferred when
//   threshold (MODE 0): !(q >= tau);
//   budget    (MODE 1): its rank in (NaN first, q ascending, index ascending) is below k;
//   top score (MODE 2): its rank in (score descending, NaN last, index ascending) is below k.
// Ranked modes map each value to a 32-bit key whose unsigned order is the ranking order
// (NaN to -inf or +inf, -0.0 to +0.0, top score negated), find the k-th smallest key by
// a four-pass 8-bit radix select (LDS histograms in 16 lane-group copies, so lanes with
// equal digits do not serialize on one address), then defer every key below it and the
// first (k - #below) keys equal to it in index order.  Tie ranks and output offsets come
// from ballots inside a wave and one exclusive scan over the 16 wave totals.
constexpr int kSelThreads = 1024, kSelWaves = kSelThreads / 64, kSelChunks = 64,
              kHistPitch = 257;

__device__ __forceinline__ uint32_t order_key(float v) {
    if (v == 0.f) v = 0.f;  // -0.0 and +0.0 rank as equal
    const uint32_t u = __float_as_uint(v);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix over waves of a wave-uniform count; *total gets the sum.
__device__ __forceinline__ uint32_t wave_exclusive_scan(uint32_t v, uint32_t* wsum,
                                                        uint32_t* total) {
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) wsum[wave] = v;
    __syncthreads();
    uint32_t before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
        const uint32_t x = wsum[w];
        before += w < wave ? x : 0u;
        all += x;
    }
    __syncthreads();  // wsum is reused by the next scan
    *total = all;
    return before;
}

template <int MODE>
__global__ __launch_bounds__(kSelThreads) void select_kernel(const float* __restrict__ q, int n,
                                                             float tau, int k,
                                                             int32_t* __restrict__ defer_idx,
                                                             int32_t* __restrict__ accept_idx,
                                                             int32_t* __restrict__ counts) {
    __shared__ uint32_t hist[16 * kHistPitch];
    __shared__ uint32_t wsum[kSelWaves];
    __shared__ uint32_t sel[2];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int P = (n + kSelThreads - 1) / kSelThreads;
    const int seg = wave * 64 * P + lane;  // candidate of chunk c is seg + 64 c
    const uint64_t below = (1ull << lane) - 1ull;

    // Slots past n hold kNone, above every ranked key (the largest, +inf, maps to
    // 0xff800000) and distinct from the threshold flags 0/1, so they are never deferred,
    // never tie with the k-th key and sort after every candidate.
    constexpr uint32_t kNone = 0xffffffffu;
    uint32_t key[kSelChunks];
#pragma unroll
    for (int c = 0; c < kSelChunks; ++c) {
        key[c] = kNone;
        if (c < P) {
            const int i = seg + 64 * c;
            if (i < n) {
                const float v = q[i];
                if (MODE == 0) key[c] = !(v >= tau);
                else if (MODE == 1) key[c] = order_key(__builtin_isnan(v) ? -INFINITY : v);
                else key[c] = order_key(__builtin_isnan(v) ? INFINITY : -v);
            }
        }
    }

    uint32_t kth = 0, take = 0;  // defer keys < kth, and the first `take` keys == kth
    if (MODE != 0 && k > 0 && k < n) {
        uint32_t prefix = 0, pmask = 0, r = (uint32_t)(k - 1);
        for (int pass = 0; pass < 4; ++pass) {
            const int shift = 24 - 8 * pass;
            for (int j = tid; j < 16 * kHistPitch; j += kSelThreads) hist[j] = 0u;
            __syncthreads();
            uint32_t* h = hist + (lane & 15) * kHistPitch;
            // rank r < n lies among the candidates, so counting the kNone slots (all in
            // the top bins) does not move the k-th key
#pragma unroll
            for (int c = 0; c < kSelChunks; ++c)
                if (c < P && (key[c] & pmask) == prefix) atomicAdd(&h[(key[c] >> shift) & 255u], 1u);
            __syncthreads();
            if (tid < 64) {
                uint32_t b4[4], sum = 0;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    uint32_t x = 0;
                    for (int cp = 0; cp < 16; ++cp) x += hist[cp * kHistPitch + 4 * lane + e];
                    b4[e] = x;
                    sum += x;
                }
                uint32_t incl = sum;
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) {
                    const uint32_t t = __shfl_up(incl, o, 64);
                    if (lane >= o) incl += t;
                }
                uint32_t c0 = incl - sum;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if (r >= c0 && r < c0 + b4[e]) {
                        sel[0] = 4 * lane + e;
                        sel[1] = r - c0;
                    }
                    c0 += b4[e];
                }
            }
            __syncthreads();
            prefix |= sel[0] << shift;
            pmask |= 255u << shift;
            r = sel[1];
        }
        kth = prefix;
        take = r + 1;
    }

    // Deferred count of the wave, then offsets, then the flags again in index order while
    // storing.  Ranked modes with 0 < k < n: a wave defers its keys below the k-th and, of
    // its keys equal to it, those whose tie rank (ties in earlier waves first) is below take.
    const bool ranked = MODE != 0 && k > 0 && k < n;
    const bool all = MODE != 0 && k >= n;
    uint32_t nf = 0, seen = 0;
    if (ranked) {
        uint32_t nless = 0, neq = 0, unused;
#pragma unroll
        for (int c = 0; c < kSelChunks; ++c) {
            if (c < P) {
                nless += __popcll(__ballot(key[c] < kth));
                neq += __popcll(__ballot(key[c] == kth));
            }
        }
        seen = wave_exclusive_scan(neq, wsum, &unused);  // ties in earlier waves
        const int left = max(0, (int)take - (int)seen);
        nf = nless + (uint32_t)min(left, (int)neq);
    } else {
#pragma unroll
        for (int c = 0; c < kSelChunks; ++c)
            if (c < P) nf += __popcll(__ballot(MODE == 0 ? key[c] == 1u : (all && key[c] != kNone)));
    }
    uint32_t n_defer;
    uint32_t j = wave_exclusive_scan(nf, wsum, &n_defer);  // deferred before this wave
#pragma unroll
    for (int c = 0; c < kSelChunks; ++c) {
        if (c < P) {
            bool f;
            if (ranked) {
                const bool eq = key[c] == kth;
                const uint64_t em = __ballot(eq);
                f = key[c] < kth || (eq && seen + __popcll(em & below) < take);
                seen += __popcll(em);
            } else {
                f = MODE == 0 ? key[c] == 1u : (all && key[c] != kNone);
            }
            const uint64_t fb = __ballot(f);
            const int i = seg + 64 * c;
            if (i < n) {
                const int pos = (int)(j + __popcll(fb & below));
                if (f) defer_idx[pos] = i;
                else accept_idx[i - pos] = i;
            }
            j += __popcll(fb);
        }
    }
    if (tid == 0) {
        counts[0] = (int32_t)n_defer;
        counts[1] = n - (int32_t)n_defer;
    }
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

hipError_t launch_embed(Act wt, const int32_t* tokens, int64_t row_stride, const int32_t* cu,
                        int B, int64_t T, const void* embed, int d, int vocab, float* x,
                        int32_t* pos, const int32_t* pos_off, const int32_t* vt_off, int32_t* vcol,
                        int32_t* err_flag, hipStream_t s) {
    if (wt == Act::BF16)
        embed_kernel<true><<<blocks_for(T, 4), 256, 0, s>>>(tokens, row_stride, cu, B, T, embed,
                                                            d, vocab, x, pos, pos_off, vt_off, vcol,
                                                            err_flag);
    else
        embed_kernel<false><<<blocks_for(T, 4), 256, 0, s>>>(tokens, row_stride, cu, B, T, embed,
                                                             d, vocab, x, pos, pos_off, vt_off,
                                                             vcol, err_flag);
    return hipGetLastError();
}

hipError_t launch_capture_rows(const void* src, int64_t ld_src, int col0, int cols, int elem_bytes,
                               const int32_t* cu, const int32_t* po, int B, int64_t rows,
                               void* dst, int64_t ld_dst, hipStream_t s) {
    if (rows == 0) return hipSuccess;
    // moved as 4-byte words: cols, col0 and both leading dimensions times elem_bytes are
    // multiples of 4 for every caller (head_dim is even)
    capture_rows_kernel<<<(unsigned)rows, 256, 0, s>>>(
        static_cast<const uint32_t*>(src), ld_src * elem_bytes / 4, col0 * elem_bytes / 4,
        cols * elem_bytes / 4, cu, po, B, static_cast<uint32_t*>(dst), ld_dst * elem_bytes / 4);
    return hipGetLastError();
}

hipError_t launch_vt_pad_zero(uint16_t* vt, int64_t ld_vt, int rows, const int32_t* cu,
                              const int32_t* vt_off, int B, hipStream_t s) {
    if (B == 0 || rows == 0) return hipSuccess;
    vt_pad_zero_kernel<<<dim3(B, 16), 256, 0, s>>>(vt, ld_vt, rows, cu, vt_off);
    return hipGetLastError();
}

hipError_t launch_rmsnorm(Act out, const float* x, int64_t ldx, const int32_t* rows,
                          int64_t n_rows, const float* g, int d, float eps, void* y, int64_t ldy,
                          hipStream_t s) {
    if (n_rows == 0) return hipSuccess;
    if (out == Act::BF16) return rmsnorm_dispatch<true>(x, ldx, rows, n_rows, g, d, eps, y, ldy, s);
    return rmsnorm_dispatch<false>(x, ldx, rows, n_rows, g, d, eps, y, ldy, s);
}

hipError_t launch_rope(Act t, void* qkv, int64_t ld, int64_t T, const int32_t* pos, int n_heads,
                       int head_dim, const float2* cs, hipStream_t s) {
    const int64_t n = T * n_heads * (head_dim / 2);
    if (n == 0) return hipSuccess;
    if (t == Act::BF16)
        rope_kernel<true><<<blocks_for(n, 256), 256, 0, s>>>(qkv, ld, T, pos, n_heads, head_dim, cs);
    else
        rope_kernel<false><<<blocks_for(n, 256), 256, 0, s>>>(qkv, ld, T, pos, n_heads, head_dim, cs);
    return hipGetLastError();
}

hipError_t launch_swiglu_f32(const float* gu, float* u, int64_t T, int d_ff, hipStream_t s) {
    const int64_t n = T * d_ff;
    if (n == 0) return hipSuccess;
    swiglu_f32_kernel<<<blocks_for(n, 256), 256, 0, s>>>(gu, u, T, d_ff);
    return hipGetLastError();
}

hipError_t launch_gather_rows(const void* src, int64_t ld_src, const int32_t* rows, int64_t n,
                              int cols, int elem_bytes, void* dst, int64_t ld_dst, hipStream_t s) {
    if (n == 0) return hipSuccess;
    // rows are moved as 4-byte words: cols * elem_bytes and the leading dimensions (in
    // bytes) are multiples of 4 for every caller (even bf16 widths).
    const int words = cols * elem_bytes / 4;
    gather_rows_kernel<<<(unsigned)n, 256, 0, s>>>(static_cast<const uint32_t*>(src),
                                                   ld_src * elem_bytes / 4, rows, words,
                                                   static_cast<uint32_t*>(dst),
                                                   ld_dst * elem_bytes / 4);
    return hipGetLastError();
}

hipError_t launch_scatter_rows(const void* src, int64_t ld_src, const int32_t* rows, int64_t n,
                               int cols, int elem_bytes, void* dst, int64_t ld_dst, hipStream_t s) {
    if (n == 0) return hipSuccess;
    if ((cols * elem_bytes) % 4 || (ld_src * elem_bytes) % 4 || (ld_dst * elem_bytes) % 4)
        return hipErrorInvalidValue;
    scatter_rows_kernel<<<(unsigned)n, 256, 0, s>>>(static_cast<const uint32_t*>(src),
                                                    ld_src * elem_bytes / 4, rows,
                                                    cols * elem_bytes / 4,
                                                    static_cast<uint32_t*>(dst),
                                                    ld_dst * elem_bytes / 4);
    return hipGetLastError();
}

hipError_t launch_lse_verdict(const float* logits, int64_t ld, int B, int V, const int32_t* vid,
                              int nv, float* lp, float* probs, float* conf, int32_t* verdict,
                              hipStream_t s) {
    lse_verdict_kernel<<<B, kLseThreads, 0, s>>>(logits, ld, V, vid, nv, lp, probs, conf, verdict);
    return hipGetLastError();
}

hipError_t launch_append_rows(const void* src, int64_t ld_src, int col0, int cols, int elem_bytes,
                              int64_t T, const int32_t* cu, int B, const int32_t* off,
                              const int32_t* len, void* dst, int64_t ld_dst, hipStream_t s) {
    if (T == 0) return hipSuccess;
    append_rows_kernel<<<(unsigned)T, 256, 0, s>>>(
        static_cast<const uint32_t*>(src), ld_src * elem_bytes / 4, col0 * elem_bytes / 4,
        cols * elem_bytes / 4, cu, B, off, len, static_cast<uint32_t*>(dst), ld_dst * elem_bytes / 4);
    return hipGetLastError();
}

hipError_t launch_append_vt(const uint16_t* vt, int64_t ld_vt, const int32_t* vt_off,
                            const int32_t* cu, int B, int max_len, const int32_t* off,
                            const int32_t* len, int rows, uint16_t* cvt, int64_t ld_c,
                            hipStream_t s) {
    if (B == 0 || max_len == 0) return hipSuccess;
    append_vt_kernel<<<dim3(B, (max_len + 63) / 64), 256, 0, s>>>(vt, ld_vt, vt_off, cu, off, len,
                                                                 rows, cvt, ld_c);
    return hipGetLastError();
}

hipError_t launch_append_kv(const uint16_t* qkv, int64_t ld_qkv, int col0, int cols, int64_t T,
                            const uint16_t* vt, int64_t ld_vt, const int32_t* vt_off,
                            const int32_t* cu, int B, int max_len, const int32_t* off,
                            const int32_t* len, uint16_t* ck, int64_t ld_ck, int rows,
                            uint16_t* cvt, int64_t ld_c, hipStream_t s) {
    if (T == 0) return hipSuccess;
    if (ld_qkv % 2 || col0 % 2 || cols % 2 || ld_ck % 2) return hipErrorInvalidValue;
    const int chunks = (max_len + 63) / 64;
    const int64_t blocks = T + (int64_t)B * chunks;
    if (blocks > INT32_MAX) return hipErrorInvalidValue;
    append_kv_kernel<<<(unsigned)blocks, 256, 0, s>>>(
        reinterpret_cast<const uint32_t*>(qkv), ld_qkv / 2, col0 / 2, cols / 2, T, vt, ld_vt, vt_off,
        cu, B, off, len, reinterpret_cast<uint32_t*>(ck), ld_ck / 2, rows, cvt, ld_c, chunks);
    return hipGetLastError();
}

hipError_t launch_lse_combine(const float4* part, int n_tiles, const float* picked, int B, int nv,
                              float* lp, float* probs, float* conf, int32_t* verdict,
                              int32_t* next_token, float* target_lp, hipStream_t s) {
    if (B <= 0) return hipSuccess;
    lse_combine_kernel<<<B, kCombThreads, 0, s>>>(part, n_tiles, picked, nv, lp, probs, conf, verdict,
                                                  next_token, target_lp);
    return hipGetLastError();
}

hipError_t launch_lse_next(const float* logits, int64_t ld, int B, int V, const int32_t* target,
                           int32_t* next_token, float* target_lp, hipStream_t s) {
    lse_next_kernel<<<B, kLseThreads, 0, s>>>(logits, ld, V, target, next_token, target_lp);
    return hipGetLastError();
}

hipError_t launch_select(const float* conf, int n, int mode, float tau, int k, int32_t* defer_idx,
                         int32_t* accept_idx, int32_t* counts, hipStream_t s) {
    if (n < 1 || n > kSelThreads * kSelChunks || k < 0) return hipErrorInvalidValue;
    if (mode == 0)
        select_kernel<0><<<1, kSelThreads, 0, s>>>(conf, n, tau, k, defer_idx, accept_idx, counts);
    else if (mode == 1)
        select_kernel<1><<<1, kSelThreads, 0, s>>>(conf, n, tau, k, defer_idx, accept_idx, counts);
    else
        select_kernel<2><<<1, kSelThreads, 0, s>>>(conf, n, tau, k, defer_idx, accept_idx, counts);
    return hipGetLastError();
}

}  // namespace surr
