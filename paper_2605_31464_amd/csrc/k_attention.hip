// Causal grouped-query prefill attention over ragged packed prompts.
//
// bf16 path (v_mfma_f32_32x32x16_bf16, online softmax in fp32).  A workgroup owns 128
// query rows of one prompt and one query head; each of its 4 wavefronts owns 32 rows.
// K/V tiles of 64 keys are staged in LDS (K row-major with a 16-byte-chunk XOR swizzle,
// V transposed to [dim][key]).  The wavefront computes the transposed score block
// S^T = K Q^T, so a lane holds one query and 16 of its keys; the probabilities P^T then
// already sit in the B-operand layout of O^T += V^T P^T once the 16 keys of each MFMA
// step are taken in the order the score layout gives them (the contraction order is
// free as long as both operands agree).  Row statistics are lane-local apart from one
// exchange between the two 32-lane halves, which hold the same queries.
//
// fp32 path: one thread per query row, exact expf, for the float32 model.
#include "common.h"
#include "kernels.h"

namespace surr {
namespace {

constexpr int kBQ = 128, kBKV = 64;

template <int HD>
__global__ __launch_bounds__(256) void attn_bf16_kernel(const uint16_t* __restrict__ qkv,
                                                        int64_t ld, uint16_t* __restrict__ out,
                                                        int64_t ld_out,
                                                        const int32_t* __restrict__ cu,
                                                        const int2* __restrict__ work, int nqh,
                                                        int nkvh, float scale_log2) {
    constexpr int NCH = HD / 8;  // 16-byte chunks per K row
    constexpr int KS = HD / 16;  // MFMA steps over the head dim for S
    constexpr int DB = HD / 32;  // 32-dim blocks of O
    constexpr int VTP = kBKV + 8;  // Vt row pitch in bf16 elements
    __shared__ uint4 Ks[kBKV * NCH];
    __shared__ __attribute__((aligned(16))) uint16_t Vt[HD * VTP];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h = lane >> 5, l32 = lane & 31;
    const int item = blockIdx.x / nqh, head = blockIdx.x - (blockIdx.x / nqh) * nqh;
    const int2 wk = work[item];
    const int start = cu[wk.x], L = cu[wk.x + 1] - start;
    const int q0 = wk.y * kBQ;
    const int kvh = head * nkvh / nqh;
    const int64_t k_col = (int64_t)(nqh + kvh) * HD, v_col = (int64_t)(nqh + nkvh + kvh) * HD;
    const uint16_t* base = qkv + (int64_t)start * ld;

    const int qw0 = q0 + wave * 32;
    const int my_q = qw0 + l32;
    const bool wave_active = qw0 < L;

    bf16x8 qf[KS];
    {
        const uint16_t* qrow = base + (int64_t)min(my_q, L - 1) * ld + (int64_t)head * HD + 8 * h;
#pragma unroll
        for (int s = 0; s < KS; ++s)
            qf[s] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(qrow + 16 * s));
    }

    f32x16 o[DB];
#pragma unroll
    for (int d = 0; d < DB; ++d) o[d] = f32x16{};
    float m_run = -INFINITY, l_run = 0.f;

    const int kv_end = min(L, q0 + kBQ);
    const int n_tiles = (kv_end + kBKV - 1) / kBKV;
    for (int t = 0; t < n_tiles; ++t) {
        const int k0 = t * kBKV;
        __syncthreads();
        for (int e = tid; e < kBKV * NCH; e += 256) {
            const int r = e / NCH, c = e - (e / NCH) * NCH;
            const int row = min(k0 + r, L - 1);
            Ks[r * NCH + (c ^ (r & (NCH - 1)))] =
                *reinterpret_cast<const uint4*>(base + (int64_t)row * ld + k_col + c * 8);
        }
        for (int e = tid; e < (kBKV / 2) * NCH; e += 256) {
            const int p = e / NCH, c = e - (e / NCH) * NCH;
            const int r0 = min(k0 + 2 * p, L - 1), r1 = min(k0 + 2 * p + 1, L - 1);
            const uint4 a = *reinterpret_cast<const uint4*>(base + (int64_t)r0 * ld + v_col + c * 8);
            const uint4 b = *reinterpret_cast<const uint4*>(base + (int64_t)r1 * ld + v_col + c * 8);
            const uint32_t av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
            uint32_t* dst = reinterpret_cast<uint32_t*>(Vt) + ((c * 8) * VTP + 2 * p) / 2;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                dst[(2 * i) * (VTP / 2)] = (av[i] & 0xffffu) | (bv[i] << 16);
                dst[(2 * i + 1) * (VTP / 2)] = (av[i] >> 16) | (bv[i] & 0xffff0000u);
            }
        }
        __syncthreads();
        if (!wave_active || k0 > qw0 + 31) continue;  // no key of this tile precedes a query

        f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const int r = kb * 32 + l32;
#pragma unroll
            for (int st = 0; st < KS; ++st) {
                const int chunk = 2 * st + h;
                const bf16x8 a = __builtin_bit_cast(bf16x8, Ks[r * NCH + (chunk ^ (r & (NCH - 1)))]);
                s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[st], s[kb], 0, 0, 0);
            }
        }
        // s[kb][e]: key k0 + 32 kb + 8 (e / 4) + 4 h + e % 4, query my_q.
        const bool need_mask = (k0 + kBKV - 1 > qw0) || (k0 + kBKV > L);
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                float v = s[kb][e] * scale_log2;
                if (need_mask) {
                    const int key = k0 + 32 * kb + 8 * (e >> 2) + 4 * h + (e & 3);
                    if (key > my_q || key >= L) v = -INFINITY;
                }
                s[kb][e] = v;
                mx = fmaxf(mx, v);
            }
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float m_new = fmaxf(m_run, mx);
        const float corr = fast_exp2(m_run - m_new);
        m_run = m_new;
        l_run *= corr;
#pragma unroll
        for (int d = 0; d < DB; ++d) o[d] *= corr;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
                float pv[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    pv[i] = fast_exp2(s[kb][8 * s2 + i] - m_new);
                    l_run += pv[i];
                }
                const uint4 pp = {pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]),
                                  pack_bf16x2(pv[4], pv[5]), pack_bf16x2(pv[6], pv[7])};
                const bf16x8 pb = __builtin_bit_cast(bf16x8, pp);
#pragma unroll
                for (int d = 0; d < DB; ++d) {
                    const uint16_t* vr = Vt + (d * 32 + l32) * VTP + 32 * kb + 16 * s2 + 4 * h;
                    const uint2 lo = *reinterpret_cast<const uint2*>(vr);
                    const uint2 hi = *reinterpret_cast<const uint2*>(vr + 8);
                    const uint4 vv = {lo.x, lo.y, hi.x, hi.y};
                    o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vv),
                                                                   pb, o[d], 0, 0, 0);
                }
            }
    }
    l_run += __shfl_xor(l_run, 32, 64);
    if (!wave_active || my_q >= L) return;
    const float inv = 1.f / l_run;
    uint16_t* orow = out + (int64_t)(start + my_q) * ld_out + (int64_t)head * HD + 4 * h;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            uint2 w;
            w.x = pack_bf16x2(o[d][4 * j] * inv, o[d][4 * j + 1] * inv);
            w.y = pack_bf16x2(o[d][4 * j + 2] * inv, o[d][4 * j + 3] * inv);
            *reinterpret_cast<uint2*>(orow + d * 32 + 8 * j) = w;
        }
}

// ---------------------------------------------------------------- fp32
constexpr int kBQ32 = 64;

template <int HD>
__global__ __launch_bounds__(64) void attn_f32_kernel(const float* __restrict__ qkv, int64_t ld,
                                                      float* __restrict__ out, int64_t ld_out,
                                                      const int32_t* __restrict__ cu,
                                                      const int2* __restrict__ work, int nqh,
                                                      int nkvh, float scale) {
    __shared__ float Ks[64][HD + 1];
    __shared__ float Vs[64][HD + 1];
    const int tid = threadIdx.x;
    const int item = blockIdx.x / nqh, head = blockIdx.x - (blockIdx.x / nqh) * nqh;
    const int2 wk = work[item];
    const int start = cu[wk.x], L = cu[wk.x + 1] - start;
    const int q0 = wk.y * kBQ32;
    const int kvh = head * nkvh / nqh;
    const float* base = qkv + (int64_t)start * ld;
    const int my_q = q0 + tid;
    float q[HD], o[HD];
    const float* qrow = base + (int64_t)min(my_q, L - 1) * ld + (int64_t)head * HD;
#pragma unroll
    for (int d = 0; d < HD; ++d) {
        q[d] = qrow[d];
        o[d] = 0.f;
    }
    float m = -INFINITY, l = 0.f;
    const int kv_end = min(L, q0 + kBQ32);
    for (int k0 = 0; k0 < kv_end; k0 += 64) {
        __syncthreads();
        const float* krow = base + (int64_t)min(k0 + tid, L - 1) * ld;
        for (int d = 0; d < HD; ++d) {
            Ks[tid][d] = krow[(int64_t)(nqh + kvh) * HD + d];
            Vs[tid][d] = krow[(int64_t)(nqh + nkvh + kvh) * HD + d];
        }
        __syncthreads();
        const int lim = min(64, kv_end - k0);
        for (int kk = 0; kk < lim; ++kk) {
            if (k0 + kk > my_q) break;
            float sdot = 0.f;
#pragma unroll
            for (int d = 0; d < HD; ++d) sdot = fmaf(q[d], Ks[kk][d], sdot);
            const float sc = sdot * scale;
            const float m_new = fmaxf(m, sc);
            const float corr = expf(m - m_new), p = expf(sc - m_new);
            l = l * corr + p;
#pragma unroll
            for (int d = 0; d < HD; ++d) o[d] = o[d] * corr + p * Vs[kk][d];
            m = m_new;
        }
    }
    if (my_q >= L) return;
    float* orow = out + (int64_t)(start + my_q) * ld_out + (int64_t)head * HD;
    const float inv = 1.f / l;
#pragma unroll
    for (int d = 0; d < HD; ++d) orow[d] = o[d] * inv;
}

}  // namespace

int attention_q_tile(Act t) { return t == Act::BF16 ? kBQ : kBQ32; }

hipError_t launch_attention(Act t, const void* qkv, int64_t ld_qkv, void* out, int64_t ld_out,
                            const int32_t* cu, const int2* work, int n_items, int n_q_heads,
                            int n_kv_heads, int head_dim, hipStream_t s) {
    if (n_items == 0) return hipSuccess;
    const unsigned grid = (unsigned)n_items * (unsigned)n_q_heads;
    if (t == Act::BF16) {
        const float sl2 = kLog2e / sqrtf((float)head_dim);
        const uint16_t* q = static_cast<const uint16_t*>(qkv);
        uint16_t* o = static_cast<uint16_t*>(out);
        switch (head_dim) {
            case 64: attn_bf16_kernel<64><<<grid, 256, 0, s>>>(q, ld_qkv, o, ld_out, cu, work, n_q_heads, n_kv_heads, sl2); break;
            case 128: attn_bf16_kernel<128><<<grid, 256, 0, s>>>(q, ld_qkv, o, ld_out, cu, work, n_q_heads, n_kv_heads, sl2); break;
            default: return hipErrorInvalidValue;
        }
    } else {
        const float sc = 1.f / sqrtf((float)head_dim);
        const float* q = static_cast<const float*>(qkv);
        float* o = static_cast<float*>(out);
        switch (head_dim) {
            case 32: attn_f32_kernel<32><<<grid, 64, 0, s>>>(q, ld_qkv, o, ld_out, cu, work, n_q_heads, n_kv_heads, sc); break;
            case 64: attn_f32_kernel<64><<<grid, 64, 0, s>>>(q, ld_qkv, o, ld_out, cu, work, n_q_heads, n_kv_heads, sc); break;
            case 128: attn_f32_kernel<128><<<grid, 64, 0, s>>>(q, ld_qkv, o, ld_out, cu, work, n_q_heads, n_kv_heads, sc); break;
            default: return hipErrorInvalidValue;
        }
    }
    return hipGetLastError();
}

}  // namespace surr
