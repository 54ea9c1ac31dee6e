// Causal grouped-query prefill attention over ragged packed prompts.
//
// bf16 path (v_mfma_f32_32x32x16_bf16, online softmax in fp32).  A workgroup owns 128
// query rows of one prompt and one query head; each of its 4 wavefronts owns 32 rows.
// Two workgroups share a compute unit, so every SIMD runs two wavefronts and the
// hardware overlaps one wavefront's softmax (vector ALU) with the other's MFMAs - a
// single wavefront cannot issue vector instructions back to back.  The wavefront
// computes the transposed score block S^T = K Q^T: a lane then holds one query and 16 of
// its keys per 32-key block, and the probabilities P^T already sit in the B-operand
// layout of O^T += V^T P^T once the 16 keys of each MFMA step are taken in the order the
// score layout gives them (the contraction order is free as long as both operands agree).
//
// Keys move in 64-key tiles from HBM straight into LDS (global_load_lds_dwordx4) through
// a 2-stage ring, the next tile loading while the current one is processed: K rows come
// from the packed qkv rows, V from a transposed copy V^T [kv head * hd + dim][key] that
// the QKV projection writes in its epilogue.  That copy gives each prompt a 64-aligned,
// zero-padded column range and stores the keys of every 16-key group with index bits 2
// and 3 swapped, so the 8 keys one lane feeds the PV MFMA are 16 contiguous bytes.  LDS
// rows are 16-byte-chunk XOR-swizzled so fragment reads are free of bank conflicts.
//
// The running maximum is re-based lazily: O and the row sum are rescaled only when a row
// maximum grows by more than 2^8 (probabilities stay below 256, well inside fp32 and bf16
// range), which is exact up to rounding because numerator and denominator share the base.
//
// Shared prefixes: a prompt that continues a cached prefix of Lp tokens first walks the
// ceil(Lp / 64) tiles of that prefix's cached K and V^T (every query sees every prefix
// key; only the padding past Lp is masked), then its own keys with the causal mask as
// above.
//
// fp32 path: one thread per query row, exact expf, for the float32 model.
#include "common.h"
#include "kernels.h"

namespace surr {
namespace {

constexpr int kWaves = 4, kThreads = 64 * kWaves;  // wavefronts of 32 query rows each
constexpr int kBQ = 32 * kWaves, kBKV = 64, kStages = 2;
constexpr float kLazy = 8.f;

// 16-byte chunk order inside an LDS row of NCH chunks: XOR with a row function such that
// 16 consecutive rows reading one logical chunk hit 16 distinct 16-byte bank groups of
// the 256-byte bank line (a ds_read_b128 serves 16 lanes per pass).  256-byte rows
// (NCH = 16) fill the line alone; 128-byte rows pair up, so the XOR uses row / 2.
template <int NCH>
__device__ __forceinline__ int lds_swz(int row) {
    if constexpr (NCH == 16) return row & 15;
    else return (row >> 1) & 7;
}

// DMA of 64-key tiles into ring stages.  Position p of a stage holds 16-byte chunk
// (p % NCH) ^ lds_swz(row) of K row p / NCH, then, for q = p - 64 NCH, chunk
// (q % 8) ^ lds_swz(d) of V^T row d = q / 8.  Thread tid moves positions i * kThreads + tid; its
// byte offsets from the tile's K row k0 and V^T column k0 are fixed, so a tile costs a
// uniform base and one load per position.  The tile that crosses the prompt's end clamps
// K rows to the last one (keys past the prompt are masked; V^T columns stay inside the
// prompt's padded range).
template <int HD>
struct AttnDma {
    static constexpr int NCH = HD / 8, KCH = kBKV * NCH, HALF = KCH / kThreads;
    static_assert(KCH % kThreads == 0, "whole loads per thread");
    uint32_t koff[HALF], voff[HALF];

    __device__ __forceinline__ AttnDma(int64_t ld, int64_t ld_vt, int tid) {
#pragma unroll
        for (int i = 0; i < HALF; ++i) {
            const int p = i * kThreads + tid;
            const int r = p / NCH, c = (p % NCH) ^ lds_swz<NCH>(r);
            koff[i] = (uint32_t)((r * ld + c * 8) * 2);
            const int d = p >> 3, cv = (p & 7) ^ lds_swz<8>(d);
            voff[i] = (uint32_t)((d * ld_vt + cv * 8) * 2);
        }
    }

    __device__ __forceinline__ void issue(const uint16_t* kbase, int64_t ld, int L,
                                          const uint16_t* vbase, int k0, uint32_t stage_lds,
                                          int tid, int wave) const {
        const uint16_t* kb = kbase + (int64_t)k0 * ld;
        const uint16_t* vb = vbase + k0;
        const uint32_t w = stage_lds + (uint32_t)wave * 64u * 16u;
        if (k0 + kBKV <= L) {
#pragma unroll
            for (int i = 0; i < HALF; ++i) dma_load_16B_sbase(kb, koff[i], w + i * (uint32_t)kThreads * 16u);
        } else {
            const int rmax = L - 1 - k0;
#pragma unroll
            for (int i = 0; i < HALF; ++i) {
                const int p = i * kThreads + tid;
                const int r = p / NCH, c = (p % NCH) ^ lds_swz<NCH>(r);
                dma_load_16B_sbase(kb, (uint32_t)((min(r, rmax) * ld + c * 8) * 2),
                                   w + i * (uint32_t)kThreads * 16u);
            }
        }
#pragma unroll
        for (int i = 0; i < HALF; ++i)
            dma_load_16B_sbase(vb, voff[i], w + (HALF + i) * (uint32_t)kThreads * 16u);
    }

    // A tile of a cached prefix: same LDS placement, the cache's own leading dimensions
    // (offsets formed per tile), never clamped (prefix blocks are whole 64-row tiles).
    __device__ __forceinline__ void issue_prefix(const uint16_t* kbase, int64_t ld_k,
                                                 const uint16_t* vbase, int64_t ld_v, int k0,
                                                 uint32_t stage_lds, int tid, int wave) const {
        const uint16_t* kb = kbase + (int64_t)k0 * ld_k;
        const uint16_t* vb = vbase + k0;
        const uint32_t w = stage_lds + (uint32_t)wave * 64u * 16u;
#pragma unroll
        for (int i = 0; i < HALF; ++i) {
            const int p = i * kThreads + tid;
            const int r = p / NCH, c = (p % NCH) ^ lds_swz<NCH>(r);
            dma_load_16B_sbase(kb, (uint32_t)((r * ld_k + c * 8) * 2), w + i * (uint32_t)kThreads * 16u);
        }
#pragma unroll
        for (int i = 0; i < HALF; ++i) {
            const int p = i * kThreads + tid;
            const int d = p >> 3, cv = (p & 7) ^ lds_swz<8>(d);
            dma_load_16B_sbase(vb, (uint32_t)((d * ld_v + cv * 8) * 2), w + (HALF + i) * (uint32_t)kThreads * 16u);
        }
    }
};

template <int HD, bool PREFIX>
__global__ __launch_bounds__(kThreads, 512 / kThreads) void attn_bf16_kernel(
    const uint16_t* __restrict__ qkv, int64_t ld, const uint16_t* __restrict__ vt, int64_t ld_vt,
    const int32_t* __restrict__ vt_off, uint16_t* __restrict__ out, int64_t ld_out,
    const int32_t* __restrict__ cu, const int2* __restrict__ work, int n_items, int nqh, int nkvh,
    float scale_log2, PrefixKV pf) {
    constexpr int NCH = HD / 8, KCH = kBKV * NCH, CHUNKS = 2 * KCH;
    constexpr int KS = HD / 16;  // MFMA steps over the head dim for S
    constexpr int DB = HD / 32;  // 32-dim blocks of O
    __shared__ uint4 lds[kStages * CHUNKS];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
    const int h = lane >> 5, l32 = lane & 31;
    // Workgroup b runs on XCD b % 8.  XCD x takes work items x, x + 8, x + 16, ... (the
    // host sorted them longest first) with all query heads of an item back to back, so
    // the heads sharing a kv head read its K/V tiles through one XCD's L2.
    const int xk = blockIdx.x >> 3;
    const int item = 8 * (xk / nqh) + (blockIdx.x & 7), head = xk - (xk / nqh) * nqh;
    if (item >= n_items) return;
    const int2 wk = work[item];
    const int start = cu[wk.x], L = cu[wk.x + 1] - start;
    const int q0 = wk.y * kBQ;
    const int kvh = head * nkvh / nqh;
    const uint16_t* kbase = qkv + (int64_t)start * ld + (int64_t)(nqh + kvh) * HD;
    const uint16_t* vbase = vt + (int64_t)kvh * HD * ld_vt + vt_off[wk.x];
    const uint32_t lds0 = lds_offset(lds);
    // Cached prefix: tiles 0 .. np - 1 come from it, the prompt's own tiles follow.
    int Lp = 0, np = 0;
    const uint16_t* kpre = nullptr;
    const uint16_t* vpre = nullptr;
    if constexpr (PREFIX) {
        Lp = pf.len[wk.x];
        np = (Lp + kBKV - 1) / kBKV;
        const int po = pf.off[wk.x];
        kpre = static_cast<const uint16_t*>(pf.k) + (int64_t)po * pf.ld_k + (int64_t)kvh * HD;
        vpre = static_cast<const uint16_t*>(pf.v) + (int64_t)kvh * HD * pf.ld_v + po;
    }

    const int kv_end = min(L, q0 + kBQ);
    const int n_tiles = np + (kv_end + kBKV - 1) / kBKV;
    const int qw0 = q0 + wave * 32;  // first query row of this wavefront
    const int my_q = qw0 + l32;
    // tiles this wavefront needs: the prefix, then keys up to its last valid query row
    const int wave_tiles = qw0 < L ? np + min(qw0 + 31, L - 1) / kBKV + 1 : 0;

    bf16x8 qf[KS];
    {
        const uint16_t* qrow =
            qkv + (int64_t)(start + min(my_q, L - 1)) * ld + (int64_t)head * HD + 8 * h;
#pragma unroll
        for (int st = 0; st < KS; ++st)
            qf[st] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(qrow + 16 * st));
    }
    const AttnDma<HD> dma(ld, ld_vt, tid);
    auto issue_tile = [&](int t, uint32_t stage_lds) {
        if (PREFIX && t < np)
            dma.issue_prefix(kpre, pf.ld_k, vpre, pf.ld_v, t * kBKV, stage_lds, tid, wave);
        else
            dma.issue(kbase, ld, L, vbase, (t - np) * kBKV, stage_lds, tid, wave);
    };
    issue_tile(0, lds0);

    f32x16 o[DB];
#pragma unroll
    for (int d = 0; d < DB; ++d) o[d] = f32x16{};
    float m_ref = -INFINITY, l_sum = 0.f;
    const int lim_q = min(my_q, L - 1);

    wait_vmcnt<0>();
    __syncthreads();
    for (int t = 0; t < n_tiles; ++t) {
        if (t + 1 < n_tiles)  // its stage was released by the barrier that ended tile t - 1
            issue_tile(t + 1, lds0 + (uint32_t)((t + 1) & 1) * CHUNKS * 16u);
        if (t < wave_tiles) {
            const uint4* Ks = lds + (t & 1) * CHUNKS;
            const uint4* Vs = Ks + KCH;
            // s[kb][4 j + i]: key 32 kb + 8 j + 4 h + i of the tile, query my_q
            f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                const int r = kb * 32 + l32;
#pragma unroll
                for (int st = 0; st < KS; ++st) {
                    const bf16x8 a =
                        __builtin_bit_cast(bf16x8, Ks[r * NCH + ((2 * st + h) ^ lds_swz<NCH>(r))]);
                    s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[st], s[kb], 0, 0, 0);
                }
            }
            // keys past lim (counted from key 4 h of the tile) are masked: in a prefix tile
            // those past the prefix; in an own tile those after the query (causal) or past
            // the prompt
            bool masked;  // wave-uniform
            int lim;
            if (PREFIX && t < np) {
                const int k0 = t * kBKV;
                masked = k0 + kBKV > Lp;
                lim = Lp - 1 - (k0 + 4 * h);
            } else {
                const int k0 = (t - np) * kBKV;
                masked = k0 + kBKV - 1 > qw0 || k0 + kBKV > L;
                lim = lim_q - (k0 + 4 * h);
            }
            if (masked) {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int e = 0; e < 16; ++e)
                        s[kb][e] = 32 * kb + 8 * (e >> 2) + (e & 3) > lim ? -INFINITY : s[kb][e];
            }
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kb][e]);
            mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
            const float m_new = mx * scale_log2;
            if (__any(m_new > m_ref + kLazy)) {
                const bool up = m_new > m_ref + kLazy;
                const float c = up ? fast_exp2(m_ref - m_new) : 1.f;
                m_ref = up ? m_new : m_ref;
                l_sum *= c;
#pragma unroll
                for (int d = 0; d < DB; ++d) o[d] *= c;
            }
            const float nm = -m_ref;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int s2 = 0; s2 < 2; ++s2) {
                    float pv[8];
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        pv[i] = fast_exp2(fmaf(s[kb][8 * s2 + i], scale_log2, nm));
                        l_sum += pv[i];
                    }
                    const uint4 pp = {pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]),
                                      pack_bf16x2(pv[4], pv[5]), pack_bf16x2(pv[6], pv[7])};
                    const bf16x8 pb = __builtin_bit_cast(bf16x8, pp);
#pragma unroll
                    for (int d = 0; d < DB; ++d) {
                        const int r = d * 32 + l32;
                        const bf16x8 a = __builtin_bit_cast(
                            bf16x8, Vs[r * 8 + ((4 * kb + 2 * s2 + h) ^ lds_swz<8>(r))]);
                        o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, o[d], 0, 0, 0);
                    }
                }
        }
        if (t + 1 < n_tiles) {
            wait_vmcnt<0>();  // this thread's part of tile t + 1
            __syncthreads();  // all of tile t + 1 visible; stage t & 1 free
        }
    }

    if (wave_tiles == 0 || my_q >= L) return;
    const float inv = 1.f / (l_sum + __shfl_xor(l_sum, 32, 64));
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

template <int HD, bool PREFIX>
__global__ __launch_bounds__(64) void attn_f32_kernel(const float* __restrict__ qkv, int64_t ld,
                                                      float* __restrict__ out, int64_t ld_out,
                                                      const int32_t* __restrict__ cu,
                                                      const int2* __restrict__ work, int nqh,
                                                      int nkvh, float scale, PrefixKV pf) {
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
    if constexpr (PREFIX) {  // every key of the cached prefix, no causal mask
        const int Lp = pf.len[wk.x], po = pf.off[wk.x];
        const float* kp = static_cast<const float*>(pf.k) + (int64_t)po * pf.ld_k + (int64_t)kvh * HD;
        const float* vp = static_cast<const float*>(pf.v) + (int64_t)po * pf.ld_v + (int64_t)kvh * HD;
        for (int k0 = 0; k0 < Lp; k0 += 64) {
            __syncthreads();
            const int r = min(k0 + tid, Lp - 1);
            for (int d = 0; d < HD; ++d) {
                Ks[tid][d] = kp[(int64_t)r * pf.ld_k + d];
                Vs[tid][d] = vp[(int64_t)r * pf.ld_v + d];
            }
            __syncthreads();
            const int lim = min(64, Lp - k0);
            for (int kk = 0; kk < lim; ++kk) {
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
    }
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


// ---------------------------------------------------------------- one-token continuations
// A decode step appends one token to each cached sequence; its attention is one query row
// per head against every key of the entry (the cached ones plus the token's own, which the
// layer has already appended to the cache).  Walking those keys with a 128-row query tile
// would serialise thousands of keys in one workgroup, so the keys are cut into kDecKS-key
// slices instead: workgroup (item, kv head) scores the group's G <= 16 query heads against
// one slice, forms the slice's softmax statistics (max and sum of exp, fp32) and its
// unnormalised weighted V sum, and attn_decode_combine_kernel merges the slices of each
// head in slice order.  Both products run on v_mfma_f32_16x16x32_bf16 with operands read
// straight from the cache in MFMA layout: S^T = K Q^T (16 keys x 16 heads per block;
// wavefront w owns keys [64 w, 64 w + 64) of the slice) and O^T = V^T P^T (16 dims x 16
// heads per block; wavefront w owns HD / 64 blocks of 16 dims), with P in bf16 as in the
// tiled kernel.  V^T column c of an entry holds key vt_key_order(c), so P^T is staged in
// LDS in column order and read back as 16-byte B fragments.  Every step runs in a fixed
// order, so a row's result depends only on its own sequence.
constexpr int kDecKS = 256, kDecMaxG = 16;

template <int HD>
__global__ __launch_bounds__(256) void attn_decode_split_kernel(
    const uint16_t* __restrict__ qkv, int64_t ld_qkv, const int32_t* __restrict__ cu,
    const int2* __restrict__ items, const int32_t* __restrict__ dprompt, int n_q_heads,
    int n_kv_heads, float scale, PrefixKV pk, float* __restrict__ part) {
    constexpr int KS = HD / 32;   // 32-dim steps of the score product
    constexpr int DB = HD / 64;   // 16-dim blocks of O per wavefront
    __shared__ __attribute__((aligned(16))) uint16_t pst[16][kDecKS + 8];  // P^T, column order
    __shared__ float red[2][4][16];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, lg = lane >> 4;
    const int item = blockIdx.x / n_kv_heads, hk = blockIdx.x % n_kv_heads;
    const int2 it = items[item];
    const int b = dprompt[it.x];
    const int G = n_q_heads / n_kv_heads;
    const int nkeys = pk.len[b] + 1;
    const int64_t off = pk.off[b];
    const int k0 = it.y * kDecKS, k1 = min(k0 + kDecKS, nkeys);
    const int64_t t = cu[b];
    const uint16_t* K = static_cast<const uint16_t*>(pk.k);
    const uint16_t* VT = static_cast<const uint16_t*>(pk.v);
    const uint4 zero = {0, 0, 0, 0};

    // all global loads first: Q fragments (head li), K fragments of this wavefront's 64
    // keys, V^T fragments of its dims over the slice (rows of keys past k1 are not read)
    uint4 qf[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s)
        qf[s] = li < G ? *reinterpret_cast<const uint4*>(qkv + t * ld_qkv + (int64_t)(hk * G + li) * HD + 32 * s + 8 * lg)
                       : zero;
    uint4 kf[4][KS];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
        const int key = k0 + 64 * wave + 16 * kb + li;
        const uint16_t* kr = K + (off + key) * pk.ld_k + (int64_t)hk * HD + 8 * lg;
#pragma unroll
        for (int s = 0; s < KS; ++s) kf[kb][s] = key < k1 ? *reinterpret_cast<const uint4*>(kr + 32 * s) : zero;
    }
    const int c_end = (k1 + 15) & ~15;  // V^T columns of 16-key groups that hold live keys
    uint4 vf[DB][kDecKS / 32];
#pragma unroll
    for (int d = 0; d < DB; ++d) {
        const uint16_t* vr = VT + (int64_t)(hk * HD + 16 * (DB * wave + d) + li) * pk.ld_v + off + 8 * lg;
#pragma unroll
        for (int s = 0; s < kDecKS / 32; ++s) {
            const int c = k0 + 32 * s + 8 * lg;
            vf[d][s] = c < c_end ? *reinterpret_cast<const uint4*>(vr + k0 + 32 * s) : zero;
        }
    }

    // S^T = K Q^T: lane holds keys 16 kb + 4 lg + r of its wavefront, head li
    f32x4 sc[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
        sc[kb] = f32x4{};
#pragma unroll
        for (int s = 0; s < KS; ++s)
            sc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kf[kb][s]),
                                                            __builtin_bit_cast(bf16x8, qf[s]), sc[kb], 0, 0, 0);
    }
    // softmax statistics per head li over the slice: max, then sum of exp, fixed order
    float m = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int key = k0 + 64 * wave + 16 * kb + 4 * lg + r;
            sc[kb][r] = key < k1 ? sc[kb][r] * scale : -INFINITY;
            m = fmaxf(m, sc[kb][r]);
        }
    m = fmaxf(m, __shfl_xor(m, 16, 64));
    m = fmaxf(m, __shfl_xor(m, 32, 64));
    if (lg == 0) red[0][wave][li] = m;
    __syncthreads();
    m = fmaxf(fmaxf(red[0][0][li], red[0][1][li]), fmaxf(red[0][2][li], red[0][3][li]));
    float l = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int kl = 64 * wave + 16 * kb + 4 * lg + r;  // key index inside the slice
            const float pv = k0 + kl < k1 ? expf(sc[kb][r] - m) : 0.f;
            l += pv;
            pst[li][vt_key_order(kl)] = (uint16_t)f32_to_bf16(pv);
        }
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    if (lg == 0) red[1][wave][li] = l;
    __syncthreads();

    // O^T = V^T P^T over the slice's 8 steps of 32 columns; dims 16 (DB wave + d) + 4 lg + r
#pragma unroll
    for (int d = 0; d < DB; ++d) {
        f32x4 o = f32x4{};
#pragma unroll
        for (int s = 0; s < kDecKS / 32; ++s) {
            const uint4 pf = *reinterpret_cast<const uint4*>(&pst[li][32 * s + 8 * lg]);
            o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vf[d][s]),
                                                       __builtin_bit_cast(bf16x8, pf), o, 0, 0, 0);
        }
        if (li < G) {
            float* pr = part + ((int64_t)item * n_q_heads + hk * G + li) * (HD + 4);
            *reinterpret_cast<f32x4*>(pr + 16 * (DB * wave + d) + 4 * lg) = o;
        }
    }
    if (wave == 0 && lg == 0 && li < G) {
        float* pr = part + ((int64_t)item * n_q_heads + hk * G + li) * (HD + 4);
        pr[HD] = m;
        pr[HD + 1] = ((red[1][0][li] + red[1][1][li]) + red[1][2][li]) + red[1][3][li];
    }
}

// Merge the slices of decode prompt i, query head a: M = max m_s, L = sum l_s e^(m_s - M),
// O = sum O_s e^(m_s - M) / L, in slice order; bf16 into the token's output row.  A slice
// record is HD floats of O, then m and l, padded to HD + 4 floats (16-byte aligned).  The
// slices' statistics are fetched in parallel into LDS first (at most kDecMaxSlices).
constexpr int kDecMaxSlices = 64;

template <int HD>
__global__ __launch_bounds__(HD) void attn_decode_combine_kernel(
    const float* __restrict__ part, const int32_t* __restrict__ dfirst,
    const int32_t* __restrict__ dprompt, const int32_t* __restrict__ cu, int n_q_heads,
    uint16_t* __restrict__ out, int64_t ld_out) {
    __shared__ float ms[kDecMaxSlices], ls[kDecMaxSlices];
    const int i = blockIdx.x / n_q_heads, a = blockIdx.x % n_q_heads, e = threadIdx.x;
    const int f0 = dfirst[i], n = dfirst[i + 1] - f0;
    for (int f = e; f < n; f += HD) {
        const float* pr = part + ((int64_t)(f0 + f) * n_q_heads + a) * (HD + 4);
        ms[f] = pr[HD];
        ls[f] = pr[HD + 1];
    }
    __syncthreads();
    float M = -INFINITY;
    for (int f = 0; f < n; ++f) M = fmaxf(M, ms[f]);
    float L = 0.f, o = 0.f;
#pragma unroll 8
    for (int f = 0; f < n; ++f) {
        const float w = expf(ms[f] - M);
        L = fmaf(ls[f], w, L);
        o = fmaf(part[((int64_t)(f0 + f) * n_q_heads + a) * (HD + 4) + e], w, o);
    }
    out[(int64_t)cu[dprompt[i]] * ld_out + (int64_t)a * HD + e] = (uint16_t)f32_to_bf16(o / L);
}

}  // namespace

int attention_q_tile(Act t) { return t == Act::BF16 ? kBQ : kBQ32; }

hipError_t launch_attention(Act t, const void* qkv, int64_t ld_qkv, const void* vt, int64_t ld_vt,
                            const int32_t* vt_off, void* out, int64_t ld_out, const int32_t* cu,
                            const int2* work, int n_items, int n_q_heads, int n_kv_heads,
                            int head_dim, hipStream_t s, const PrefixKV* pf) {
    if (n_items == 0) return hipSuccess;
    const PrefixKV pk = pf ? *pf : PrefixKV();
    if (pf && (!pk.k || !pk.v || !pk.len || !pk.off)) return hipErrorInvalidValue;
    if (t == Act::BF16) {
        const unsigned grid = (unsigned)((n_items + 7) / 8 * 8) * (unsigned)n_q_heads;
        const float sl2 = kLog2e / sqrtf((float)head_dim);
        const uint16_t* q = static_cast<const uint16_t*>(qkv);
        const uint16_t* v = static_cast<const uint16_t*>(vt);
        uint16_t* o = static_cast<uint16_t*>(out);
        // per-lane DMA offsets are 32-bit: V^T rows of one kv head and 64 K rows
        if (!v || !vt_off || ld_vt % 8 || (int64_t)head_dim * ld_vt * 2 > UINT32_MAX ||
            64 * ld_qkv * 2 > UINT32_MAX)
            return hipErrorInvalidValue;
        if (pf && (pk.ld_k % 8 || pk.ld_v % 8 || (int64_t)head_dim * pk.ld_v * 2 > UINT32_MAX ||
                   64 * pk.ld_k * 2 > UINT32_MAX))
            return hipErrorInvalidValue;
#define SURR_ATTN_BF16(HD, PRE)                                                                 \
    attn_bf16_kernel<HD, PRE><<<grid, kThreads, 0, s>>>(q, ld_qkv, v, ld_vt, vt_off, o, ld_out, cu, \
                                                   work, n_items, n_q_heads, n_kv_heads, sl2, pk)
        switch (head_dim) {
            case 64: if (pf) SURR_ATTN_BF16(64, true); else SURR_ATTN_BF16(64, false); break;
            case 128: if (pf) SURR_ATTN_BF16(128, true); else SURR_ATTN_BF16(128, false); break;
            default: return hipErrorInvalidValue;
        }
#undef SURR_ATTN_BF16
    } else {
        const unsigned grid = (unsigned)n_items * (unsigned)n_q_heads;
        const float sc = 1.f / sqrtf((float)head_dim);
        const float* q = static_cast<const float*>(qkv);
        float* o = static_cast<float*>(out);
#define SURR_ATTN_F32(HD, PRE)                                                               \
    attn_f32_kernel<HD, PRE><<<grid, 64, 0, s>>>(q, ld_qkv, o, ld_out, cu, work, n_q_heads, \
                                                 n_kv_heads, sc, pk)
        switch (head_dim) {
            case 32: if (pf) SURR_ATTN_F32(32, true); else SURR_ATTN_F32(32, false); break;
            case 64: if (pf) SURR_ATTN_F32(64, true); else SURR_ATTN_F32(64, false); break;
            case 128: if (pf) SURR_ATTN_F32(128, true); else SURR_ATTN_F32(128, false); break;
            default: return hipErrorInvalidValue;
        }
#undef SURR_ATTN_F32
    }
    return hipGetLastError();
}


int attention_decode_slice() { return kDecKS; }
int attention_decode_max_slices() { return kDecMaxSlices; }

hipError_t launch_attention_decode(const void* qkv, int64_t ld_qkv, const int32_t* cu,
                                   const int2* items, int n_items, const int32_t* dprompt,
                                   const int32_t* dfirst, int n_prompts, int n_q_heads,
                                   int n_kv_heads, int head_dim, const PrefixKV& pk, float* part,
                                   void* out, int64_t ld_out, hipStream_t s) {
    if (n_items == 0) return hipSuccess;
    const int G = n_q_heads / n_kv_heads;
    if (G < 1 || G > kDecMaxG || G * n_kv_heads != n_q_heads || !pk.k || !pk.v || !pk.len ||
        !pk.off || pk.ld_k % 8 || pk.ld_v % 8)
        return hipErrorInvalidValue;
    const float scale = 1.f / sqrtf((float)head_dim);
    const uint16_t* q = static_cast<const uint16_t*>(qkv);
    uint16_t* o = static_cast<uint16_t*>(out);
    const unsigned g1 = (unsigned)n_items * (unsigned)n_kv_heads;
    const unsigned g2 = (unsigned)n_prompts * (unsigned)n_q_heads;
    switch (head_dim) {
        case 64:
            attn_decode_split_kernel<64><<<g1, 256, 0, s>>>(q, ld_qkv, cu, items, dprompt, n_q_heads, n_kv_heads, scale, pk, part);
            attn_decode_combine_kernel<64><<<g2, 64, 0, s>>>(part, dfirst, dprompt, cu, n_q_heads, o, ld_out);
            break;
        case 128:
            attn_decode_split_kernel<128><<<g1, 256, 0, s>>>(q, ld_qkv, cu, items, dprompt, n_q_heads, n_kv_heads, scale, pk, part);
            attn_decode_combine_kernel<128><<<g2, 128, 0, s>>>(part, dfirst, dprompt, cu, n_q_heads, o, ld_out);
            break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace surr
