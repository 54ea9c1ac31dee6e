// Projection GEMMs C = A[M,K] * B[N,K]^T with fused epilogues.
//
// bf16 path: v_mfma_f32_32x32x16_bf16 or v_mfma_f32_16x16x32_bf16 (MF = 32 or 16) on a
// BM x BN workgroup tile of WM x WN wavefront tiles, K in steps of BK.  Both MFMA shapes
// accumulate k in the same order and give bitwise the same sums.  Both operands are
// K-contiguous, so one 16-byte chunk of a row is exactly the 8 consecutive k values an
// MFMA lane supplies; the weight operand B is panel-packed (kernels.h), so the 16 rows one
// wavefront load fetches are one 1 KB run.  Tiles move from HBM straight into LDS with global_load_lds_dwordx4
// (no staging registers) through an NST-stage ring, one barrier per K step; LDS rows hold
// BK/8 chunks whose order is XOR-swizzled by the row to spread the 16-byte reads over the
// banks.  The MFMA is issued with the weight fragment as its A operand and the activation
// fragment as its B operand, so each lane ends up owning one output row m and runs of 4
// consecutive output columns n.
//
// Few-row path (decode steps, last-position rows): gemm_rows_kernel below.
// fp32 path: a plain LDS-tiled FMA kernel for the float32 model.
#include <algorithm>
#include <climits>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace surr {
namespace gemm {

template <int BM, int BN, int BK, int WM, int WN, int NST, int MF = 32>
struct Tile {
    static constexpr int WAVES_N = BN / WN;
    static constexpr int NW = (BM / WM) * (BN / WN);  // wavefronts per workgroup
    static constexpr int THREADS = 64 * NW;
    static_assert(NW == 4 || NW == 8 || NW == 16, "4, 8 or 16 wavefronts per workgroup");
    static constexpr int FM = WM / MF, FN = WN / MF;  // MFMA fragments per wavefront tile
    static constexpr int CH = BK / 8;               // 16-byte chunks per tile row
    static constexpr int A_SLOTS = BM * CH, B_SLOTS = BN * CH;
    static constexpr int STAGE = A_SLOTS + B_SLOTS;  // 16-byte LDS slots per stage
    static constexpr int LOADS = STAGE / THREADS;    // DMA loads per thread per stage
    static_assert(A_SLOTS % 64 == 0 && STAGE % THREADS == 0, "whole wavefront loads");
    static_assert(NST >= 2 && (NST - 2) * LOADS <= 63, "vmcnt range");
};

// Chunk order inside an LDS row: XOR with row bits so that the rows one ds_read_b128
// reads at one logical chunk spread over the 16-byte bank groups.  SWZ = 0 puts 16
// consecutive rows on 16 distinct groups of a 256-byte line; SWZ = 3 ((row / 2) mod CH)
// puts 8 consecutive 64-byte rows on 8 distinct groups of a 128-byte line, which is what
// the fragment reads of 32-column stages want (rows l % 16 or l % 32): rocprofv3 counts
// SQ_LDS_BANK_CONFLICT 1.67e9 -> 2.9e7 cycles per 7B gate/up launch on the 256 x 256
// tiles, which run 3% faster (the 128 x 128 tiles 1%).
template <int CH, int SWZ = 0>
__device__ __forceinline__ int swz(int row) {
    if constexpr (SWZ == 1) return row & (CH - 1);
    if constexpr (SWZ == 3) return (row >> 1) & (CH - 1);
    if constexpr (CH == 8) return (row >> 1) & 7;
    else return (row >> 2) & 3;
}

// silu(g) = g / (1 + e^-g), with the hardware reciprocal (1 ulp) instead of an IEEE
// division (about ten instructions): the result is rounded to bf16 right after.
__device__ __forceinline__ float silu(float g) {
    return g * __builtin_amdgcn_rcpf(1.f + __expf(-g));
}

// Fragment rows staged per epilogue pass: the largest power of two (dividing fm) whose
// rows * pitch bytes fit in the ring.
constexpr int staged_rows_per_pass(int fm, int rows, int pitch, int ring) {
    int pg = fm;
    while (pg > 1 && pg * rows * pitch > ring) pg /= 2;
    return pg;
}

// One MFMA step on a 32x32 (16 fp32 per lane) or 16x16 (4 per lane) accumulator.
__device__ __forceinline__ f32x16 mfma_step(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_step(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Rotate-half RoPE of one value x with its partner y (the value half a head away) and
// the angle's cos c and sin s: first half x c - y s, second half x c + y s.  Written
// with explicit fused operations so every kernel rounds the same way.
__device__ __forceinline__ float rope_rot(float x, float y, float c, float s, bool first_half) {
    return first_half ? fmaf(x, c, -(y * s)) : fmaf(x, c, y * s);
}

// Tile order.  The hardware hands workgroup i to XCD i % 8, and each XCD has its own
// L2.  With XCD remapping, XCD x receives the contiguous virtual range
// [x * per_xcd, (x + 1) * per_xcd); virtual ids then walk GROUP M-tiles down before
// moving one N-tile right, so the ~32 tiles resident on one XCD form a compact
// GROUP x (32 / GROUP) block that shares A and B slabs in that XCD's L2.
template <int GROUP, bool XCD>
__device__ __forceinline__ void tile_coords(int pid, int tiles_m, int tiles_n, int* tm, int* tn) {
    if constexpr (XCD) {
        const int total = tiles_m * tiles_n;
        const int per_xcd = total / 8;
        if (pid < per_xcd * 8) pid = (pid % 8) * per_xcd + pid / 8;
    }
    const int width = GROUP * tiles_n;
    const int first_m = (pid / width) * GROUP;
    const int gsz = min(tiles_m - first_m, GROUP);
    *tm = first_m + (pid % width) % gsz;
    *tn = (pid % width) / gsz;
}

template <int BM, int BN, int BK, int WM, int WN, int NST, Epi EPI, int GROUP = 8, bool XCD = false,
          int SWZ = 0, int MINB = 1, int MF = 32, bool ILV = true>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64, MINB) void gemm_bf16_kernel(const uint16_t* __restrict__ A,
                                                        int64_t lda,
                                                        const uint16_t* __restrict__ B,
                                                        int64_t ldb, void* __restrict__ C,
                                                        int64_t ldc, int M, int N, int K,
                                                        EpiArgs ep) {
    using S = Tile<BM, BN, BK, WM, WN, NST, MF>;
    using Acc = typename std::conditional<MF == 32, f32x16, f32x4>::type;
    // SwiGLU pairs the gate fragment j of a wavefront with its up fragment 32 columns on,
    // so a wavefront's columns must hold whole 64-column gate/up block pairs
    static_assert(EPI != Epi::SwiGLU || WN % 64 == 0, "SwiGLU needs wavefront tiles of whole gate/up pairs");
    __shared__ uint4 lds[NST * S::STAGE];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / S::WAVES_N, wn = wave % S::WAVES_N;

    const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
    int tm, tn;
    tile_coords<GROUP, XCD>(blockIdx.x, tiles_m, tiles_n, &tm, &tn);
    const int m0 = tm * BM, n0 = tn * BN;

    // Direct-to-LDS loads: wavefront `wave`, load j fills the 64 consecutive slots
    // (wave * LOADS + j) * 64 + lane of a stage (the hardware places lane l's 16 bytes at
    // slot base + l), i.e. 16 rows x 4 chunks.  Slot -> (row, physical chunk) -> logical
    // chunk via the swizzle; rows past M or N are clamped (their results are never
    // stored).  B is panel-packed: the 16 rows of a load are 1 KB of consecutive bytes of
    // one block, and a stage k0 further sits k0 * kPanel values on in every panel; a tile
    // may span two panels when b_row0 is not a multiple of BN.  Each load reads either
    // the A tile or the B tile (uniform per wavefront and load), so a thread keeps only a
    // 32-bit byte offset per load against the tile's base pointer.
    static_assert(BK == 32, "panel blocks are 32 columns wide");
    const int64_t nb = (int64_t)ep.b_row0 + n0;  // first weight row of the tile
    const char* a_tile = reinterpret_cast<const char*>(A + (int64_t)m0 * lda);
    const char* b_tile = reinterpret_cast<const char*>(B + (nb / kPanel) * kPanel * K + (nb % kPanel) * 32);
    uint32_t goff[S::LOADS];
    const uint32_t lds_base = lds_offset(lds);
#pragma unroll
    for (int j = 0; j < S::LOADS; ++j) {
        const int slot = (wave * S::LOADS + j) * 64 + lane;
        if (slot < S::A_SLOTS) {
            const int r = slot / S::CH, c = (slot % S::CH) ^ swz<S::CH, SWZ>(r);
            goff[j] = (uint32_t)(((int64_t)(min(m0 + r, M - 1) - m0) * lda + c * 8) * 2);
        } else {
            const int sb = slot - S::A_SLOTS;
            const int r = sb / S::CH, c = (sb % S::CH) ^ swz<S::CH, SWZ>(r);
            const int64_t q = (int64_t)ep.b_row0 + min(n0 + r, N - 1);
            goff[j] = (uint32_t)(((q / kPanel - nb / kPanel) * kPanel * K + (q % kPanel - nb % kPanel) * 32 + c * 8) * 2);
        }
    }
    // Source of load j of this thread for the stage starting at column k0.
#define SURR_DMA_SRC(j, k0)                                                                  \
    ((((wave * S::LOADS + (j)) * 64) < S::A_SLOTS ? a_tile + 2 * (int64_t)(k0)                   \
                                                  : b_tile + 2 * (int64_t)(k0) * kPanel) + goff[j])

    // One stage of direct-to-LDS loads: load j of wavefront `wave` fills the 64 slots
    // starting at (wave * LOADS + j) * 64.
#define SURR_ISSUE_STAGE(stage, k0)                                                              \
    do {                                                                                         \
        _Pragma("unroll") for (int j = 0; j < S::LOADS; ++j)                                     \
            dma_load_16B(SURR_DMA_SRC(j, k0), lds_base + (uint32_t)((((stage) * S::STAGE) +      \
                                                                (wave * S::LOADS + j) * 64) * 16)); \
    } while (0)

    Acc acc[S::FM][S::FN];
#pragma unroll
    for (int i = 0; i < S::FM; ++i)
#pragma unroll
        for (int j = 0; j < S::FN; ++j) acc[i][j] = Acc{};

    // Fragment reads for MFMA step s of the stage at L: lane l supplies row l % MF of the
    // fragment and its 16-byte chunk l / MF of the step's MFMA_K columns.
    constexpr int MFMA_K = MF == 32 ? 16 : 32;
    auto read_a = [&](const uint4* L, int s, bf16x8 (&af)[S::FM]) {
        const int chunk = (MFMA_K / 8) * s + lane / MF;
#pragma unroll
        for (int i = 0; i < S::FM; ++i) {
            const int r = wm * WM + i * MF + lane % MF;
            af[i] = __builtin_bit_cast(bf16x8, L[r * S::CH + (chunk ^ swz<S::CH, SWZ>(r))]);
        }
    };
    auto read_b = [&](const uint4* L, int s, bf16x8 (&bw)[S::FN]) {
        const int chunk = (MFMA_K / 8) * s + lane / MF;
#pragma unroll
        for (int j = 0; j < S::FN; ++j) {
            const int r = wn * WN + j * MF + lane % MF;
            bw[j] = __builtin_bit_cast(bf16x8, L[S::A_SLOTS + r * S::CH + (chunk ^ swz<S::CH, SWZ>(r))]);
        }
    };
    // MFMAs of fragment rows [i0, i1) for the fragments in buffer cb.
#define SURR_MFMA_ROWS(cb, i0, i1)                                                            \
    _Pragma("unroll") for (int mi_ = (i0); mi_ < (i1); ++mi_)                                 \
        _Pragma("unroll") for (int mj_ = 0; mj_ < S::FN; ++mj_)                               \
            acc[mi_][mj_] = mfma_step(fb[cb][mj_], fa[cb][mi_], acc[mi_][mj_])

    // Software pipeline.  Stage ring of NST >= 3 buffers; the fragments of MFMA step s+1
    // are read while the MFMAs of step s run.  The DMA of stage kt+NST-1 is spread between
    // the MFMA rows of the first step of stage kt (its buffer was released by the barrier
    // that opened stage kt), keeping NST-1 stages in flight without stalling MFMA issue.
    // The last step of a stage runs half its MFMA rows, waits for the next stage (vmcnt),
    // passes the barrier and runs the other half, reading the next stage's first fragments
    // between its MFMAs.
    // With one MFMA step per stage (16x16x32 at BK = 32) the refill goes between the rows
    // of that half, and the fragment buffers alternate between stages (the stage loop is
    // unrolled by two).  sched_barrier pins this order.
    constexpr int KSTEPS = BK / MFMA_K;
    constexpr int FH = S::FM / 2;
    static_assert(NST >= 3, "ring of at least three stages");
    static_assert((KSTEPS == 1 || KSTEPS % 2 == 0) && S::FM % 2 == 0, "fragment double buffer");
    const int nk = K / BK;
    // Stage loads past the end of K re-load the last stage (always in bounds) into a
    // buffer that is never read again; this keeps the loop free of branches, which the
    // register allocator needs to keep all accumulators resident.
#pragma unroll
    for (int st = 0; st < NST - 1; ++st) SURR_ISSUE_STAGE(st, min(st, nk - 1) * BK);
    wait_vmcnt<(NST - 2) * S::LOADS>();
    __syncthreads();
    bf16x8 fa[2][S::FM], fb[2][S::FN];
    read_a(lds, 0, fa[0]);
    read_b(lds, 0, fb[0]);
    // Fragment q of MFMA step 0 into buffer nb: B fragments 0..FN-1, then A 0..FM-1.
    auto read_frag = [&](const uint4* L, int q, int nb) {
        const int chunk = lane / MF;
        if (q < S::FN) {
            const int r = wn * WN + q * MF + lane % MF;
            fb[nb][q] = __builtin_bit_cast(bf16x8, L[S::A_SLOTS + r * S::CH + (chunk ^ swz<S::CH, SWZ>(r))]);
        } else {
            const int r = wm * WM + (q - S::FN) * MF + lane % MF;
            fa[nb][q - S::FN] = __builtin_bit_cast(bf16x8, L[r * S::CH + (chunk ^ swz<S::CH, SWZ>(r))]);
        }
    };

    // refill loads [row * LOADS / ROWS, (row + 1) * LOADS / ROWS) after MFMA row `row`
#define SURR_REFILL_AFTER_ROWS(cb, rows_, rs_, rk_)                                                     \
    _Pragma("unroll") for (int row = 0; row < (rows_); ++row) {                                         \
        SURR_MFMA_ROWS(cb, row, row + 1);                                                               \
        __builtin_amdgcn_sched_barrier(0);                                                              \
        _Pragma("unroll") for (int jj = row * S::LOADS / (rows_); jj < (row + 1) * S::LOADS / (rows_); ++jj) \
            dma_load_16B(SURR_DMA_SRC(jj, rk_),                                                         \
                         lds_base + (uint32_t)(((rs_) * S::STAGE + (wave * S::LOADS + jj) * 64) * 16)); \
        __builtin_amdgcn_sched_barrier(0);                                                              \
    }

    auto stage_fn = [&](int kt, auto cb0_c) {
        constexpr int CB0 = decltype(cb0_c)::value;
        const uint4* L = lds + (kt % NST) * S::STAGE;
        const int rs = (kt + NST - 1) % NST, rk = min(kt + NST - 1, nk - 1) * BK;
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) {
            const int cb = (s + CB0) & 1;
            if (s + 1 < KSTEPS) {
                read_b(L, s + 1, fb[cb ^ 1]);
                read_a(L, s + 1, fa[cb ^ 1]);
                __builtin_amdgcn_sched_barrier(0);
                if (s == 0) {
                    SURR_REFILL_AFTER_ROWS(cb, S::FM, rs, rk);
                } else {
                    SURR_MFMA_ROWS(cb, 0, S::FM);
                }
                __builtin_amdgcn_sched_barrier(0);
            } else {
                if (KSTEPS == 1) {
                    SURR_REFILL_AFTER_ROWS(cb, FH, rs, rk);
                } else {
                    SURR_MFMA_ROWS(cb, 0, FH);
                }
                __builtin_amdgcn_sched_barrier(0);
                // every wave's reads of stage kt are done before anyone refills it; then
                // stage kt+1 (issued NST-1 stages ago) must have landed
                __builtin_amdgcn_s_waitcnt((0 << 8) | (7 << 4) | 15 | (3 << 14));  // lgkmcnt(0)
                wait_vmcnt<(NST - 2) * S::LOADS>();
                __syncthreads();
                const uint4* Ln = lds + ((kt + 1) % NST) * S::STAGE;
                if constexpr (ILV && KSTEPS == 1) {
                    // The next stage's fragments (B first, then A in row order) are read
                    // one or two at a time between this half's MFMAs rather than in one
                    // burst right after the barrier, when all eight wavefronts would fill
                    // the LDS command queue at once: 0.8% faster on the gate/up and O
                    // shapes, bitwise the same results.
                    constexpr int NR = S::FM + S::FN, NM = (S::FM - FH) * S::FN;
#pragma unroll
                    for (int t = 0; t < NM; ++t) {
                        const int mi = FH + t / S::FN, mj = t % S::FN;
                        acc[mi][mj] = mfma_step(fb[cb][mj], fa[cb][mi], acc[mi][mj]);
                        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                        for (int q = t * NR / NM; q < (t + 1) * NR / NM; ++q) read_frag(Ln, q, cb ^ 1);
                        __builtin_amdgcn_sched_barrier(0);
                    }
                } else {
                    read_a(Ln, 0, fa[cb ^ 1]);
                    read_b(Ln, 0, fb[cb ^ 1]);
                    __builtin_amdgcn_sched_barrier(0);
                    SURR_MFMA_ROWS(cb, FH, S::FM);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
    };
    if constexpr (KSTEPS % 2 == 0) {
        for (int kt = 0; kt < nk; ++kt) stage_fn(kt, std::integral_constant<int, 0>());
    } else {
        int kt = 0;
        for (; kt + 1 < nk; kt += 2) {
            stage_fn(kt, std::integral_constant<int, 0>());
            stage_fn(kt + 1, std::integral_constant<int, 1>());
        }
        if (kt < nk) stage_fn(kt, std::integral_constant<int, 0>());
    }
#undef SURR_REFILL_AFTER_ROWS
    wait_vmcnt<0>();  // no DMA may still target LDS when the workgroup retires
#undef SURR_MFMA_ROWS

#undef SURR_ISSUE_STAGE
#undef SURR_DMA_SRC

    // Lane owns row m = m0 + wm*WM + MF i + lane % MF and, per fragment j, groups of 4
    // consecutive columns: with MF = 32 the columns j*32 + 8 q + 4 (lane / 32) + {0..3} in
    // acc[i][j][4 q + {0..3}] (q < 4); with MF = 16 the columns j*16 + 4 (lane / 16) + {0..3}
    // in acc[i][j][0..3].
    constexpr int NQ = MF == 32 ? 4 : 1;  // column groups per fragment
    auto gcol = [&](int j, int q) {        // first column (tile-local) of group q of fragment j
        return MF == 32 ? j * 32 + 8 * q + 4 * (lane >> 5) : j * 16 + 4 * (lane >> 4);
    };

    // ---- Staged epilogue.  Stored straight from the accumulators, one wavefront
    // instruction would scatter 8- or 16-byte pieces over 32 rows, and with every CU
    // reaching its epilogue at once those partial-line writes run far below HBM rate.
    // Instead, once the LDS ring is idle, the accumulators are written to LDS in output
    // layout, as many fragment rows (MF rows of every row block) per pass as the ring holds,
    // and the workgroup then stores the pass in 16-byte chunks, each wavefront instruction
    // covering whole row segments (the residual of ResidAddF32 is read the same way).  Few
    // passes mean few barriers: the whole SwiGLU tile goes in one pass, fp32 tiles in four.  The RoPE epilogue stages the fp32 accumulators:
    // a chunk and its rotation partner (half a head away, in the same staged row) are
    // combined at store time, so no wavefront needs to hold whole heads; columns of V
    // heads are stored transposed, walking the staged block column by column so that a
    // wavefront instruction writes 64 consecutive tokens of one row of V^T.
    constexpr bool ROPE = EPI == Epi::StoreActRope;
    constexpr bool LSE = EPI == Epi::LseTile;
    constexpr bool F32OUT = EPI == Epi::StoreF32 || EPI == Epi::ResidAddF32;
    constexpr int SESZ = (F32OUT || ROPE || LSE) ? 4 : 2;      // staged element size
    constexpr int ESZ = F32OUT ? 4 : 2;                        // output element size
    constexpr int OCOLS = EPI == Epi::SwiGLU ? BN / 2 : BN;    // output columns per tile
    constexpr int FROWS = (BM / WM) * MF;                      // rows of one fragment row i
    constexpr int PITCH = OCOLS * SESZ + 16;                   // staged row, bytes
    constexpr int RCH = OCOLS * SESZ / 16;                     // 16-byte chunks per row
    constexpr int PG = staged_rows_per_pass(S::FM, FROWS, PITCH, NST * S::STAGE * 16);
    constexpr int PROWS = PG * FROWS;                          // rows per pass
    static_assert(PROWS * PITCH <= NST * S::STAGE * 16 && S::FM % PG == 0, "staging fits the ring");
    // staged row rr of the pass starting at fragment row i0 -> output row
    auto row_of = [&](int rr, int i0) {
        const int rf = rr % FROWS;
        return m0 + (rf / MF) * WM + (i0 + rr / FROWS) * MF + rf % MF;
    };
    char* stg = reinterpret_cast<char*>(lds);
    const int rl = wm * MF + lane % MF;  // staged row of this lane
    const int ncol0 = EPI == Epi::SwiGLU ? n0 / 2 : n0;
    const int nlim = EPI == Epi::SwiGLU ? N / 2 : N;
    // RoPE tiles: columns [n0, rot_end) are rotated, [rot_end, n_end) are V columns
    const int n_end = min(n0 + BN, N);
    const int rot_end = ROPE ? max(n0, min(n_end, ep.cols)) : n_end;
    const bool vt_cols = ROPE && ep.vt && rot_end < n_end;
    // Residual add: the fp32 tile takes several passes, and a pass's residual loads would
    // each wait a full memory round trip after its barrier.  Instead every thread loads
    // its residual chunks two passes ahead (chunk k of a pass is c = tid + k * THREADS),
    // so those loads overlap the staging and stores of the passes before.
    constexpr bool RESID = EPI == Epi::ResidAddF32;
    constexpr int SWEEP = (PROWS * RCH) / S::THREADS;  // 16-byte chunks per thread and pass
    constexpr int NPASS = S::FM / PG;
    f32x4 res[RESID ? 2 : 1][RESID ? SWEEP : 1];
    auto load_res = [&](int i0, int b) {
#pragma unroll
        for (int k = 0; k < SWEEP; ++k) {
            const int c = tid + k * S::THREADS;
            const int rr = c / RCH, cc = c - rr * RCH;
            const int m = row_of(rr, i0);
            const int n = ncol0 + cc * (16 / ESZ);
            res[b][k] = (m < M && n < nlim)
                            ? *reinterpret_cast<const f32x4*>(static_cast<const float*>(C) + (int64_t)m * ldc + n)
                            : f32x4{};
        }
    };
    if constexpr (RESID) {
        load_res(0, 0);
        if constexpr (NPASS > 1) load_res(PG, 1);
    }
    __syncthreads();  // every wavefront is done with the ring
#pragma unroll
    for (int i0 = 0; i0 < S::FM; i0 += PG) {
#pragma unroll
      for (int i = i0; i < i0 + PG; ++i) {
        char* srow = stg + ((i - i0) * FROWS + rl) * PITCH;
        if constexpr (EPI == Epi::SwiGLU) {
            // gate and up rows of B alternate in 32-row blocks: the gate fragment j pairs
            // with the up fragment 32 columns on (j + 1 for MF = 32, j + 2 for MF = 16)
            constexpr int UP = 32 / MF;
#pragma unroll
            for (int j = 0; j < S::FN; ++j) {
                if ((j / UP) % 2) continue;  // an up fragment
#pragma unroll
                for (int q = 0; q < NQ; ++q) {
                    float v[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        v[e] = silu(acc[i][j][4 * q + e]) * acc[i][j + UP][4 * q + e];
                    const int gc = wn * WN + gcol(j, q);  // tile column of the gate value
                    const int col = (gc / 64) * 32 + gc % 32;
                    *reinterpret_cast<uint2*>(srow + col * 2) =
                        make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < S::FN; ++j)
#pragma unroll
                for (int q = 0; q < NQ; ++q) {
                    const int col = wn * WN + gcol(j, q);
                    if constexpr (SESZ == 4) {
                        *reinterpret_cast<f32x4*>(srow + col * 4) =
                            f32x4{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                  acc[i][j][4 * q + 3]};
                    } else {
                        *reinterpret_cast<uint2*>(srow + col * 2) = make_uint2(
                            pack_bf16x2(acc[i][j][4 * q], acc[i][j][4 * q + 1]),
                            pack_bf16x2(acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]));
                    }
                }
        }
      }
        __syncthreads();
        if constexpr (ROPE) {
            // Rotated q/k columns (and V columns when there is no transposed copy): a
            // thread keeps one 4-column chunk and walks rows RSTEP apart; positions and
            // cos/sin values of all its rows are loaded before any is used.
            static_assert(S::THREADS % RCH == 0 && PROWS % (S::THREADS / RCH) == 0, "chunk walk");
            constexpr int RSTEP = S::THREADS / RCH, NR = PROWS / RSTEP;
            const int hd = ep.head_dim, half = hd >> 1;
            const int lim = vt_cols ? rot_end : n_end;
            const int cc = tid % RCH, r0 = tid / RCH;
            const int n = n0 + cc * 4;
            const int hi = n % hd;  // the 4 columns lie inside one half of a head
            const bool lo = hi < half, rot = n < ep.cols;
            const int poff = (lo ? half : -half) * 4;  // partner chunk, bytes
            const int coff = lo ? hi : hi - half;
            int mr[NR];
            int pr[NR];
#pragma unroll
            for (int k = 0; k < NR; ++k) {
                const int rr = r0 + k * RSTEP;
                mr[k] = row_of(rr, i0);
                pr[k] = rot ? ep.pos[min(mr[k], M - 1)] : 0;
            }
            float4 cs[NR][2];
#pragma unroll
            for (int k = 0; k < NR; ++k) {
                const float4* t = reinterpret_cast<const float4*>(ep.cs + (int64_t)pr[k] * half + coff);
                cs[k][0] = rot ? t[0] : float4{1.f, 0.f, 1.f, 0.f};
                cs[k][1] = rot ? t[1] : float4{1.f, 0.f, 1.f, 0.f};
            }
            if (n < lim) {
#pragma unroll
                for (int k = 0; k < NR; ++k) {
                    const int rr = r0 + k * RSTEP;
                    if (mr[k] >= M) continue;
                    const char* sr = stg + rr * PITCH + cc * 16;
                    const f32x4 x = *reinterpret_cast<const f32x4*>(sr);
                    const f32x4 y = *reinterpret_cast<const f32x4*>(sr + poff);
                    const float c4[4] = {cs[k][0].x, cs[k][0].z, cs[k][1].x, cs[k][1].z};
                    const float s4[4] = {cs[k][0].y, cs[k][0].w, cs[k][1].y, cs[k][1].w};
                    f32x4 r;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        // first half: x1 c - x2 s; second half: x2 c + x1 s (x1 = first-half value)
                        r[e] = rot ? rope_rot(x[e], y[e], c4[e], s4[e], lo) : x[e];
                    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(C) + (int64_t)mr[k] * ldc + n) =
                        make_uint2(pack_bf16x2(r[0], r[1]), pack_bf16x2(r[2], r[3]));
                }
            }
            if (vt_cols) {
                // V columns, transposed: consecutive threads take consecutive tokens of one
                // V dimension, i.e. consecutive columns of one row of V^T
                static_assert(S::THREADS % PROWS == 0, "token walk");
                const int rr = tid % PROWS;
                const int m = row_of(rr, i0);
                if (m < M) {
                    const int64_t vc = ep.vcol[m];
                    for (int n2 = rot_end + tid / PROWS; n2 < n_end; n2 += S::THREADS / PROWS) {
                        const float v = *reinterpret_cast<const float*>(stg + rr * PITCH + (n2 - n0) * 4);
                        ep.vt[(int64_t)(n2 - ep.cols) * ep.ld_vt + vc] = (uint16_t)f32_to_bf16(v);
                    }
                }
            }
        } else if constexpr (LSE) {
            // LM-head read-out: per staged row the tile's max, first argmax and sum of
            // exp(z - max) over its valid columns.  TPR consecutive threads share a row,
            // each walking CPT columns in order; their partials merge by a butterfly (the
            // same sums on both lanes of a pair: addition commutes), so the record does not
            // depend on timing.
            constexpr int TPR = S::THREADS / PROWS, CPT = OCOLS / TPR;
            static_assert(S::THREADS % PROWS == 0 && TPR <= 64 && (TPR & (TPR - 1)) == 0 &&
                              OCOLS % TPR == 0, "row split");
            const HeadArgs& hd = ep.head;
            const int rr = tid / TPR, q = tid % TPR;
            const int m = row_of(rr, i0);
            const float* srow = reinterpret_cast<const float*>(stg + rr * PITCH);
            const int c0 = q * CPT;
            float mx = -INFINITY;
            int am = INT_MAX;
            for (int c = c0; c < c0 + CPT; ++c)
                if (n0 + c < N && srow[c] > mx) {
                    mx = srow[c];
                    am = n0 + c;
                }
            float sum = 0.f;
            if (mx > -INFINITY)
                for (int c = c0; c < c0 + CPT; ++c)
                    if (n0 + c < N) sum += expf(srow[c] - mx);
#pragma unroll
            for (int o = 1; o < TPR; o <<= 1) {
                const float om = __shfl_xor(mx, o, 64), os = __shfl_xor(sum, o, 64);
                const int oa = __shfl_xor(am, o, 64);
                const float nm = fmaxf(mx, om);
                const float a1 = mx > -INFINITY ? sum * expf(mx - nm) : 0.f;
                const float a2 = om > -INFINITY ? os * expf(om - nm) : 0.f;
                am = om > mx ? oa : (mx > om ? am : min(am, oa));
                sum = a1 + a2;
                mx = nm;
            }
            if (q == 0 && m < M)
                hd.part[(int64_t)m * tiles_n + tn] = make_float4(mx, sum, __int_as_float(am), 0.f);
            // the logits at the shared verdict ids and at each row's own target id
            for (int idx = tid; idx < PROWS * kPicked; idx += S::THREADS) {
                const int r2 = idx / kPicked, v = idx - r2 * kPicked;
                const int m2 = row_of(r2, i0);
                if (m2 >= M) continue;
                int col = -1;
                if (v < kMaxVerdicts) {
                    if (v < hd.n_vid) col = hd.vid[v];
                } else if (hd.target) {
                    col = hd.target[m2];
                }
                if (col >= n0 && col < n_end)
                    hd.picked[(int64_t)m2 * kPicked + v] =
                        *reinterpret_cast<const float*>(stg + r2 * PITCH + (col - n0) * 4);
            }
        } else {
            // unrolled: every LDS read of the pass is in flight at once
            static_assert((PROWS * RCH) % S::THREADS == 0, "whole store sweeps");
            const int rb = (i0 / PG) & 1;  // residual buffer of this pass
#pragma unroll
            for (int k = 0; k < SWEEP; ++k) {
                const int c = tid + k * S::THREADS;
                const int rr = c / RCH, cc = c - rr * RCH;
                const int m = row_of(rr, i0);
                const int n = ncol0 + cc * (16 / ESZ);
                if (m >= M || n >= nlim) continue;
                const uint4 v = *reinterpret_cast<const uint4*>(stg + rr * PITCH + cc * 16);
                char* g = static_cast<char*>(C) + ((int64_t)m * ldc + n) * ESZ;
                if constexpr (RESID) {
                    *reinterpret_cast<f32x4*>(g) = res[rb][k] + __builtin_bit_cast(f32x4, v);
                } else {
                    *reinterpret_cast<uint4*>(g) = v;
                }
            }
            if constexpr (RESID) {
                if (i0 + 2 * PG < S::FM) load_res(i0 + 2 * PG, rb);
            }
        }
        __syncthreads();
    }
}



// ---------------------------------------------------------------- few-row GEMM
// C = A[M,K] * B[N,K]^T for M <= 16 MB rows (decode steps, last-position rows).  With so
// few rows the work is reading B once, so each workgroup streams NF 16-row slices of B
// over the whole K through a deep LDS ring of BK-column stages (direct-to-LDS loads; the
// ring holds 128 KB, or all 160 KB of LDS for paired single-slice launches, where that
// measured faster; about half of it B), together with the M rows of A; wavefront w < MB
// multiplies row block w (v_mfma_f32_16x16x32_bf16).  One barrier per stage: with BK = 256
// a stage carries 8 dependent MFMA steps, enough to amortise the barrier and the LDS
// latency (128-column stages halve that and run about half as fast).  Each output still accumulates k in ascending MFMA steps in
// one fp32 accumulator, as in the tiled kernel (whose 32x32x16 steps give bitwise the same
// sums), so a row's result does not depend on how many rows share the call.
// The NF slices of workgroup g: plain epilogues one slice, rows [16 g, 16 g + 16); SwiGLU a
// gate slice and its up slice 32 rows further (gate/up rows interleave in 32-row blocks);
// RoPE a slice of the first half of a head and its partner half a head further, and, past
// the rotated columns, two consecutive slices of V columns.
template <int MB, int NF, Epi EPI, int BK_ = 256, int RING = 8192>
struct RowsCfg {
    static constexpr int BK = BK_, CH = BK / 8;          // 16-byte chunks per row and stage
    static constexpr int ROWS_B = 16 * NF, ROWS_A = 16 * MB;
    static constexpr int STAGE = (ROWS_B + ROWS_A) * CH;  // 16-byte slots per stage
    static constexpr int THREADS = 256;
    static constexpr int LOADS = STAGE / THREADS;
    static constexpr int NST0 = RING / STAGE;
    static constexpr int NST = NST0 > 16 ? 16 : NST0;
    static_assert(CH >= 16, "swizzle with the row's low 4 bits");
    static_assert(STAGE % THREADS == 0 && (ROWS_B * CH) % 64 == 0, "whole wavefront loads");
    static_assert(NST >= 3 && (NST - 2) * LOADS <= 63, "ring depth");
    static_assert(MB <= 4, "one row block per wavefront");
};

template <int NF, Epi EPI>
__device__ __forceinline__ int rows_slice(int g, int f, const EpiArgs& ep) {
    if constexpr (EPI == Epi::SwiGLU) {
        return 64 * (g >> 1) + 16 * (g & 1) + 32 * f;
    } else if constexpr (EPI == Epi::StoreActRope) {
        const int rot_groups = ep.cols / 32;
        if (g < rot_groups) {
            const int half = ep.head_dim >> 1, per_head = half / 16;
            return (g / per_head) * ep.head_dim + 16 * (g % per_head) + half * f;
        }
        return ep.cols + 32 * (g - rot_groups) + 16 * f;
    } else {
        return 16 * (g * NF + f);
    }
}

template <int MB, int NF, Epi EPI, int BK, bool PAIR = false, int RING = 8192>
__global__ __launch_bounds__(256) void gemm_rows_kernel(const uint16_t* __restrict__ A, int64_t lda,
                                                        const uint16_t* __restrict__ B, int64_t ldb,
                                                        void* __restrict__ C, int64_t ldc, int M,
                                                        int N, int K, EpiArgs ep, int groups) {
    using R = RowsCfg<MB, NF, EPI, BK, RING>;
    __shared__ uint4 lds[R::NST * R::STAGE];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int g = blockIdx.x;
    if constexpr (PAIR) {
        // Up to 2 * 16 MB rows: workgroups b and b + 8 take the two row halves of one slice
        // group.  The hardware deals workgroup b to XCD b % 8, so both run on one XCD at
        // about the same time and the second reads the weight slices from its L2.
        const int half = (blockIdx.x >> 3) & 1;
        g = (blockIdx.x & 7) | ((blockIdx.x >> 4) << 3);
        const int r0 = 16 * MB * half;
        if (g >= groups || r0 >= M) return;
        constexpr int esz = (EPI == Epi::StoreF32 || EPI == Epi::ResidAddF32) ? 4 : 2;
        A += (int64_t)r0 * lda;
        C = static_cast<char*>(C) + (int64_t)r0 * ldc * esz;
        M = min(M - r0, 16 * MB);
        if (ep.pos) ep.pos += r0;
        if (ep.vcol) ep.vcol += r0;
    }
    int slice[NF];
#pragma unroll
    for (int f = 0; f < NF; ++f) slice[f] = rows_slice<NF, EPI>(g, f, ep);
    // Load j of this thread fills slot (wave * LOADS + j) * 64 + lane of a stage: slots
    // [0, ROWS_B * CH) hold the B slices, the rest the A rows.  B (panel-packed) is kept
    // block-major in LDS as in HBM: slot (b * ROWS_B + r) * 4 + (c ^ ((r >> 2) & 3)) holds
    // chunk c of the stage's 32-column block b for slice row r, so a load copies one
    // 1 KB run (16 rows of one block) and the 16 rows that one fragment read takes at a
    // chunk hit 16 distinct bank groups.  A rows are row-major, the chunk order inside a
    // row XOR-swizzled with the row's low 4 bits.  Offsets are relative to b_base (the
    // panel of the first slice row) and a_base.
    const int64_t q0 = (int64_t)ep.b_row0 + slice[0];
    const char* b_base = reinterpret_cast<const char*>(B + (q0 / kPanel) * kPanel * K);
    const char* a_base = reinterpret_cast<const char*>(A);
    uint32_t goff[R::LOADS];
#pragma unroll
    for (int j = 0; j < R::LOADS; ++j) {
        const int slot = (wave * R::LOADS + j) * 64 + lane;
        if (slot < R::ROWS_B * R::CH) {
            const int b = slot / (R::ROWS_B * 4), r = (slot / 4) % R::ROWS_B;
            const int c = (slot % 4) ^ ((r >> 2) & 3);
            const int64_t q = (int64_t)ep.b_row0 + min(slice[r >> 4] + (r & 15), N - 1);
            goff[j] = (uint32_t)(((q / kPanel - q0 / kPanel) * kPanel * K + (int64_t)b * kPanel * 32 +
                                  (q % kPanel) * 32 + c * 8) * 2);
        } else {
            const int sa = slot - R::ROWS_B * R::CH;
            const int r = sa / R::CH, c = (sa % R::CH) ^ (r & 15);
            goff[j] = (uint32_t)(((int64_t)min(r, M - 1) * lda + c * 8) * 2);
        }
    }
    const uint32_t lds_base = lds_offset(lds);
    auto issue = [&](int stage, int k0) {
#pragma unroll
        for (int j = 0; j < R::LOADS; ++j) {
            const bool is_b = (wave * R::LOADS + j) * 64 < R::ROWS_B * R::CH;
            dma_load_16B((is_b ? b_base + 2 * (int64_t)k0 * kPanel : a_base + 2 * (int64_t)k0) + goff[j],
                         lds_base + (uint32_t)((stage * R::STAGE + (wave * R::LOADS + j) * 64) * 16));
        }
    };
    const int nk = K / R::BK;
#pragma unroll
    for (int st = 0; st < R::NST - 1; ++st) issue(st, min(st, nk - 1) * R::BK);
    f32x4 acc[NF];
#pragma unroll
    for (int f = 0; f < NF; ++f) acc[f] = f32x4{};
    const int rb = lane & 15, ck = lane >> 4;
    for (int kt = 0; kt < nk; ++kt) {
        wait_vmcnt<(R::NST - 2) * R::LOADS>();  // this thread's part of stage kt landed
        __syncthreads();                         // everyone's part; stage kt-1 fully read
        issue((kt + R::NST - 1) % R::NST, min(kt + R::NST - 1, nk - 1) * R::BK);
        if (wave < MB) {
            const uint4* L = lds + (kt % R::NST) * R::STAGE;
#pragma unroll
            for (int s = 0; s < R::BK / 32; ++s) {
                const int c = 4 * s + ck;
                bf16x8 fw[NF];
#pragma unroll
                for (int f = 0; f < NF; ++f) {
                    const int r = 16 * f + rb;
                    fw[f] = __builtin_bit_cast(bf16x8, L[(s * R::ROWS_B + r) * 4 + (ck ^ ((r >> 2) & 3))]);
                }
                const int ra = 16 * wave + rb;
                const bf16x8 fx = __builtin_bit_cast(bf16x8, L[R::ROWS_B * R::CH + ra * R::CH + (c ^ (ra & 15))]);
#pragma unroll
                for (int f = 0; f < NF; ++f)
                    acc[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[f], fx, acc[f], 0, 0, 0);
            }
        }
    }
    wait_vmcnt<0>();  // no DMA may still target LDS when the workgroup retires
    if (wave >= MB) return;

    // Lane owns row m = 16 wave + (lane & 15) and, per slice f, columns
    // slice[f] + 4 (lane >> 4) + {0..3} in acc[f][0..3].
    const int m = 16 * wave + rb;
    if (m >= M) return;
    if constexpr (EPI == Epi::SwiGLU) {
        const int col = 32 * (g >> 1) + 16 * (g & 1) + 4 * ck;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = silu(acc[0][e]) * acc[1][e];
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(C) + (int64_t)m * ldc + col) =
            make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
    } else if constexpr (EPI == Epi::StoreActRope) {
        if (slice[0] < ep.cols) {
            const int hd = ep.head_dim, half = hd >> 1;
            const int i0 = slice[0] % hd + 4 * ck;  // first-half index of this lane's 4 columns
            const float4* t = reinterpret_cast<const float4*>(ep.cs + (int64_t)ep.pos[m] * half + i0);
            const float4 t0 = t[0], t1 = t[1];
            const float c4[4] = {t0.x, t0.z, t1.x, t1.z};
            const float s4[4] = {t0.y, t0.w, t1.y, t1.w};
            float v[4], w[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[e] = rope_rot(acc[0][e], acc[1][e], c4[e], s4[e], true);
                w[e] = rope_rot(acc[1][e], acc[0][e], c4[e], s4[e], false);
            }
            uint16_t* out = static_cast<uint16_t*>(C) + (int64_t)m * ldc;
            *reinterpret_cast<uint2*>(out + slice[0] + 4 * ck) =
                make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
            *reinterpret_cast<uint2*>(out + slice[1] + 4 * ck) =
                make_uint2(pack_bf16x2(w[0], w[1]), pack_bf16x2(w[2], w[3]));
        } else {
#pragma unroll
            for (int f = 0; f < NF; ++f) {
                const int n = slice[f] + 4 * ck;
                if (ep.vt) {
                    const int64_t vc = ep.vcol[m];
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        ep.vt[(int64_t)(n + e - ep.cols) * ep.ld_vt + vc] = (uint16_t)f32_to_bf16(acc[f][e]);
                } else {
                    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(C) + (int64_t)m * ldc + n) =
                        make_uint2(pack_bf16x2(acc[f][0], acc[f][1]), pack_bf16x2(acc[f][2], acc[f][3]));
                }
            }
        }
    } else {
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const int n = slice[f] + 4 * ck;
            if (n >= N) continue;
            if constexpr (EPI == Epi::StoreAct) {
                *reinterpret_cast<uint2*>(static_cast<uint16_t*>(C) + (int64_t)m * ldc + n) =
                    make_uint2(pack_bf16x2(acc[f][0], acc[f][1]), pack_bf16x2(acc[f][2], acc[f][3]));
            } else if constexpr (EPI == Epi::StoreF32) {
                *reinterpret_cast<f32x4*>(static_cast<float*>(C) + (int64_t)m * ldc + n) = acc[f];
            } else {
                f32x4* p = reinterpret_cast<f32x4*>(static_cast<float*>(C) + (int64_t)m * ldc + n);
                *p = *p + acc[f];
            }
        }
    }
}

#ifndef SURR_GEMM_KERNELS_ONLY  // (kernel-only builds for standalone tuning harnesses)
template <int BM, int BN, int BK, int WM, int WN, int NST, Epi EPI, int MF = 32, int SWZ = 0,
          int GROUP = 8>
hipError_t run_bf16(const void* A, int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc,
                    int M, int N, int K, hipStream_t s, const EpiArgs& ep) {
    const int64_t tiles = (int64_t)((M + BM - 1) / BM) * ((N + BN - 1) / BN);
    gemm_bf16_kernel<BM, BN, BK, WM, WN, NST, EPI, GROUP, true, SWZ, 1, MF>
        <<<(unsigned)tiles, Tile<BM, BN, BK, WM, WN, NST, MF>::THREADS, 0, s>>>(
        static_cast<const uint16_t*>(A), lda, static_cast<const uint16_t*>(B), ldb, C, ldc, M, N, K,
        ep);
    return hipGetLastError();
}

template <int MB, Epi EPI, bool PAIR = false>
hipError_t run_rows(const void* A, int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc,
                    int M, int N, int K, hipStream_t s, const EpiArgs& ep) {
    constexpr int NF = (EPI == Epi::SwiGLU || EPI == Epi::StoreActRope) ? 2 : 1;
    const int groups = N / (16 * NF);
    const unsigned grid = PAIR ? (unsigned)(16 * ((groups + 7) / 8)) : (unsigned)groups;
    const uint16_t* a = static_cast<const uint16_t*>(A);
    const uint16_t* b = static_cast<const uint16_t*>(B);
    constexpr int RING = PAIR && NF == 1 ? 10240 : 8192;  // 16-byte slots: 160 KB or 128 KB
    if constexpr (MB <= 2 && !PAIR) {
        // Many slice groups (wide weights: gate/up, LM heads): a 64 KB ring of 128-column
        // stages, so two workgroups share a CU and the last round of workgroups is short
        // (measured at 8 rows: 7B gate/up 50 -> 41 us, a 36,864-row head 58 -> 42 us).
        // Narrow weights (< 256 groups) lose with it and keep the deep ring.
        if (groups >= 512) {
            gemm_rows_kernel<MB, NF, EPI, 128, false, 4096><<<grid, RowsCfg<MB, NF, EPI, 128, 4096>::THREADS, 0, s>>>(
                a, lda, b, ldb, C, ldc, M, N, K, ep, groups);
            return hipGetLastError();
        }
    }
    if constexpr (MB + NF <= 4) {  // 256-column stages while the ring keeps >= 4 of them
        if (K % 256 == 0) {
            gemm_rows_kernel<MB, NF, EPI, 256, PAIR, RING><<<grid, RowsCfg<MB, NF, EPI, 256, RING>::THREADS, 0, s>>>(
                a, lda, b, ldb, C, ldc, M, N, K, ep, groups);
            return hipGetLastError();
        }
    }
    gemm_rows_kernel<MB, NF, EPI, 128, PAIR, RING><<<grid, RowsCfg<MB, NF, EPI, 128, RING>::THREADS, 0, s>>>(
        a, lda, b, ldb, C, ldc, M, N, K, ep, groups);
    return hipGetLastError();
}

// Tile choice (measured on the 7B projection shapes): 256 x 256 x 32 tiles, eight
// wavefronts of 128 x 64 (two per SIMD, so one hides the other's waits) on 16x16x32
// MFMAs (1-2 points above 32x32x16), a 4-stage ring and XCD-grouped order; up to 64 rows (decode steps, last-position rows) the few-row
// kernel, up to 128 rows the few-row kernel on two 64-row halves unless B is wide enough
// to keep the chip busy with 128 x 128 tiles (at 128 rows of the 7B gate/up projection,
// N = 37,888: 92 us on tiles against 132 us on the few-row kernel).
template <Epi EPI>
hipError_t dispatch_bf16(const void* A, int64_t lda, const void* B, int64_t ldb, void* C,
                         int64_t ldc, int M, int N, int K, hipStream_t s, const EpiArgs& ep) {
    // the few-row kernel needs whole 32-row slice pairs and K in 128-column stages; RoPE
    // slices pair whole half-heads, so the rotated width and V width split into 32-row groups
    const bool rows_ok = N % 32 == 0 && K % 128 == 0 &&
                         (EPI != Epi::StoreActRope || (ep.cols % 32 == 0 && (ep.head_dim >> 1) % 16 == 0));
    if (M <= 64 && rows_ok) {
        if (M <= 16) return run_rows<1, EPI>(A, lda, B, ldb, C, ldc, M, N, K, s, ep);
        if (M <= 32) return run_rows<2, EPI>(A, lda, B, ldb, C, ldc, M, N, K, s, ep);
        return run_rows<4, EPI>(A, lda, B, ldb, C, ldc, M, N, K, s, ep);
    }
    // 65..128 rows against a narrow B: 128 x 128 tiles would leave most CUs idle (N / 128
    // workgroups), so the few-row kernel takes the rows in two 64-row halves, paired on
    // one XCD so each weight slice comes from HBM once.  From N = 32768 (256 tiles, a
    // workgroup per CU) the tiles are faster.
    if (M <= 128 && N < 32768 && rows_ok)
        return run_rows<4, EPI, true>(A, lda, B, ldb, C, ldc, M, N, K, s, ep);
    if (M <= 128)
        return run_bf16<128, 128, 32, 64, 64, 4, EPI, 32, 3>(A, lda, B, ldb, C, ldc, M, N, K, s, ep);
    // Tile group height (M-tiles per column of the XCD-local block, see tile_coords).  The
    // tiles that finish together store their outputs together: the fewer M-tiles a group
    // spans, the longer the row segments of that store.  Narrow outputs gain from short
    // groups, most of all the fp32 read-modify-write of the residual add (7B O projection
    // at 262,144 rows: 6.7 ms with groups of 8, 6.0 ms with 2; down 2% faster), while the
    // wide gate/up projection is fastest with 8.
    if constexpr (EPI == Epi::ResidAddF32)
        return run_bf16<256, 256, 32, 128, 64, 4, EPI, 16, 3, 2>(A, lda, B, ldb, C, ldc, M, N, K, s, ep);
    if (N <= 8192)
        return run_bf16<256, 256, 32, 128, 64, 4, EPI, 16, 3, 4>(A, lda, B, ldb, C, ldc, M, N, K, s, ep);
    return run_bf16<256, 256, 32, 128, 64, 4, EPI, 16, 3, 8>(A, lda, B, ldb, C, ldc, M, N, K, s, ep);
}

#endif  // SURR_GEMM_KERNELS_ONLY

// ---------------------------------------------------------------- fp32 FMA GEMM
template <Epi EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A, int64_t lda,
                                                       const float* __restrict__ B, int64_t ldb,
                                                       float* __restrict__ C, int64_t ldc, int M,
                                                       int N, int K) {
    __shared__ float As[16][68];
    __shared__ float Bs[16][68];
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int idx = tid + 256 * e, r = idx >> 4, kk = idx & 15;
            As[kk][r] = A[(int64_t)min(m0 + r, M - 1) * lda + k0 + kk];
            Bs[kk][r] = B[(int64_t)min(n0 + r, N - 1) * ldb + k0 + kk];
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < 16; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
    const int n = n0 + tx * 4;
    if (n >= N) return;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = m0 + ty * 4 + i;
        if (m >= M) continue;
        float* p = C + (int64_t)m * ldc + n;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (EPI == Epi::ResidAddF32) p[j] += acc[i][j];
            else p[j] = acc[i][j];
        }
    }
}

template <Epi EPI>
hipError_t run_f32(const void* A, int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc,
                   int M, int N, int K, hipStream_t s) {
    dim3 grid((unsigned)((N + 63) / 64), (unsigned)((M + 63) / 64));
    gemm_f32_kernel<EPI><<<grid, 256, 0, s>>>(static_cast<const float*>(A), lda,
                                               static_cast<const float*>(B), ldb,
                                               static_cast<float*>(C), ldc, M, N, K);
    return hipGetLastError();
}

}  // namespace gemm

#ifndef SURR_GEMM_KERNELS_ONLY
using namespace gemm;

// One 16-byte chunk (8 values) of the packed matrix per thread.
__global__ __launch_bounds__(256) void pack_panels_kernel(const uint4* __restrict__ src, int64_t rows,
                                                          int64_t K, uint4* __restrict__ dst,
                                                          int64_t chunks) {
    const int64_t per_panel = (int64_t)kPanel * K / 8;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < chunks;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t p = i / per_panel, rem = i % per_panel;
        const int64_t blk = rem / (kPanel * 4), r = (rem / 4) % kPanel, c = rem % 4;
        const int64_t n = p * kPanel + r;
        dst[i] = n < rows ? src[(n * K + blk * 32 + c * 8) / 8] : make_uint4(0, 0, 0, 0);
    }
}

hipError_t launch_pack_panels(const uint16_t* src, int64_t rows, int64_t K, uint16_t* dst,
                              hipStream_t s) {
    if (rows <= 0 || K <= 0 || K % 32) return hipErrorInvalidValue;
    const int64_t chunks = packed_rows(rows) * K / 8;
    const int64_t blocks = std::min<int64_t>((chunks + 255) / 256, 65536);
    pack_panels_kernel<<<(unsigned)blocks, 256, 0, s>>>(reinterpret_cast<const uint4*>(src), rows, K,
                                                        reinterpret_cast<uint4*>(dst), chunks);
    return hipGetLastError();
}

hipError_t launch_gemm(Act t, Epi e, const void* A, int64_t lda, const void* B, int64_t ldb,
                       void* C, int64_t ldc, int M, int N, int K, hipStream_t s,
                       const EpiArgs& ep) {
    if (M <= 0 || N <= 0) return hipSuccess;
    if (t == Act::F32) {
        switch (e) {
            case Epi::ResidAddF32: return run_f32<Epi::ResidAddF32>(A, lda, B, ldb, C, ldc, M, N, K, s);
            case Epi::StoreAct:
            case Epi::StoreF32: return run_f32<Epi::StoreF32>(A, lda, B, ldb, C, ldc, M, N, K, s);
            default: return hipErrorInvalidValue;  // fp32 SwiGLU runs as its own kernel
        }
    }
    switch (e) {
        case Epi::StoreAct: return dispatch_bf16<Epi::StoreAct>(A, lda, B, ldb, C, ldc, M, N, K, s, ep);
        case Epi::ResidAddF32: return dispatch_bf16<Epi::ResidAddF32>(A, lda, B, ldb, C, ldc, M, N, K, s, ep);
        case Epi::SwiGLU: return dispatch_bf16<Epi::SwiGLU>(A, lda, B, ldb, C, ldc, M, N, K, s, ep);
        case Epi::StoreF32: return dispatch_bf16<Epi::StoreF32>(A, lda, B, ldb, C, ldc, M, N, K, s, ep);
        case Epi::StoreActRope:
            if (ep.head_dim != 64 && ep.head_dim != 128) return hipErrorInvalidValue;
            return dispatch_bf16<Epi::StoreActRope>(A, lda, B, ldb, C, ldc, M, N, K, s, ep);
        case Epi::LseTile:
            // records of 128-column tiles for any number of rows (reading the head's weights
            // once per 128 rows; at 128 rows and more it is the fastest shape measured)
            if (!ep.head.part || !ep.head.picked || ep.head.n_vid < 0 || ep.head.n_vid > kMaxVerdicts)
                return hipErrorInvalidValue;
            return run_bf16<128, 128, 32, 64, 64, 4, Epi::LseTile, 32, 3>(A, lda, B, ldb, C, ldc, M, N, K, s, ep);
    }
    return hipErrorInvalidValue;
}

#endif  // SURR_GEMM_KERNELS_ONLY

}  // namespace surr
