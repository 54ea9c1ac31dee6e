// Host-side launchers of the gfx950 kernels (one translation unit per kernel family).
// Every launcher enqueues on `stream` and returns the hipError_t of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace surr {

enum class Act { F32, BF16 };  // storage type of activations and matrices

// ---- k_elementwise.hip
// Gather embedding rows of the packed tokens into the fp32 residual x[T, d] and
// record each token's position: its index j inside its prompt, plus pos_off[b] when
// pos_off is set (tokens that continue a cached prefix).  cu[B+1] are prompt offsets.
// With vt_off (per-prompt first column of the transposed V copy), vcol[t] receives the
// token's column there: vt_off[b] + vt_key_order(j).
hipError_t launch_embed(Act wt, const int32_t* tokens, int64_t row_stride, const int32_t* cu,
                        int B, int64_t T, const void* embed, int d, int vocab, float* x,
                        int32_t* pos, const int32_t* pos_off, const int32_t* vt_off, int32_t* vcol,
                        int32_t* err_flag, hipStream_t s);

// Copy columns [col0, col0 + cols) of the packed rows of B prompts into a cache of
// 64-row-aligned blocks: row j of prompt b goes to row po[b] + j; rows po[b] + L_b up to
// the next block are zeroed (rows = po[B]).
hipError_t launch_capture_rows(const void* src, int64_t ld_src, int col0, int cols, int elem_bytes,
                               const int32_t* cu, const int32_t* po, int B, int64_t rows,
                               void* dst, int64_t ld_dst, hipStream_t s);

// Zero the padding columns of the transposed V copy (rows x [vt_off[b] + L_b,
// vt_off[b + 1]) in stored order) so masked keys multiply finite values.
hipError_t launch_vt_pad_zero(uint16_t* vt, int64_t ld_vt, int rows, const int32_t* cu,
                              const int32_t* vt_off, int B, hipStream_t s);

// y[r] = x[rows ? rows[r] : r] * rsqrt(mean(x^2) + eps) * g, stored as `out` type.
hipError_t launch_rmsnorm(Act out, const float* x, int64_t ldx, const int32_t* rows,
                          int64_t n_rows, const float* g, int d, float eps, void* y, int64_t ldy,
                          hipStream_t s);

// In-place rotate-half RoPE on the first n_heads heads of each row of qkv.
hipError_t launch_rope(Act t, void* qkv, int64_t ld, int64_t T, const int32_t* pos, int n_heads,
                       int head_dim, const float2* cs, hipStream_t s);

// u[t, j] = silu(gu[t, gate(j)]) * gu[t, up(j)] with gate/up interleaved in 32-column
// blocks (fp32 path; the bf16 path fuses this into the GEMM epilogue).
hipError_t launch_swiglu_f32(const float* gu, float* u, int64_t T, int d_ff, hipStream_t s);

// Copy rows rows[r] of src into dst row r (elem_bytes per element).
hipError_t launch_gather_rows(const void* src, int64_t ld_src, const int32_t* rows, int64_t n,
                              int cols, int elem_bytes, void* dst, int64_t ld_dst, hipStream_t s);
// dst[rows[r], :] = src[r, :] for r < n (the inverse of launch_gather_rows; the same
// 4-byte-multiple width rule).
hipError_t launch_scatter_rows(const void* src, int64_t ld_src, const int32_t* rows, int64_t n,
                               int cols, int elem_bytes, void* dst, int64_t ld_dst, hipStream_t s);

// Per prompt b: full-vocab log-softmax of logits[b] at the verdict ids, then the
// renormalised verdict distribution, its max and first argmax.
hipError_t launch_lse_verdict(const float* logits, int64_t ld, int B, int V, const int32_t* vid,
                              int nv, float* lp, float* probs, float* conf, int32_t* verdict,
                              hipStream_t s);

// Sequence caches: the packed tokens (prompt b's token j at row cu[b] + j) continue their
// sequences at positions len[b] + j.  append_rows copies columns [col0, col0 + cols) of
// each row to cache row off[b] + len[b] + j; append_vt copies the transposed V columns
// vt_off[b] + vt_key_order(j) to cache columns off[b] + vt_key_order(len[b] + j) for the
// `rows` rows of V^T (max_len: the longest prompt).
hipError_t launch_append_rows(const void* src, int64_t ld_src, int col0, int cols, int elem_bytes,
                              int64_t T, const int32_t* cu, int B, const int32_t* off,
                              const int32_t* len, void* dst, int64_t ld_dst, hipStream_t s);
hipError_t launch_append_vt(const uint16_t* vt, int64_t ld_vt, const int32_t* vt_off,
                            const int32_t* cu, int B, int max_len, const int32_t* off,
                            const int32_t* len, int rows, uint16_t* cvt, int64_t ld_c,
                            hipStream_t s);
// Both of a bf16 layer's appends in one launch: the K columns [col0, col0 + cols) of the
// qkv rows as append_rows (bf16 elements; ld_qkv, col0, cols and ld_ck even) and the
// `rows` rows of V^T as append_vt.
hipError_t launch_append_kv(const uint16_t* qkv, int64_t ld_qkv, int col0, int cols, int64_t T,
                            const uint16_t* vt, int64_t ld_vt, const int32_t* vt_off,
                            const int32_t* cu, int B, int max_len, const int32_t* off,
                            const int32_t* len, uint16_t* ck, int64_t ld_ck, int rows,
                            uint16_t* cvt, int64_t ld_c, hipStream_t s);

// Merge the per-tile records of an Epi::LseTile head (n_tiles per row, in tile order) into
// each row's full-vocabulary log-sum-exp, then, as launch_lse_verdict, the verdict
// log-probs, their renormalised distribution, its max and first argmax (when nv > 0), and,
// as launch_lse_next, the first argmax over the vocabulary and the log-prob at the row's
// target id (each output optional).
hipError_t launch_lse_combine(const float4* part, int n_tiles, const float* picked, int B, int nv,
                              float* lp, float* probs, float* conf, int32_t* verdict,
                              int32_t* next_token, float* target_lp, hipStream_t s);

// Per row of logits: the first argmax over the vocabulary (next_token, optional) and the
// full-vocabulary log-softmax at target[b] (target_lp, optional).
hipError_t launch_lse_next(const float* logits, int64_t ld, int B, int V, const int32_t* target,
                           int32_t* next_token, float* target_lp, hipStream_t s);

// Selection and ordered compaction in one workgroup, 1 <= n <= 65536.  mode 0: defer
// !(q >= tau); mode 1: defer the k lowest (NaN first); mode 2: defer the k highest (NaN
// last); ties by ascending index.
hipError_t launch_select(const float* conf, int n, int mode, float tau, int k, int32_t* defer_idx,
                         int32_t* accept_idx, int32_t* counts, hipStream_t s);

// ---- k_forecast.hip
constexpr int kMaxBins = 16, kMaxCutoffs = 8;

// Per-bin weights of the forecast head: w[b][0] = representative speedup m_b,
// w[b][1 + c] = share of bin b's mass at or above cutoff c.
struct BinWeights {
    float w[kMaxBins][1 + kMaxCutoffs];
};

// speedup[i] = sum_b probs[i, b] w[b][0] and disc[i, c] = sum_b probs[i, b] w[b][1 + c]
// (either output may be null), probs row-major [n, n_bins].
hipError_t launch_forecast_head(const float* probs, int64_t n, int n_bins, const BinWeights& w,
                                int n_cutoffs, float* speedup, float* disc, hipStream_t s);

// ---- k_evaluate.hip
// Bin edges (float64, compared against float32 speedups) and representatives of the
// forecast bins.
struct EvalBins {
    double edge[kMaxBins - 1];
    float value[kMaxBins];
};

// Per candidate: measured bin, Brier, CRPS (outputs optional), plus per-workgroup partial
// sums in `partial` (eval_partial_bytes(n, n_budgets) bytes).  Then eval_finalize, after
// the top-score selection of every budget into lists + 2 n c (counts[2 c] entries), writes
// summary[0..6] = accuracy, mean Brier, mean CRPS, mean r_corr + 1 - Brier, mean
// r_corr + 1 - CRPS, ECE (10 buckets), forecast error; summary[8 + c] = 100 * max speedup
// over budget c's list / max speedup and summary[7] their mean.  2 <= n_bins <= 16.
size_t eval_partial_bytes(int n, int n_budgets);
hipError_t launch_eval_metrics(const float* probs, const float* speedup, int n, int n_bins,
                               const EvalBins& bins, int32_t* bin_out, float* brier_out,
                               float* crps_out, double* partial, hipStream_t s);
hipError_t launch_eval_finalize(const float* speedup, int n, const int32_t* lists,
                                const int32_t* counts, int n_budgets, double* partial,
                                double* summary, hipStream_t s);

// ---- k_gemm.hip
enum class Epi { StoreAct, ResidAddF32, SwiGLU, StoreF32, StoreActRope, LseTile };

// Full-vocabulary read-out of an LM head inside the GEMM epilogue (Epi::LseTile): the
// logits never leave the workgroup.  For output row m and column tile t (BN columns) the
// epilogue writes part[m * n_tiles + t] = (max, sum of exp(z - max), first argmax as int
// bits, 0) over the tile's valid columns, and copies the logits it holds at the shared
// ids vid[0 .. n_vid) to picked[m * kPicked + v] and at the row's own id target[m] to
// picked[m * kPicked + kMaxVerdicts].  launch_lse_combine merges the tiles.
constexpr int kMaxVerdicts = 16, kPicked = kMaxVerdicts + 1;
struct HeadArgs {
    const int32_t* vid = nullptr;     // [n_vid], shared by every row
    int n_vid = 0;
    const int32_t* target = nullptr;  // [M] or null
    float4* part = nullptr;           // [M][n_tiles]
    float* picked = nullptr;          // [M][kPicked]
};

// Extra arguments of the fused epilogues.
// RoPE (Epi::StoreActRope): columns [0, cols) hold whole heads of head_dim; within each
// head, columns i and i + hd/2 of row m rotate by the angle of position pos[m] (table
// cs[pos][i] = (cos, sin)).  With vt set, columns [cols, N) (the V heads) go transposed to
// vt[n - cols][vcol[m]] instead of C.
struct EpiArgs {
    const int32_t* pos = nullptr;
    const float2* cs = nullptr;
    int cols = 0;
    int head_dim = 0;
    uint16_t* vt = nullptr;
    int64_t ld_vt = 0;
    const int32_t* vcol = nullptr;
    HeadArgs head;
    int b_row0 = 0;  // bf16: first row of B inside its packed matrix (a multiple of 16)
};

// Layout of every bf16 weight matrix W [N, K] (K a multiple of 32), written once at load
// time: panels of kPanel rows, each panel K / 32 consecutive blocks of kPanel x 32 values
// (row-major inside a block); rows past N are zero.  Element (n, k) sits at
//   (n / kPanel) * kPanel * K + (k / 32) * kPanel * 32 + (n % kPanel) * 32 + k % 32.
// Sixteen consecutive rows of one 32-column block are 1 KB of consecutive bytes, which is
// what one wavefront's direct-to-LDS load reads.
constexpr int kPanel = 256;
inline int64_t packed_rows(int64_t n) { return (n + kPanel - 1) / kPanel * kPanel; }
// dst [packed_rows(rows) * K] <- src [rows][K] (row-major, K-contiguous)
hipError_t launch_pack_panels(const uint16_t* src, int64_t rows, int64_t K, uint16_t* dst,
                              hipStream_t s);

// C = A[M,K] * B[N,K]^T, fp32 accumulation, fused epilogue.  A is row-major (lda); for
// fp32 models B is row-major too (ldb), for bf16 models B is a panel-packed weight matrix
// (above) whose rows [rope.b_row0, rope.b_row0 + N) are the operand (ldb unused).
// Epilogues:
//   StoreAct    C (activation type) [M, N]
//   ResidAddF32 C (fp32) += result
//   SwiGLU      B rows interleave gate/up in 32-row blocks; C[M, N/2] = silu(g) * u
//   StoreF32    C (fp32) [M, N]
//   StoreActRope  as StoreAct, with RoPE applied first (bf16 only)
//   LseTile     per-tile head records (HeadArgs), no C (bf16 only; 128 x 128 tiles)
hipError_t launch_gemm(Act t, Epi e, const void* A, int64_t lda, const void* B, int64_t ldb,
                       void* C, int64_t ldc, int M, int N, int K, hipStream_t s,
                       const EpiArgs& rope = EpiArgs());

// ---- k_attention.hip
// Keys and values of shared prompt prefixes, computed once and attended by every prompt
// that continues one.  Per layer, prefix g owns rows [off, off + roundup(len, 64)) of k
// (keys after RoPE, [rows][ld_k], kv heads side by side) and the same range of v: bf16
// keeps V transposed like the vt copy ([kv head * hd + dim][ld_v] columns, 16-key groups
// in vt_key_order), fp32 keeps V rows [rows][ld_v].  Padding rows and columns are zero.
// len[b] / off[b] give prompt b's prefix length (0: none) and its first row.
struct PrefixKV {
    const void* k = nullptr;
    int64_t ld_k = 0;
    const void* v = nullptr;
    int64_t ld_v = 0;
    const int32_t* len = nullptr;
    const int32_t* off = nullptr;
};

// Causal GQA attention over the packed qkv rows.  work[i] = (prompt, q_tile) items;
// grid = n_items * n_q_heads.  q_tile covers rows [q_tile * attention_q_tile, +tile) of
// the prompt.  bf16 reads V from the transposed copy vt (see EpiArgs; ld_vt % 8 == 0,
// vt_off[b] % 64 == 0); the fp32 kernel reads V from qkv and ignores vt.  With a prefix
// (pf != nullptr), every query of prompt b also attends, before its own keys, all
// pf->len[b] keys of its cached prefix.
hipError_t launch_attention(Act t, const void* qkv, int64_t ld_qkv, const void* vt, int64_t ld_vt,
                            const int32_t* vt_off, void* out, int64_t ld_out, const int32_t* cu,
                            const int2* work, int n_items, int n_q_heads, int n_kv_heads,
                            int head_dim, hipStream_t s, const PrefixKV* pf = nullptr);
int attention_q_tile(Act t);

// One-token continuations of cached sequences (bf16): for decode prompt i = items[n].x
// (prompt dprompt[i], whose only row is cu[b] and whose entry holds pk.len[b] + 1 keys
// once this layer's key is appended), slice items[n].y covers keys
// [y * attention_decode_slice(), +slice).  Items of prompt i are dfirst[i] .. dfirst[i+1]-1.
// part holds n_items * n_q_heads * (head_dim + 4) floats; the merged rows go to out.
int attention_decode_slice();
int attention_decode_max_slices();  // per prompt
hipError_t launch_attention_decode(const void* qkv, int64_t ld_qkv, const int32_t* cu,
                                   const int2* items, int n_items, const int32_t* dprompt,
                                   const int32_t* dfirst, int n_prompts, int n_q_heads,
                                   int n_kv_heads, int head_dim, const PrefixKV& pk, float* part,
                                   void* out, int64_t ld_out, hipStream_t s);

}  // namespace surr
