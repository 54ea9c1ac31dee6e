// Host runtime behind the C ABI of include/surrogate.h: argument checks, the device
// weight arena (re-laid out for the kernels), the per-call planner and the launch
// sequence of one prefill-only scoring pass.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <numeric>
#include <string>
#include <vector>

#include "host.h"
#include "kernels.h"
#include "surrogate.h"

using surr::Act;
using surr::Epi;

namespace {

thread_local std::string g_last_error;

surrogate_status fail(surrogate_status s, const std::string& msg) {
    g_last_error = msg;
    return s;
}

// Fault injection for the cleanup paths, forced from the host.  SURROGATE_FAULT=alloc:N
// makes the N-th device or pinned allocation of a call fail as out of memory, launch:N
// the N-th HIP call the runtime checks (kernel launches, copies, event calls) fail as a
// HIP error without being made.  Only the entry points that load weights, build
// prefixes, create caches or run a pass count (each opens a FaultScope, which re-reads
// the variable and starts counting at 1); every other call, and every call while the
// variable is unset, is untouched.  Every kernel that is launched runs to its normal end.
enum FaultKind { kFaultNone = 0, kFaultAlloc = 1, kFaultLaunch = 2 };
thread_local int t_fault_depth = 0, t_fault_kind = kFaultNone;
thread_local long t_fault_n = 0, t_fault_count = 0;

struct FaultScope {
    FaultScope() {
        if (t_fault_depth++ > 0) return;  // nested entry point: the outer call counts
        const char* v = std::getenv("SURROGATE_FAULT");
        const std::string spec = v ? v : "";
        t_fault_kind = spec.rfind("alloc:", 0) == 0 ? kFaultAlloc
                       : spec.rfind("launch:", 0) == 0 ? kFaultLaunch : kFaultNone;
        t_fault_n = t_fault_kind == kFaultNone ? 0 : std::strtol(spec.c_str() + spec.find(':') + 1, nullptr, 10);
        t_fault_count = 0;
    }
    ~FaultScope() {
        if (--t_fault_depth == 0) t_fault_kind = kFaultNone;
    }
    FaultScope(const FaultScope&) = delete;
    FaultScope& operator=(const FaultScope&) = delete;
};

bool fault(int kind) {
    return t_fault_depth > 0 && t_fault_kind == kind && ++t_fault_count == t_fault_n;
}

#define SURR_HIP(expr)                                                                      \
    do {                                                                                    \
        if (fault(kFaultLaunch))                                                            \
            return fail(SURR_E_HIP, std::string("injected failure (SURROGATE_FAULT) of ") + #expr); \
        hipError_t e_ = (expr);                                                             \
        if (e_ != hipSuccess)                                                               \
            return fail(SURR_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_));     \
    } while (0)

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct LayerW {
    float* attn_norm;
    void* w_qkv;  // [d_q + 2 d_kv, d]: q heads, k heads, v heads
    void* w_o;
    float* mlp_norm;
    void* w_gu;  // [2 d_ff, d]: 32-row blocks alternate gate rows and up rows
    void* w_down;
};

// Byte offsets of one call's workspace regions.
struct WsLayout {
    size_t cu, last, pos_last, vid, work, work_last, vt_off, pfx_len, pfx_off, target, dec_items, dec_first,
        dec_prompt, pos, vcol, x, h, qkv, vt, o, u, gu, o_last, x_last, h_last, u_last, gu_last, y,
        logits, head_part, picked, dec_part, total;
    int64_t dec_cap;  // decode-attention slice items the workspace holds (bf16 models)
    int64_t ld_vt;  // columns of the transposed V copy (bf16 models)
};

using surr::host::tensor_shape;
using surr::host::valid_config;

}  // namespace

struct surrogate_model {
    surrogate_config cfg{};
    Act act = Act::BF16;
    size_t esz = 2;

    char* arena = nullptr;
    void* embed = nullptr;
    void* lm_head = nullptr;
    float* final_norm = nullptr;
    std::vector<LayerW> layers;
    float2* rope_cs = nullptr;
    int32_t* err_flag = nullptr;
    std::mutex mu;  // guards the pinned staging buffer
    void* pinned = nullptr;
    size_t pinned_bytes = 0;
    hipEvent_t staged = nullptr;
    bool staged_pending = false;
    // measurement hook
    bool profiling = false;
    std::vector<hipEvent_t> ev_pool;          // events owned by the model
    std::vector<std::pair<int, size_t>> rec;  // (phase, index of the start event)
    size_t ev_used = 0;

    int64_t d_q() const { return (int64_t)cfg.n_q_heads * cfg.head_dim; }
    int64_t d_kv() const { return (int64_t)cfg.n_kv_heads * cfg.head_dim; }
    int64_t d_qkv() const { return d_q() + 2 * d_kv(); }
};

// Keys (after RoPE) and values of every layer for a set of token sequences: shared prompt
// prefixes, or sequences that grow by prefill and decode steps.  Entry g owns rows
// [off[g], off[g] + cap[g]) (cap a multiple of 64) of each layer's K [rows][d_kv] and the
// same range of its V: bf16 stores V transposed ([d_kv][rows], keys of each 16-key group
// in the order of the kernels' V^T copy), fp32 stores V rows [rows][d_kv].  The first
// len[g] rows hold the entry's tokens; the rest are zero or stale (never read unmasked).
struct surrogate_prefix_cache {
    const surrogate_model* model = nullptr;
    std::vector<int32_t> len, off, cap;
    int64_t rows = 0;
    char* mem = nullptr;
    size_t k_bytes = 0, v_bytes = 0;  // per layer
    void* k(int l) const { return mem + (size_t)l * (k_bytes + v_bytes); }
    void* v(int l) const { return mem + (size_t)l * (k_bytes + v_bytes) + k_bytes; }
};

namespace {

WsLayout layout(const surrogate_model* m, int64_t B, int64_t T) {
    const surrogate_config& c = m->cfg;
    const int64_t qt = surr::attention_q_tile(m->act);
    const int64_t items = (T + qt - 1) / qt + B;
    const size_t e = m->esz;
    const bool f32 = m->act == Act::F32;
    WsLayout w{};
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off += align_up(bytes); return o; };
    w.cu = take(4 * (B + 1));
    w.last = take(4 * B);
    w.pos_last = take(4 * B);
    w.vid = take(4 * 16);
    w.work = take(8 * items);
    w.work_last = take(8 * B);
    w.vt_off = take(4 * (B + 1));
    w.pfx_len = take(4 * B);
    w.pfx_off = take(4 * B);
    w.target = take(4 * B);
    // one-token continuations: up to ceil(max_pos / slice) key slices per prompt
    w.dec_cap = f32 ? 0 : B * ((c.max_pos + surr::attention_decode_slice() - 1) / surr::attention_decode_slice());
    w.dec_items = take(8 * w.dec_cap);
    w.dec_first = take(4 * (B + 1));
    w.dec_prompt = take(4 * B);
    w.pos = take(4 * T);
    // Transposed V copy: every prompt's keys start on a 64-column boundary, so its
    // padded ranges need at most T + 63 B columns.
    w.ld_vt = f32 ? 0 : (T + 63 * B + 63) / 64 * 64;
    w.vcol = f32 ? 0 : take(4 * T);
    w.x = take(4 * T * c.d_model);
    w.h = take(e * T * c.d_model);
    w.qkv = take(e * T * m->d_qkv());
    w.vt = f32 ? 0 : take(2 * (size_t)w.ld_vt * c.n_kv_heads * c.head_dim);
    w.o = take(e * T * m->d_q());
    w.u = take(e * T * c.d_ff);
    w.gu = f32 ? take(4 * T * 2 * c.d_ff) : 0;
    w.o_last = take(e * B * m->d_q());
    w.x_last = take(4 * B * c.d_model);
    w.h_last = take(e * B * c.d_model);
    w.u_last = take(e * B * c.d_ff);
    w.gu_last = f32 ? take(4 * B * 2 * c.d_ff) : 0;
    w.y = take(e * B * c.d_model);
    // LM head: the float32 model writes the logits; bf16 models keep them inside the head
    // GEMM's workgroups and write per-tile records plus the logits at the ids read out
    w.logits = f32 ? take(4 * B * c.vocab) : 0;
    w.head_part = f32 ? 0 : take(16 * B * ((c.vocab + 127) / 128));
    w.picked = f32 ? 0 : take(4 * B * surr::kPicked);
    w.dec_part = take(4 * (size_t)w.dec_cap * c.n_q_heads * (c.head_dim + 4));
    w.total = off;
    return w;
}

}  // namespace

namespace {

// What one pass over a ragged batch does besides the decoder layers.
struct PassIO {
    bool build = false;  // capture every layer's K/V into `capture`; no attention or MLP in
                         // the final layer and no LM head
    surrogate_prefix_cache* capture = nullptr;
    const surrogate_prefix_cache* prefix = nullptr;  // prompts continue cached prefixes
    const int32_t* prefix_id_h = nullptr;            // per prompt: prefix index or -1
    surrogate_prefix_cache* append = nullptr;  // prompts extend these entries (prefix_id_h)
    const int32_t* target_ids_h = nullptr;     // per prompt: next-token id to score
    int32_t* next_token_d = nullptr;           // per prompt: first argmax of the next token
    float* target_lp_d = nullptr;              // per prompt: log-softmax at target_ids_h
    const int32_t* verdict_ids_h = nullptr;
    int32_t n_verdict = 0;
    float* logprobs_d = nullptr;
    float* probs_d = nullptr;
    float* confidence_d = nullptr;
    int32_t* verdict_d = nullptr;
};

surrogate_status check_verdicts(const surrogate_config& c, const int32_t* vid, int32_t n) {
    if (n < 1 || n > 16) return fail(SURR_E_INVALID_ARG, "n_verdict must be in [1, 16]");
    for (int i = 0; i < n; ++i) {
        if (vid[i] < 0 || vid[i] >= c.vocab) return fail(SURR_E_INVALID_ARG, "verdict id out of range");
        for (int j = 0; j < i; ++j)
            if (vid[j] == vid[i]) return fail(SURR_E_INVALID_ARG, "duplicate verdict id");
    }
    return SURR_OK;
}

surrogate_status run_chunks(surrogate_model* m, const int32_t* tokens_d, int64_t row_stride,
                            const int32_t* lengths_h, int32_t batch, void* workspace_d,
                            size_t workspace_bytes, const PassIO& io, hipStream_t stream);

surrogate_status run_pass(surrogate_model* m, const int32_t* tokens_d, int64_t row_stride,
                          const int32_t* lengths_h, int32_t batch, void* workspace_d,
                          size_t workspace_bytes, const PassIO& io, hipStream_t stream) {
    FaultScope fault_scope;
    const surrogate_config& c = m->cfg;
    if (batch < 1) return fail(SURR_E_INVALID_ARG, "batch must be >= 1");
    if (row_stride < 1) return fail(SURR_E_INVALID_ARG, "row_stride must be >= 1");
    std::vector<int32_t> plen(batch, 0), poff(batch, 0), room(batch, INT32_MAX);
    if (io.prefix) {
        const int np = (int)io.prefix->len.size();
        std::vector<char> seen(np, 0);
        for (int b = 0; b < batch; ++b) {
            const int g = io.prefix_id_h[b];
            if (g < (io.append ? 0 : -1) || g >= np)
                return fail(SURR_E_INVALID_ARG, "entry id of prompt " + std::to_string(b) + (io.append ? " outside [0, n_entries)" : " outside [-1, n_prefix)"));
            if (g >= 0) {
                plen[b] = io.prefix->len[g];
                poff[b] = io.prefix->off[g];
                if (io.append) {
                    if (seen[g]) return fail(SURR_E_INVALID_ARG, "entry " + std::to_string(g) + " appears twice in one call");
                    seen[g] = 1;
                    room[b] = io.prefix->cap[g] - plen[b];
                }
            }
        }
    }
    if (io.target_ids_h)
        for (int b = 0; b < batch; ++b)
            if (io.target_ids_h[b] < 0 || io.target_ids_h[b] >= c.vocab)
                return fail(SURR_E_INVALID_ARG, "target id of prompt " + std::to_string(b) + " outside [0, vocab)");
    const bool dec_path = m->act == Act::BF16 && io.append && c.n_q_heads / c.n_kv_heads <= 16 &&
                          (c.max_pos + surr::attention_decode_slice() - 1) / surr::attention_decode_slice() <=
                              surr::attention_decode_max_slices();
    surr::host::PlanArgs pa;
    pa.lengths = lengths_h;
    pa.batch = batch;
    pa.row_stride = row_stride;
    pa.max_pos = c.max_pos;
    pa.q_tile = surr::attention_q_tile(m->act);
    pa.plen = plen.data();
    pa.room = room.data();
    pa.build = io.build;
    pa.append = io.append != nullptr;
    pa.prefix = io.prefix != nullptr;
    pa.dec_path = dec_path;
    pa.dec_slice = surr::attention_decode_slice();
    surr::host::Plan plan;
    {
        std::string why;
        const surrogate_status ps = surr::host::plan_batch(pa, &plan, &why);
        if (ps != SURR_OK) return fail(ps, why);
    }
    const int64_t T = plan.T;
    const int max_len = plan.max_len;
    if (reinterpret_cast<uintptr_t>(workspace_d) % kAlign) return fail(SURR_E_INVALID_ARG, "workspace must be 256-byte aligned");
    const WsLayout w = layout(m, batch, T);
    if (workspace_bytes < w.total) {
        // Token budget: score consecutive chunks of whole prompts, each as large as the
        // workspace holds (prompts are independent, so every output is unchanged).  A
        // prefix build lays its cache out per call and is never split.
        if (io.build || batch == 1)
            return fail(SURR_E_WORKSPACE, "workspace needs " + std::to_string(w.total) + " bytes");
        return run_chunks(m, tokens_d, row_stride, lengths_h, batch, workspace_d, workspace_bytes, io, stream);
    }
    const int32_t n_verdict = io.n_verdict;
    const int32_t* verdict_ids_h = io.verdict_ids_h;
    float* logprobs_d = io.logprobs_d;
    float* probs_d = io.probs_d;
    float* confidence_d = io.confidence_d;
    int32_t* verdict_d = io.verdict_d;
    // ---- plan: prompt offsets, last rows, verdict ids, attention work lists
    const std::vector<int32_t>& cu = plan.cu;
    const std::vector<int32_t>& last = plan.last;
    const std::vector<int32_t>& pos_last = plan.pos_last;
    const std::vector<int32_t>& vt_off = plan.vt_off;
    const std::vector<int32_t>& dprompt = plan.dprompt;
    const std::vector<int32_t>& dfirst = plan.dfirst;
    const std::vector<surr::host::Int2>& ditems = plan.ditems;
    const std::vector<surr::host::Int2>& work = plan.work;
    const std::vector<surr::host::Int2>& work_last = plan.work_last;
    static_assert(sizeof(surr::host::Int2) == sizeof(int2), "work items are copied as int2");

    const size_t meta_bytes = w.pos;  // cu .. vt_off are contiguous from offset 0
    {
        std::lock_guard<std::mutex> lock(m->mu);
        if (m->staged_pending) SURR_HIP(hipEventSynchronize(m->staged));
        m->staged_pending = false;
        if (m->pinned_bytes < meta_bytes) {
            if (m->pinned) SURR_HIP(hipHostFree(m->pinned));
            m->pinned = nullptr;
            m->pinned_bytes = 0;
            if (fault(kFaultAlloc) || hipHostMalloc(&m->pinned, meta_bytes, hipHostMallocDefault) != hipSuccess) {
                m->pinned = nullptr;
                return fail(SURR_E_OOM, "pinned staging buffer");
            }
            m->pinned_bytes = meta_bytes;
        }
        char* P = static_cast<char*>(m->pinned);
        std::memcpy(P + w.cu, cu.data(), 4 * cu.size());
        std::memcpy(P + w.last, last.data(), 4 * last.size());
        std::memcpy(P + w.pos_last, pos_last.data(), 4 * pos_last.size());
        if (n_verdict) std::memcpy(P + w.vid, verdict_ids_h, 4 * (size_t)n_verdict);
        std::memcpy(P + w.work, work.data(), 8 * work.size());
        std::memcpy(P + w.work_last, work_last.data(), 8 * work_last.size());
        std::memcpy(P + w.vt_off, vt_off.data(), 4 * vt_off.size());
        std::memcpy(P + w.pfx_len, plen.data(), 4 * plen.size());
        std::memcpy(P + w.pfx_off, poff.data(), 4 * poff.size());
        if (io.target_ids_h) std::memcpy(P + w.target, io.target_ids_h, 4 * (size_t)batch);
        if (!dprompt.empty()) {
            std::memcpy(P + w.dec_items, ditems.data(), 8 * ditems.size());
            std::memcpy(P + w.dec_first, dfirst.data(), 4 * dfirst.size());
            std::memcpy(P + w.dec_prompt, dprompt.data(), 4 * dprompt.size());
        }
        // Once the copy may be in flight, the buffer is not refilled before it is done: the
        // event marks that, and if it cannot be recorded the stream is drained instead.
        bool injected = fault(kFaultLaunch);
        hipError_t e = injected ? hipErrorLaunchFailure
                                : hipMemcpyAsync(workspace_d, P, meta_bytes, hipMemcpyHostToDevice, stream);
        if (e == hipSuccess) {
            injected = fault(kFaultLaunch);
            e = injected ? hipErrorLaunchFailure : hipEventRecord(m->staged, stream);
        }
        if (e != hipSuccess) {
            hipStreamSynchronize(stream);
            return fail(SURR_E_HIP, std::string("staging the batch plan: ") +
                                        (injected ? "injected failure (SURROGATE_FAULT)" : hipGetErrorString(e)));
        }
        m->staged_pending = true;
    }

    char* W = static_cast<char*>(workspace_d);
    const int32_t* d_cu = reinterpret_cast<const int32_t*>(W + w.cu);
    const int32_t* d_last = reinterpret_cast<const int32_t*>(W + w.last);
    const int32_t* d_pos_last = reinterpret_cast<const int32_t*>(W + w.pos_last);
    const int32_t* d_vid = reinterpret_cast<const int32_t*>(W + w.vid);
    const int2* d_work = reinterpret_cast<const int2*>(W + w.work);
    const int2* d_work_last = reinterpret_cast<const int2*>(W + w.work_last);
    const int2* d_dec_items = reinterpret_cast<const int2*>(W + w.dec_items);
    const int32_t* d_dec_first = reinterpret_cast<const int32_t*>(W + w.dec_first);
    const int32_t* d_dec_prompt = reinterpret_cast<const int32_t*>(W + w.dec_prompt);
    float* d_dec_part = reinterpret_cast<float*>(W + w.dec_part);
    int32_t* d_pos = reinterpret_cast<int32_t*>(W + w.pos);
    const int32_t* d_po = reinterpret_cast<const int32_t*>(W + w.vt_off);  // 64-aligned row blocks
    const int32_t* d_pfx_len = reinterpret_cast<const int32_t*>(W + w.pfx_len);
    const int32_t* d_pfx_off = reinterpret_cast<const int32_t*>(W + w.pfx_off);
    const int32_t* d_target = reinterpret_cast<const int32_t*>(W + w.target);
    const bool bf16 = m->act == Act::BF16;
    const int32_t* d_vt_off = bf16 ? reinterpret_cast<const int32_t*>(W + w.vt_off) : nullptr;
    int32_t* d_vcol = bf16 ? reinterpret_cast<int32_t*>(W + w.vcol) : nullptr;
    uint16_t* vt = bf16 ? reinterpret_cast<uint16_t*>(W + w.vt) : nullptr;
    float* x = reinterpret_cast<float*>(W + w.x);
    void* h = W + w.h;
    void* qkv = W + w.qkv;
    void* o = W + w.o;
    void* u = W + w.u;
    float* gu = reinterpret_cast<float*>(W + w.gu);
    void* o_last = W + w.o_last;
    float* x_last = reinterpret_cast<float*>(W + w.x_last);
    void* h_last = W + w.h_last;
    void* u_last = W + w.u_last;
    float* gu_last = reinterpret_cast<float*>(W + w.gu_last);
    void* y = W + w.y;
    float* logits = reinterpret_cast<float*>(W + w.logits);

    const Act a = m->act;
    const int d = c.d_model, ff = c.d_ff, nq = c.n_q_heads, nkv = c.n_kv_heads, hd = c.head_dim;
    const int dq = (int)m->d_q(), dqkv = (int)m->d_qkv();
    const int Ti = (int)T;


    // Phase bracketing for the measurement hook (a no-op unless profiling is on).
    auto mark = [&](int phase) -> hipError_t {
        if (!m->profiling) return hipSuccess;
        while (m->ev_used + 2 > m->ev_pool.size()) {
            hipEvent_t e;
            hipError_t r = hipEventCreate(&e);
            if (r != hipSuccess) return r;
            m->ev_pool.push_back(e);
        }
        m->rec.emplace_back(phase, m->ev_used);
        const hipEvent_t e0 = m->ev_pool[m->ev_used];
        m->ev_used += 2;
        return hipEventRecord(e0, stream);
    };
    auto done = [&]() -> hipError_t {
        if (!m->profiling) return hipSuccess;
        return hipEventRecord(m->ev_pool[m->rec.back().second + 1], stream);
    };
#define SURR_PHASE_RUN(phase, expr)  \
    do {                             \
        SURR_HIP(mark(phase));       \
        SURR_HIP(expr);              \
        SURR_HIP(done());            \
    } while (0)

    auto mlp = [&](const LayerW& L, void* hin, void* uout, float* gtmp, float* xres, int M,
                   int ph_gu, int ph_down) -> surrogate_status {
        if (a == Act::BF16) {
            SURR_PHASE_RUN(ph_gu, surr::launch_gemm(a, Epi::SwiGLU, hin, d, L.w_gu, d, uout, ff, M, 2 * ff, d, stream));
        } else {
            SURR_PHASE_RUN(ph_gu, surr::launch_gemm(a, Epi::StoreF32, hin, d, L.w_gu, d, gtmp, 2 * ff, M, 2 * ff, d, stream));
            SURR_PHASE_RUN(ph_gu, surr::launch_swiglu_f32(gtmp, static_cast<float*>(uout), M, ff, stream));
        }
        SURR_PHASE_RUN(ph_down, surr::launch_gemm(a, Epi::ResidAddF32, uout, ff, L.w_down, ff, xres, d, M, d, ff, stream));
        return SURR_OK;
    };

    SURR_PHASE_RUN(SURR_PHASE_EMBED, surr::launch_embed(a, tokens_d, row_stride, d_cu, batch, T, m->embed, d, c.vocab, x, d_pos, io.prefix ? d_pfx_len : nullptr, d_vt_off, d_vcol, m->err_flag, stream));
    if (bf16)  // the projection epilogues never write these columns
        SURR_PHASE_RUN(SURR_PHASE_EMBED, surr::launch_vt_pad_zero(vt, w.ld_vt, nkv * hd, d_cu, d_vt_off, batch, stream));
    for (int l = 0; l < c.n_layers; ++l) {
        const LayerW& L = m->layers[l];
        const bool final_layer = l == c.n_layers - 1;
        surr::PrefixKV pk;
        if (io.prefix) {
            pk.k = io.prefix->k(l);
            pk.ld_k = m->d_kv();
            pk.v = io.prefix->v(l);
            pk.ld_v = bf16 ? io.prefix->rows : m->d_kv();
            pk.len = d_pfx_len;
            pk.off = d_pfx_off;
        }
        const surr::PrefixKV* pkp = io.prefix ? &pk : nullptr;
        SURR_PHASE_RUN(SURR_PHASE_RMSNORM, surr::launch_rmsnorm(a, x, d, nullptr, T, L.attn_norm, d, c.rms_eps, h, d, stream));
        if (a == Act::BF16) {
            // RoPE on the q and k heads happens in the GEMM epilogue (one rounding)
            surr::EpiArgs rope;
            rope.pos = d_pos;
            rope.cs = m->rope_cs;
            rope.cols = (nq + nkv) * hd;
            rope.head_dim = hd;
            rope.vt = vt;
            rope.ld_vt = w.ld_vt;
            rope.vcol = d_vcol;
            // The final layer needs keys and values of every token but queries only at the
            // last positions (and none when building a prefix cache): the K/V weight rows
            // run over all tokens, the query rows over the gathered last rows, whose
            // queries then go to their rows of qkv for the attention below.  Same sums and
            // roundings as the full projection.  With few tokens per prompt (decode steps)
            // the full projection is cheaper than the extra launches.
            const bool q_last_only = final_layer && (io.build || T > 2 * (int64_t)batch);
            if (!q_last_only) {
                SURR_PHASE_RUN(SURR_PHASE_GEMM_QKV, surr::launch_gemm(a, Epi::StoreActRope, h, d, L.w_qkv, d, qkv, dqkv, Ti, dqkv, d, stream, rope));
            } else {
                surr::EpiArgs rkv = rope;
                rkv.cols = nkv * hd;  // columns [0, nkv hd) of this product are keys
                rkv.b_row0 = (int)dq;  // the K and V rows of the packed w_qkv
                SURR_PHASE_RUN(SURR_PHASE_GEMM_QKV, surr::launch_gemm(a, Epi::StoreActRope, h, d, L.w_qkv, d, static_cast<char*>(qkv) + 2 * (size_t)dq, dqkv, Ti, dqkv - dq, d, stream, rkv));
                if (!io.build) {
                    surr::EpiArgs rq;
                    rq.pos = d_pos_last;
                    rq.cs = m->rope_cs;
                    rq.cols = dq;
                    rq.head_dim = hd;
                    SURR_PHASE_RUN(SURR_PHASE_GEMM_QKV, surr::launch_gather_rows(h, d, d_last, batch, d, 2, h_last, d, stream));
                    SURR_PHASE_RUN(SURR_PHASE_GEMM_QKV, surr::launch_gemm(a, Epi::StoreActRope, h_last, d, L.w_qkv, d, o_last, dq, batch, dq, d, stream, rq));
                    SURR_PHASE_RUN(SURR_PHASE_GEMM_QKV, surr::launch_scatter_rows(o_last, dq, d_last, batch, dq, 2, qkv, dqkv, stream));
                }
            }
        } else {
            SURR_PHASE_RUN(SURR_PHASE_GEMM_QKV, surr::launch_gemm(a, Epi::StoreAct, h, d, L.w_qkv, d, qkv, dqkv, Ti, dqkv, d, stream));
            SURR_PHASE_RUN(SURR_PHASE_ROPE, surr::launch_rope(a, qkv, dqkv, T, d_pos, nq + nkv, hd, m->rope_cs, stream));
        }
        if (io.build) {
            // keep this layer's keys and values for the prompts that will continue them
            surrogate_prefix_cache* pc = io.capture;
            SURR_PHASE_RUN(SURR_PHASE_PREFIX_CAPTURE, surr::launch_capture_rows(qkv, dqkv, dq, (int)m->d_kv(), (int)m->esz, d_cu, d_po, batch, pc->rows, pc->k(l), m->d_kv(), stream));
            if (bf16)
                SURR_PHASE_RUN(SURR_PHASE_PREFIX_CAPTURE, hipMemcpy2DAsync(pc->v(l), 2 * pc->rows, vt, 2 * w.ld_vt, 2 * pc->rows, m->d_kv(), hipMemcpyDeviceToDevice, stream));
            else
                SURR_PHASE_RUN(SURR_PHASE_PREFIX_CAPTURE, surr::launch_capture_rows(qkv, dqkv, dq + (int)m->d_kv(), (int)m->d_kv(), 4, d_cu, d_po, batch, pc->rows, pc->v(l), m->d_kv(), stream));
            if (final_layer) break;  // nothing past the last layer's K/V is needed
        }
        if (io.append) {
            // the new tokens' keys and values continue their entries (rows past the
            // entries' current lengths, which this layer's attention does not read)
            surrogate_prefix_cache* pc = io.append;
            const int dkv = (int)m->d_kv();
            if (bf16) {
                SURR_PHASE_RUN(SURR_PHASE_PREFIX_CAPTURE, surr::launch_append_kv(static_cast<const uint16_t*>(qkv), dqkv, dq, dkv, T, vt, w.ld_vt, d_vt_off, d_cu, batch, max_len, d_pfx_off, d_pfx_len, static_cast<uint16_t*>(pc->k(l)), dkv, dkv, static_cast<uint16_t*>(pc->v(l)), pc->rows, stream));
            } else {
                SURR_PHASE_RUN(SURR_PHASE_PREFIX_CAPTURE, surr::launch_append_rows(qkv, dqkv, dq, dkv, (int)m->esz, T, d_cu, batch, d_pfx_off, d_pfx_len, pc->k(l), dkv, stream));
                SURR_PHASE_RUN(SURR_PHASE_PREFIX_CAPTURE, surr::launch_append_rows(qkv, dqkv, dq + dkv, dkv, 4, T, d_cu, batch, d_pfx_off, d_pfx_len, pc->v(l), dkv, stream));
            }
        }
        if (!final_layer) {
            SURR_PHASE_RUN(SURR_PHASE_ATTENTION, surr::launch_attention(a, qkv, dqkv, vt, w.ld_vt, d_vt_off, o, dq, d_cu, d_work, (int)work.size(), nq, nkv, hd, stream, pkp));
            if (!dprompt.empty())
                SURR_PHASE_RUN(SURR_PHASE_ATTENTION, surr::launch_attention_decode(qkv, dqkv, d_cu, d_dec_items, (int)ditems.size(), d_dec_prompt, d_dec_first, (int)dprompt.size(), nq, nkv, hd, pk, d_dec_part, o, dq, stream));
            SURR_PHASE_RUN(SURR_PHASE_GEMM_O, surr::launch_gemm(a, Epi::ResidAddF32, o, dq, L.w_o, dq, x, d, Ti, d, dq, stream));
            SURR_PHASE_RUN(SURR_PHASE_RMSNORM, surr::launch_rmsnorm(a, x, d, nullptr, T, L.mlp_norm, d, c.rms_eps, h, d, stream));
            const surrogate_status st = mlp(L, h, u, gu, x, Ti, SURR_PHASE_GEMM_GATE_UP, SURR_PHASE_GEMM_DOWN);
            if (st != SURR_OK) return st;
        } else {
            // Only the last position of each prompt feeds the LM head: K/V above cover
            // every token; attention, O projection and MLP run for the last rows only.
            SURR_PHASE_RUN(SURR_PHASE_ATTENTION, surr::launch_attention(a, qkv, dqkv, vt, w.ld_vt, d_vt_off, o, dq, d_cu, d_work_last, (int)work_last.size(), nq, nkv, hd, stream, pkp));
            if (!dprompt.empty())
                SURR_PHASE_RUN(SURR_PHASE_ATTENTION, surr::launch_attention_decode(qkv, dqkv, d_cu, d_dec_items, (int)ditems.size(), d_dec_prompt, d_dec_first, (int)dprompt.size(), nq, nkv, hd, pk, d_dec_part, o, dq, stream));
            SURR_PHASE_RUN(SURR_PHASE_LAST_ROWS, surr::launch_gather_rows(o, dq, d_last, batch, dq, (int)m->esz, o_last, dq, stream));
            SURR_PHASE_RUN(SURR_PHASE_LAST_ROWS, surr::launch_gather_rows(x, d, d_last, batch, d, 4, x_last, d, stream));
            SURR_PHASE_RUN(SURR_PHASE_LAST_ROWS, surr::launch_gemm(a, Epi::ResidAddF32, o_last, dq, L.w_o, dq, x_last, d, batch, d, dq, stream));
            SURR_PHASE_RUN(SURR_PHASE_LAST_ROWS, surr::launch_rmsnorm(a, x_last, d, nullptr, batch, L.mlp_norm, d, c.rms_eps, h_last, d, stream));
            const surrogate_status st = mlp(L, h_last, u_last, gu_last, x_last, batch, SURR_PHASE_LAST_ROWS, SURR_PHASE_LAST_ROWS);
            if (st != SURR_OK) return st;
        }
    }
    if (io.build) return SURR_OK;
    SURR_PHASE_RUN(SURR_PHASE_LAST_ROWS, surr::launch_rmsnorm(a, x_last, d, nullptr, batch, m->final_norm, d, c.rms_eps, y, d, stream));
    if (bf16) {
        // Full-vocabulary read-out without logits in memory: the head GEMM's epilogue
        // writes per-tile (max, sum of exp, first argmax) records and the logits at the
        // verdict and target ids; one small kernel merges the tiles in order.
        surr::EpiArgs hk;
        hk.head.vid = n_verdict ? d_vid : nullptr;
        hk.head.n_vid = n_verdict;
        hk.head.target = io.target_ids_h ? d_target : nullptr;
        hk.head.part = reinterpret_cast<float4*>(W + w.head_part);
        hk.head.picked = reinterpret_cast<float*>(W + w.picked);
        SURR_PHASE_RUN(SURR_PHASE_LM_HEAD, surr::launch_gemm(a, Epi::LseTile, y, d, m->lm_head, d, nullptr, 0, batch, c.vocab, d, stream, hk));
        SURR_PHASE_RUN(SURR_PHASE_LSE_VERDICT, surr::launch_lse_combine(hk.head.part, (c.vocab + 127) / 128, hk.head.picked, batch, n_verdict, logprobs_d, probs_d, confidence_d, verdict_d, io.next_token_d, io.target_ids_h ? io.target_lp_d : nullptr, stream));
    } else {
        SURR_PHASE_RUN(SURR_PHASE_LM_HEAD, surr::launch_gemm(a, Epi::StoreF32, y, d, m->lm_head, d, logits, c.vocab, batch, c.vocab, d, stream));
        if (n_verdict)
            SURR_PHASE_RUN(SURR_PHASE_LSE_VERDICT, surr::launch_lse_verdict(logits, c.vocab, batch, c.vocab, d_vid, n_verdict, logprobs_d, probs_d, confidence_d, verdict_d, stream));
        if (io.next_token_d || io.target_lp_d)
            SURR_PHASE_RUN(SURR_PHASE_LSE_VERDICT, surr::launch_lse_next(logits, c.vocab, batch, c.vocab, io.target_ids_h ? d_target : nullptr, io.next_token_d, io.target_ids_h ? io.target_lp_d : nullptr, stream));
    }
#undef SURR_PHASE_RUN
    if (io.append)  // the work above is enqueued: the entries now hold the new tokens
        for (int b = 0; b < batch; ++b) io.append->len[io.prefix_id_h[b]] += lengths_h[b];
    return SURR_OK;
}

// Host-side form of an evaluator call: validated arguments, per-bin constants, the
// measured count of each budget and the workspace it needs.
struct EvalCall {
    surr::EvalBins eb{};
    surr::BinWeights hw{};
    int ks[8] = {};
    size_t need = 0;
};

surrogate_status evaluate_args(const float* probs_d, const float* speedup_d, int32_t n,
                               int32_t n_bins, const double* bin_values_h, const double* bin_edges_h,
                               const double* budgets_h, int32_t n_budgets, double* summary_d,
                               EvalCall* ec) {
    if (!probs_d || !speedup_d || !bin_values_h || !bin_edges_h || !budgets_h || !summary_d)
        return fail(SURR_E_INVALID_ARG, "null argument");
    if (n_bins < 2 || n_bins > surr::kMaxBins) return fail(SURR_E_INVALID_ARG, "n_bins must be in [2, 16]");
    const surrogate_status st = surrogate_evaluate_workspace_size(n, n_budgets, &ec->need);
    if (st != SURR_OK) return st;  // also bounds n_budgets by 8
    for (int b = 0; b < n_bins; ++b) {
        if (!std::isfinite(bin_values_h[b])) return fail(SURR_E_INVALID_ARG, "non-finite bin value");
        ec->eb.value[b] = (float)bin_values_h[b];
        ec->hw.w[b][0] = (float)bin_values_h[b];
    }
    for (int j = 0; j < n_bins - 1; ++j) {
        if (!std::isfinite(bin_edges_h[j]) || !(bin_edges_h[j] > 0.0) ||
            (j > 0 && !(bin_edges_h[j] > bin_edges_h[j - 1])))
            return fail(SURR_E_INVALID_ARG, "bin edges must be finite, positive, strictly increasing");
        ec->eb.edge[j] = bin_edges_h[j];
    }
    for (int c = 0; c < n_budgets; ++c) {
        if (!(budgets_h[c] > 0.0 && budgets_h[c] <= 1.0)) return fail(SURR_E_INVALID_ARG, "budgets must lie in (0, 1]");
        ec->ks[c] = std::max(1, (int)std::floor(budgets_h[c] * n));  // top c%, at least one
    }
    return SURR_OK;
}

// The evaluator's launches on a device buffer W of ec.need bytes: expected speedups, per
// budget the two index lists, the counts, the per-workgroup partial rows.  Every byte it
// reads was written earlier in the same call, so W needs no clearing.
surrogate_status evaluate_launch(const EvalCall& ec, const float* probs_d, const float* speedup_d,
                                 int32_t n, int32_t n_bins, int32_t n_budgets, char* W,
                                 int32_t* bin_d, float* brier_d, float* crps_d, double* summary_d,
                                 hipStream_t stream) {
    float* shat = reinterpret_cast<float*>(W);
    int32_t* lists = reinterpret_cast<int32_t*>(W + align_up(4 * (size_t)n));
    int32_t* counts = reinterpret_cast<int32_t*>(W + align_up(4 * (size_t)n) + align_up(8 * (size_t)n * n_budgets));
    double* partial = reinterpret_cast<double*>(W + align_up(4 * (size_t)n) + align_up(8 * (size_t)n * n_budgets) + align_up(8 * (size_t)n_budgets));
    SURR_HIP(surr::launch_eval_metrics(probs_d, speedup_d, n, n_bins, ec.eb, bin_d, brier_d, crps_d, partial, stream));
    SURR_HIP(surr::launch_forecast_head(probs_d, n, n_bins, ec.hw, 0, shat, nullptr, stream));
    for (int c = 0; c < n_budgets; ++c) {
        int32_t* d = lists + (size_t)c * 2 * n;
        SURR_HIP(surr::launch_select(shat, n, 2, 0.f, ec.ks[c], d, d + n, counts + 2 * c, stream));
    }
    SURR_HIP(surr::launch_eval_finalize(speedup_d, n, lists, counts, n_budgets, partial, summary_d, stream));
    return SURR_OK;
}

// Scratch of surrogate_evaluate_noalloc: room for the evaluator's largest call (65,536
// forecasts, 8 budgets: 4,536,576 bytes).  Each device the library runs on holds its own
// copy until the process ends.  Host code never passes the name `scratch` to a kernel or
// a copy (on the host it is only a stand-in for the device symbol): it takes the device
// address from device_scratch().
constexpr size_t kScratchBytes = 4608 * 1024;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_addr[kMaxScratchDevices] = {};

// Device address of the current device's scratch, looked up once per device (with that
// device current) on the first call that needs it.
surrogate_status device_scratch(char** out) {
    int dev = -1;
    SURR_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxScratchDevices) return fail(SURR_E_HIP, "device ordinal beyond the scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_addr[dev]) {
        void* p = nullptr;
        SURR_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) return fail(SURR_E_HIP, "hipGetSymbolAddress returned no address for the scratch");
        g_scratch_addr[dev] = static_cast<char*>(p);
    }
    *out = g_scratch_addr[dev];
    return SURR_OK;
}

// The batch in consecutive chunks of whole prompts, each the longest run from the current
// prompt whose workspace fits in workspace_bytes (lengths already checked by the caller).
surrogate_status run_chunks(surrogate_model* m, const int32_t* tokens_d, int64_t row_stride,
                            const int32_t* lengths_h, int32_t batch, void* workspace_d,
                            size_t workspace_bytes, const PassIO& io, hipStream_t stream) {
    int start = 0;
    while (start < batch) {
        int end = start;
        int64_t t = 0;
        while (end < batch && layout(m, end - start + 1, t + lengths_h[end]).total <= workspace_bytes)
            t += lengths_h[end++];
        if (end == start)
            return fail(SURR_E_WORKSPACE, "workspace needs " +
                                              std::to_string(layout(m, 1, lengths_h[start]).total) +
                                              " bytes for prompt " + std::to_string(start) + " alone");
        PassIO sub = io;
        const int nv = io.n_verdict;
        if (io.prefix_id_h) sub.prefix_id_h = io.prefix_id_h + start;
        if (io.target_ids_h) sub.target_ids_h = io.target_ids_h + start;
        if (io.next_token_d) sub.next_token_d = io.next_token_d + start;
        if (io.target_lp_d) sub.target_lp_d = io.target_lp_d + start;
        if (io.logprobs_d) sub.logprobs_d = io.logprobs_d + (size_t)start * nv;
        if (io.probs_d) sub.probs_d = io.probs_d + (size_t)start * nv;
        if (io.confidence_d) sub.confidence_d = io.confidence_d + start;
        if (io.verdict_d) sub.verdict_d = io.verdict_d + start;
        const surrogate_status st = run_pass(m, tokens_d + (int64_t)start * row_stride, row_stride,
                                             lengths_h + start, end - start, workspace_d,
                                             workspace_bytes, sub, stream);
        if (st != SURR_OK) return st;
        start = end;
    }
    return SURR_OK;
}

}  // namespace

extern "C" {

surrogate_status surrogate_tensor_count(const surrogate_config* cfg, int32_t* n_out) {
    if (!cfg || !n_out) return fail(SURR_E_INVALID_ARG, "null argument");
    if (cfg->n_layers < 1) return fail(SURR_E_SHAPE, "n_layers must be >= 1");
    *n_out = 3 + 9 * cfg->n_layers;
    return SURR_OK;
}

surrogate_status surrogate_tensor_shape(const surrogate_config* cfg, int32_t index, int64_t* rows,
                                        int64_t* cols, int32_t* dtype_out) {
    if (!cfg || !rows || !cols || !dtype_out) return fail(SURR_E_INVALID_ARG, "null argument");
    std::string why;
    if (!valid_config(cfg, &why)) return fail(SURR_E_SHAPE, why);
    if (index < 0 || index >= 3 + 9 * cfg->n_layers) return fail(SURR_E_INVALID_ARG, "tensor index out of range");
    tensor_shape(cfg, index, rows, cols, dtype_out);
    return SURR_OK;
}

void surrogate_free(surrogate_model* m) {
    if (!m) return;
    for (hipEvent_t e : m->ev_pool) hipEventDestroy(e);
    if (m->staged) {
        hipEventSynchronize(m->staged);
        hipEventDestroy(m->staged);
    }
    if (m->pinned) hipHostFree(m->pinned);
    if (m->arena) hipFree(m->arena);
    delete m;
}

surrogate_status surrogate_load_weights_tensors(const surrogate_config* cfg, const void* const* tensors,
                                                int32_t n_tensors, int32_t tensors_on_device,
                                                hipStream_t stream, surrogate_model** out) {
    FaultScope fault_scope;
    if (!cfg || !tensors || !out) return fail(SURR_E_INVALID_ARG, "null argument");
    *out = nullptr;
    std::string why;
    if (!valid_config(cfg, &why)) return fail(SURR_E_SHAPE, why);
    const int32_t want = 3 + 9 * cfg->n_layers;
    if (n_tensors != want)
        return fail(SURR_E_WEIGHTS, "expected " + std::to_string(want) + " tensors, got " + std::to_string(n_tensors));
    for (int i = 0; i < n_tensors; ++i)
        if (!tensors[i]) return fail(SURR_E_INVALID_ARG, "tensor " + std::to_string(i) + " is null");

    surrogate_model* m = new surrogate_model();
    m->cfg = *cfg;
    m->act = cfg->dtype == SURR_BF16 ? Act::BF16 : Act::F32;
    m->esz = cfg->dtype == SURR_BF16 ? 2 : 4;
    const surrogate_config& c = m->cfg;
    const size_t e = m->esz, d = c.d_model, ff = c.d_ff, V = c.vocab;
    const size_t dq = m->d_q(), dkv = m->d_kv(), half = c.head_dim / 2;

    // Arena: embed, layers, final norm, head, RoPE table, error word.  bf16 projection
    // matrices are stored panel-packed (rows padded to whole panels).
    const bool packed = m->act == Act::BF16;
    auto mat = [&](size_t rows, size_t k) { return (packed ? (size_t)surr::packed_rows((int64_t)rows) : rows) * k * e; };
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off += align_up(bytes); return o; };
    const size_t o_embed = take(V * d * e);
    struct LOff { size_t an, qkv, o, mn, gu, dn; };
    std::vector<LOff> lo(c.n_layers);
    for (auto& l : lo) {
        l.an = take(4 * d);
        l.qkv = take(mat(dq + 2 * dkv, d));
        l.o = take(mat(d, dq));
        l.mn = take(4 * d);
        l.gu = take(mat(2 * ff, d));
        l.dn = take(mat(d, ff));
    }
    const size_t o_fn = take(4 * d), o_head = take(mat(V, d));
    const size_t o_rope = take((size_t)c.max_pos * half * sizeof(float2)), o_err = take(4);
    if (fault(kFaultAlloc) || hipMalloc(&m->arena, off) != hipSuccess) {
        m->arena = nullptr;
        surrogate_free(m);
        return fail(SURR_E_OOM, "weight arena of " + std::to_string(off) + " bytes");
    }
    char* A = m->arena;
    m->embed = A + o_embed;
    m->final_norm = reinterpret_cast<float*>(A + o_fn);
    m->lm_head = A + o_head;
    m->rope_cs = reinterpret_cast<float2*>(A + o_rope);
    m->err_flag = reinterpret_cast<int32_t*>(A + o_err);
    for (auto& l : lo)
        m->layers.push_back({reinterpret_cast<float*>(A + l.an), A + l.qkv, A + l.o,
                             reinterpret_cast<float*>(A + l.mn), A + l.gu, A + l.dn});

    const hipMemcpyKind kind = tensors_on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
    std::vector<float2> cs((size_t)c.max_pos * half);
    // bf16 matrices are first assembled row-major in a staging buffer (the largest one's
    // size, freed when loading ends), then packed into the arena; fp32 ones go straight in.
    char* stage = nullptr;
    auto body = [&]() -> surrogate_status {
        auto cp = [&](void* dst, const void* src, size_t bytes) {
            return hipMemcpyAsync(dst, src, bytes, kind, stream);
        };
        if (packed) {
            const size_t most = std::max({(dq + 2 * dkv) * d, d * dq, 2 * ff * d, d * ff, V * d}) * e;
            if (fault(kFaultAlloc) || hipMalloc(&stage, most) != hipSuccess) {
                stage = nullptr;
                return fail(SURR_E_OOM, "weight staging buffer of " + std::to_string(most) + " bytes");
            }
        }
        // matrix [rows, k] assembled at `rm` (row-major) by fill(rm), then placed at dst
        auto put = [&](void* dst, size_t rows, size_t k, auto fill) -> hipError_t {
            char* rm = packed ? stage : static_cast<char*>(dst);
            hipError_t err = fill(rm);
            if (err == hipSuccess && packed)
                err = surr::launch_pack_panels(reinterpret_cast<const uint16_t*>(rm), (int64_t)rows, (int64_t)k,
                                               static_cast<uint16_t*>(dst), stream);
            return err;
        };
        SURR_HIP(cp(m->embed, tensors[0], V * d * e));
        for (int l = 0; l < c.n_layers; ++l) {
            const void* const* t = tensors + 1 + 9 * l;
            SURR_HIP(cp(m->layers[l].attn_norm, t[0], 4 * d));
            SURR_HIP(put(m->layers[l].w_qkv, dq + 2 * dkv, d, [&](char* qkv) {
                hipError_t err = cp(qkv, t[1], dq * d * e);
                if (err == hipSuccess) err = cp(qkv + dq * d * e, t[2], dkv * d * e);
                if (err == hipSuccess) err = cp(qkv + (dq + dkv) * d * e, t[3], dkv * d * e);
                return err;
            }));
            SURR_HIP(put(m->layers[l].w_o, d, dq, [&](char* w) { return cp(w, t[4], d * dq * e); }));
            SURR_HIP(cp(m->layers[l].mlp_norm, t[5], 4 * d));
            // gate/up interleave: block p of 32 gate rows goes to rows [64p, 64p+32), the
            // matching up rows to [64p+32, 64p+64).
            SURR_HIP(put(m->layers[l].w_gu, 2 * ff, d, [&](char* gu) {
                const size_t blk = 32 * d * e;
                hipError_t err = hipMemcpy2DAsync(gu, 2 * blk, t[6], blk, blk, ff / 32, kind, stream);
                if (err == hipSuccess) err = hipMemcpy2DAsync(gu + blk, 2 * blk, t[7], blk, blk, ff / 32, kind, stream);
                return err;
            }));
            SURR_HIP(put(m->layers[l].w_down, d, ff, [&](char* w) { return cp(w, t[8], d * ff * e); }));
        }
        const int last = 1 + 9 * c.n_layers;
        SURR_HIP(cp(m->final_norm, tensors[last], 4 * d));
        SURR_HIP(put(m->lm_head, V, d, [&](char* w) { return cp(w, tensors[last + 1], V * d * e); }));
        // RoPE: theta = pos * base^(-2i/hd) in float64, stored as float32 (cos, sin).
        for (int p = 0; p < c.max_pos; ++p)
            for (size_t i = 0; i < half; ++i) {
                const double th = (double)p * std::pow((double)c.rope_base, -2.0 * (double)i / c.head_dim);
                cs[(size_t)p * half + i] = make_float2((float)std::cos(th), (float)std::sin(th));
            }
        SURR_HIP(hipMemcpyAsync(m->rope_cs, cs.data(), cs.size() * sizeof(float2),
                                hipMemcpyHostToDevice, stream));
        SURR_HIP(hipMemsetAsync(m->err_flag, 0, 4, stream));
        SURR_HIP(hipStreamSynchronize(stream));
        SURR_HIP(hipEventCreateWithFlags(&m->staged, hipEventDisableTiming));
        return SURR_OK;
    };
    const surrogate_status st = body();
    if (stage) {
        hipStreamSynchronize(stream);
        hipFree(stage);
    }
    if (st != SURR_OK) {
        hipStreamSynchronize(stream);
        surrogate_free(m);
        return st;
    }
    *out = m;
    return SURR_OK;
}

surrogate_status surrogate_weight_file_config(const char* path, surrogate_config* out) {
    if (!path || !out) return fail(SURR_E_INVALID_ARG, "null argument");
    surr::host::MappedFile f;
    std::string why;
    if (!surr::host::map_file(path, &f, &why)) return fail(SURR_E_IO, why);
    surr::host::WeightFile wf;
    const bool ok = surr::host::parse_weight_file(f.data, f.size, f.size, &wf, &why);
    surr::host::unmap_file(&f);
    if (!ok) return fail(SURR_E_WEIGHTS, std::string(path) + ": " + why);
    *out = wf.cfg;
    return SURR_OK;
}

surrogate_status surrogate_load_weights(const char* path, hipStream_t stream, surrogate_model** out) {
    if (!path || !out) return fail(SURR_E_INVALID_ARG, "null argument");
    *out = nullptr;
    surr::host::MappedFile f;
    std::string why;
    if (!surr::host::map_file(path, &f, &why)) return fail(SURR_E_IO, why);
    surr::host::WeightFile wf;
    if (!surr::host::parse_weight_file(f.data, f.size, f.size, &wf, &why)) {
        surr::host::unmap_file(&f);
        return fail(SURR_E_WEIGHTS, std::string(path) + ": " + why);
    }
    // The file's fused w_qkv rows are the q, k and v matrices back to back: the tensor list
    // of surrogate_load_weights_tensors points into it.
    const surrogate_config& c = wf.cfg;
    const size_t e = c.dtype == SURR_BF16 ? 2 : 4, d = c.d_model;
    const size_t dq = (size_t)c.n_q_heads * c.head_dim, dkv = (size_t)c.n_kv_heads * c.head_dim;
    std::vector<const void*> t;
    t.reserve(3 + 9 * (size_t)c.n_layers);
    auto at = [&](int i) { return static_cast<const void*>(f.data + wf.tensors[i].offset); };
    t.push_back(at(0));
    for (int l = 0; l < c.n_layers; ++l) {
        const int b = 1 + 7 * l;
        const unsigned char* qkv = f.data + wf.tensors[b + 1].offset;
        t.push_back(at(b));                      // attn_norm
        t.push_back(qkv);                        // w_q
        t.push_back(qkv + dq * d * e);           // w_k
        t.push_back(qkv + (dq + dkv) * d * e);   // w_v
        for (int k = 2; k < 7; ++k) t.push_back(at(b + k));  // w_o, mlp_norm, w_gate, w_up, w_down
    }
    t.push_back(at(1 + 7 * c.n_layers));      // final_norm
    t.push_back(at(2 + 7 * c.n_layers));      // lm_head
    const surrogate_status st = surrogate_load_weights_tensors(&c, t.data(), (int32_t)t.size(), 0, stream, out);
    surr::host::unmap_file(&f);  // the load has synchronized the stream
    return st;
}

surrogate_status surrogate_get_config(const surrogate_model* m, surrogate_config* out) {
    if (!m || !out) return fail(SURR_E_INVALID_ARG, "null argument");
    *out = m->cfg;
    return SURR_OK;
}

surrogate_status surrogate_workspace_size(const surrogate_model* m, int32_t batch,
                                          int64_t total_tokens, int32_t max_len, size_t* bytes) {
    if (!m || !bytes) return fail(SURR_E_INVALID_ARG, "null argument");
    if (batch < 1 || total_tokens < batch || max_len < 1 || max_len > m->cfg.max_pos ||
        total_tokens > (int64_t)batch * max_len)
        return fail(SURR_E_SHAPE, "need 1 <= batch <= total_tokens <= batch * max_len, max_len <= max_pos");
    *bytes = layout(m, batch, total_tokens).total;
    return SURR_OK;
}

surrogate_status surrogate_score_pairs(surrogate_model* m, const int32_t* tokens_d,
                                       int64_t row_stride, const int32_t* lengths_h,
                                       int32_t batch, const int32_t* verdict_ids_h,
                                       int32_t n_verdict, void* workspace_d,
                                       size_t workspace_bytes, float* logprobs_d, float* probs_d,
                                       float* confidence_d, int32_t* verdict_d,
                                       hipStream_t stream) {
    if (!m || !tokens_d || !lengths_h || !verdict_ids_h || !workspace_d || !logprobs_d ||
        !confidence_d)
        return fail(SURR_E_INVALID_ARG, "null argument");
    if (batch < 1) return fail(SURR_E_INVALID_ARG, "batch must be >= 1");
    const surrogate_status vs = check_verdicts(m->cfg, verdict_ids_h, n_verdict);
    if (vs != SURR_OK) return vs;
    PassIO io;
    io.verdict_ids_h = verdict_ids_h;
    io.n_verdict = n_verdict;
    io.logprobs_d = logprobs_d;
    io.probs_d = probs_d;
    io.confidence_d = confidence_d;
    io.verdict_d = verdict_d;
    return run_pass(m, tokens_d, row_stride, lengths_h, batch, workspace_d, workspace_bytes, io, stream);
}

surrogate_status surrogate_prefix_build(surrogate_model* m, const int32_t* tokens_d,
                                        int64_t row_stride, const int32_t* lengths_h,
                                        int32_t n_prefix, void* workspace_d,
                                        size_t workspace_bytes, hipStream_t stream,
                                        surrogate_prefix_cache** out) {
    FaultScope fault_scope;
    if (!m || !tokens_d || !lengths_h || !workspace_d || !out) return fail(SURR_E_INVALID_ARG, "null argument");
    *out = nullptr;
    if (n_prefix < 1) return fail(SURR_E_INVALID_ARG, "n_prefix must be >= 1");
    auto* pc = new surrogate_prefix_cache();
    pc->model = m;
    pc->len.assign(lengths_h, lengths_h + n_prefix);
    pc->off.resize(n_prefix);
    pc->cap.resize(n_prefix);
    for (int g = 0; g < n_prefix; ++g) {
        pc->off[g] = (int32_t)pc->rows;
        pc->cap[g] = (std::max(lengths_h[g], 0) + 63) / 64 * 64;
        pc->rows += pc->cap[g];
    }
    // 32-bit DMA offsets over one kv head's V^T rows of the cache
    if (pc->rows * m->cfg.head_dim * 2 > (int64_t)UINT32_MAX || pc->rows > INT32_MAX) {
        delete pc;
        return fail(SURR_E_SHAPE, "prefixes too long for one cache");
    }
    pc->k_bytes = align_up((size_t)pc->rows * m->d_kv() * m->esz);
    pc->v_bytes = pc->k_bytes;
    const size_t bytes = (size_t)m->cfg.n_layers * (pc->k_bytes + pc->v_bytes);
    PassIO io;
    io.build = true;
    io.capture = pc;
    // arguments are checked before the cache memory is taken
    surrogate_status st = SURR_OK;
    for (int g = 0; g < n_prefix && st == SURR_OK; ++g)
        if (lengths_h[g] < 1 || lengths_h[g] > std::min<int64_t>(row_stride, m->cfg.max_pos - 1))
            st = fail(SURR_E_SHAPE, "length of prefix " + std::to_string(g) + " outside [1, min(row_stride, max_pos - 1)]");
    if (st == SURR_OK && (fault(kFaultAlloc) || hipMalloc(&pc->mem, bytes) != hipSuccess)) {
        pc->mem = nullptr;
        st = fail(SURR_E_OOM, "prefix cache of " + std::to_string(bytes) + " bytes");
    }
    if (st == SURR_OK)
        st = run_pass(m, tokens_d, row_stride, lengths_h, n_prefix, workspace_d, workspace_bytes, io, stream);
    if (st != SURR_OK) {
        if (pc->mem) {
            hipStreamSynchronize(stream);
            hipFree(pc->mem);
        }
        delete pc;
        return st;
    }
    *out = pc;
    return SURR_OK;
}

surrogate_status surrogate_score_suffixes(surrogate_model* m, const surrogate_prefix_cache* cache,
                                          const int32_t* prefix_id_h, const int32_t* tokens_d,
                                          int64_t row_stride, const int32_t* lengths_h,
                                          int32_t batch, const int32_t* verdict_ids_h,
                                          int32_t n_verdict, void* workspace_d,
                                          size_t workspace_bytes, float* logprobs_d,
                                          float* probs_d, float* confidence_d, int32_t* verdict_d,
                                          hipStream_t stream) {
    if (!m || !cache || !prefix_id_h || !tokens_d || !lengths_h || !verdict_ids_h ||
        !workspace_d || !logprobs_d || !confidence_d)
        return fail(SURR_E_INVALID_ARG, "null argument");
    if (cache->model != m) return fail(SURR_E_INVALID_ARG, "prefix cache was built by another model");
    if (batch < 1) return fail(SURR_E_INVALID_ARG, "batch must be >= 1");
    const surrogate_status vs = check_verdicts(m->cfg, verdict_ids_h, n_verdict);
    if (vs != SURR_OK) return vs;
    PassIO io;
    io.prefix = cache;
    io.prefix_id_h = prefix_id_h;
    io.verdict_ids_h = verdict_ids_h;
    io.n_verdict = n_verdict;
    io.logprobs_d = logprobs_d;
    io.probs_d = probs_d;
    io.confidence_d = confidence_d;
    io.verdict_d = verdict_d;
    return run_pass(m, tokens_d, row_stride, lengths_h, batch, workspace_d, workspace_bytes, io, stream);
}

surrogate_status surrogate_cache_create(surrogate_model* m, int32_t n_entries,
                                        const int32_t* capacity_h, surrogate_prefix_cache** out) {
    FaultScope fault_scope;
    if (!m || !capacity_h || !out) return fail(SURR_E_INVALID_ARG, "null argument");
    *out = nullptr;
    if (n_entries < 1) return fail(SURR_E_INVALID_ARG, "n_entries must be >= 1");
    auto* pc = new surrogate_prefix_cache();
    pc->model = m;
    pc->len.assign(n_entries, 0);
    pc->off.resize(n_entries);
    pc->cap.resize(n_entries);
    for (int g = 0; g < n_entries; ++g) {
        if (capacity_h[g] < 1 || capacity_h[g] > m->cfg.max_pos) {
            delete pc;
            return fail(SURR_E_SHAPE, "capacity of entry " + std::to_string(g) + " outside [1, max_pos]");
        }
        pc->off[g] = (int32_t)pc->rows;
        pc->cap[g] = (capacity_h[g] + 63) / 64 * 64;
        pc->rows += pc->cap[g];
    }
    if (pc->rows * m->cfg.head_dim * 2 > (int64_t)UINT32_MAX || pc->rows > INT32_MAX) {
        delete pc;
        return fail(SURR_E_SHAPE, "entries too long for one cache");
    }
    pc->k_bytes = align_up((size_t)pc->rows * m->d_kv() * m->esz);
    pc->v_bytes = pc->k_bytes;
    const size_t bytes = (size_t)m->cfg.n_layers * (pc->k_bytes + pc->v_bytes);
    if (fault(kFaultAlloc) || hipMalloc(&pc->mem, bytes) != hipSuccess) {
        delete pc;
        return fail(SURR_E_OOM, "cache of " + std::to_string(bytes) + " bytes");
    }
    // masked rows past an entry's length are still multiplied: they must be finite
    if (fault(kFaultLaunch) || hipMemset(pc->mem, 0, bytes) != hipSuccess) {
        hipFree(pc->mem);
        delete pc;
        return fail(SURR_E_HIP, "clearing the cache");
    }
    *out = pc;
    return SURR_OK;
}

surrogate_status surrogate_cache_lengths(const surrogate_prefix_cache* cache, int32_t* lengths_h) {
    if (!cache || !lengths_h) return fail(SURR_E_INVALID_ARG, "null argument");
    std::copy(cache->len.begin(), cache->len.end(), lengths_h);
    return SURR_OK;
}

surrogate_status surrogate_cache_reset(surrogate_prefix_cache* cache, const int32_t* entry_ids_h,
                                       int32_t n) {
    if (!cache || (n > 0 && !entry_ids_h)) return fail(SURR_E_INVALID_ARG, "null argument");
    for (int i = 0; i < n; ++i)
        if (entry_ids_h[i] < 0 || entry_ids_h[i] >= (int)cache->len.size())
            return fail(SURR_E_INVALID_ARG, "entry id outside [0, n_entries)");
    for (int i = 0; i < n; ++i) cache->len[entry_ids_h[i]] = 0;
    return SURR_OK;
}

surrogate_status surrogate_cache_extend(surrogate_model* m, surrogate_prefix_cache* cache,
                                        const int32_t* entry_ids_h, const int32_t* tokens_d,
                                        int64_t row_stride, const int32_t* lengths_h,
                                        int32_t batch, const int32_t* target_ids_h,
                                        void* workspace_d, size_t workspace_bytes,
                                        int32_t* next_token_d, float* target_logprob_d,
                                        hipStream_t stream) {
    if (!m || !cache || !entry_ids_h || !tokens_d || !lengths_h || !workspace_d)
        return fail(SURR_E_INVALID_ARG, "null argument");
    if (cache->model != m) return fail(SURR_E_INVALID_ARG, "cache was created for another model");
    if (target_logprob_d && !target_ids_h) return fail(SURR_E_INVALID_ARG, "target log-probs need target ids");
    PassIO io;
    io.prefix = cache;
    io.append = cache;
    io.prefix_id_h = entry_ids_h;
    io.target_ids_h = target_ids_h;
    io.next_token_d = next_token_d;
    io.target_lp_d = target_logprob_d;
    return run_pass(m, tokens_d, row_stride, lengths_h, batch, workspace_d, workspace_bytes, io, stream);
}

surrogate_status surrogate_prefix_cache_bytes(const surrogate_prefix_cache* cache, size_t* bytes) {
    if (!cache || !bytes) return fail(SURR_E_INVALID_ARG, "null argument");
    *bytes = (size_t)cache->model->cfg.n_layers * (cache->k_bytes + cache->v_bytes);
    return SURR_OK;
}

void surrogate_prefix_free(surrogate_prefix_cache* cache) {
    if (!cache) return;
    if (cache->mem) hipFree(cache->mem);
    delete cache;
}

surrogate_status surrogate_select(const float* confidence_d, int32_t n, surrogate_select_mode mode,
                                  float threshold, int32_t budget_k, int32_t* defer_idx_d,
                                  int32_t* accept_idx_d, int32_t* counts_d, hipStream_t stream) {
    if (!confidence_d || !defer_idx_d || !accept_idx_d || !counts_d)
        return fail(SURR_E_INVALID_ARG, "null argument");
    if (n < 1 || n > 65536) return fail(SURR_E_INVALID_ARG, "n must be in [1, 65536]");
    if (mode != SURR_SELECT_THRESHOLD && mode != SURR_SELECT_BUDGET && mode != SURR_SELECT_TOP_SCORE)
        return fail(SURR_E_INVALID_ARG, "unknown select mode");
    const bool ranked = mode != SURR_SELECT_THRESHOLD;
    if (ranked && budget_k < 0) return fail(SURR_E_INVALID_ARG, "budget_k must be >= 0");
    const int k = ranked ? std::min(budget_k, n) : 0;
    const int kmode = mode == SURR_SELECT_THRESHOLD ? 0 : mode == SURR_SELECT_BUDGET ? 1 : 2;
    SURR_HIP(surr::launch_select(confidence_d, n, kmode, threshold, k, defer_idx_d, accept_idx_d,
                                 counts_d, stream));
    return SURR_OK;
}

surrogate_status surrogate_forecast_head(const float* probs_d, int64_t n, int32_t n_bins,
                                         const double* bin_values_h, const double* bin_edges_h,
                                         const double* cutoffs_h, int32_t n_cutoffs,
                                         float* expected_speedup_d, float* discovery_d,
                                         hipStream_t stream) {
    using surr::kMaxBins;
    using surr::kMaxCutoffs;
    if (n < 0) return fail(SURR_E_INVALID_ARG, "n must be >= 0");
    if (n_bins < 1 || n_bins > kMaxBins) return fail(SURR_E_INVALID_ARG, "n_bins must be in [1, 16]");
    if (n_cutoffs < 0 || n_cutoffs > kMaxCutoffs) return fail(SURR_E_INVALID_ARG, "n_cutoffs must be in [0, 8]");
    if (!bin_values_h) return fail(SURR_E_INVALID_ARG, "null bin values");
    if (n > 0 && !probs_d && (expected_speedup_d || discovery_d)) return fail(SURR_E_INVALID_ARG, "null probs");
    if (n_cutoffs > 0 && (n_bins < 2 || !bin_edges_h || !cutoffs_h))
        return fail(SURR_E_INVALID_ARG, "discovery cutoffs need n_bins >= 2, edges and cutoffs");
    if (n > INT64_MAX / kMaxBins) return fail(SURR_E_INVALID_ARG, "n too large");
    surr::BinWeights w{};
    for (int b = 0; b < n_bins; ++b) {
        if (!std::isfinite(bin_values_h[b])) return fail(SURR_E_INVALID_ARG, "non-finite bin value");
        w.w[b][0] = (float)bin_values_h[b];
    }
    if (n_cutoffs > 0) {
        const int ne = n_bins - 1;
        for (int j = 0; j < ne; ++j) {
            if (!std::isfinite(bin_edges_h[j]) || !(bin_edges_h[j] > 0.0) ||
                (j > 0 && !(bin_edges_h[j] > bin_edges_h[j - 1])))
                return fail(SURR_E_INVALID_ARG, "bin edges must be finite, positive, strictly increasing");
        }
        for (int c = 0; c < n_cutoffs; ++c) {
            const double x = cutoffs_h[c];
            if (!(x >= bin_edges_h[0] && x <= bin_edges_h[ne - 1]))
                return fail(SURR_E_INVALID_ARG, "cutoff outside [first edge, last edge]");
            // Share of each bin's mass at or above x: the first bin lies wholly below any
            // admissible cutoff and the last wholly above it; interior bin (lo, hi] is
            // log-uniform, so the share above an inner x is ln(hi / x) / ln(hi / lo).
            w.w[0][1 + c] = 0.f;
            w.w[n_bins - 1][1 + c] = 1.f;
            for (int b = 1; b < n_bins - 1; ++b) {
                const double lo = bin_edges_h[b - 1], hi = bin_edges_h[b];
                double share;
                if (x <= lo) share = 1.0;
                else if (x >= hi) share = 0.0;
                else share = (std::log(hi) - std::log(x)) / (std::log(hi) - std::log(lo));
                w.w[b][1 + c] = (float)share;
            }
        }
    }
    SURR_HIP(surr::launch_forecast_head(probs_d, n, n_bins, w, n_cutoffs, expected_speedup_d,
                                        n_cutoffs > 0 ? discovery_d : nullptr, stream));
    return SURR_OK;
}

surrogate_status surrogate_evaluate_workspace_size(int32_t n, int32_t n_budgets, size_t* bytes) {
    if (!bytes) return fail(SURR_E_INVALID_ARG, "null argument");
    if (n < 1 || n > 65536) return fail(SURR_E_INVALID_ARG, "n must be in [1, 65536]");
    if (n_budgets < 1 || n_budgets > 8) return fail(SURR_E_INVALID_ARG, "n_budgets must be in [1, 8]");
    // expected speedups, per budget the two index lists, the counts, the partial rows
    *bytes = align_up(4 * (size_t)n) + align_up(8 * (size_t)n * n_budgets) +
             align_up(8 * (size_t)n_budgets) + align_up(surr::eval_partial_bytes(n, n_budgets));
    return SURR_OK;
}

surrogate_status surrogate_evaluate(const float* probs_d, const float* speedup_d, int32_t n,
                                    int32_t n_bins, const double* bin_values_h,
                                    const double* bin_edges_h, const double* budgets_h,
                                    int32_t n_budgets, void* workspace_d, size_t workspace_bytes,
                                    int32_t* bin_d, float* brier_d, float* crps_d,
                                    double* summary_d, hipStream_t stream) {
    EvalCall ec;
    const surrogate_status st = evaluate_args(probs_d, speedup_d, n, n_bins, bin_values_h, bin_edges_h,
                                              budgets_h, n_budgets, summary_d, &ec);
    if (st != SURR_OK) return st;
    if (!workspace_d) return fail(SURR_E_INVALID_ARG, "null argument");
    if (workspace_bytes < ec.need) return fail(SURR_E_WORKSPACE, "workspace needs " + std::to_string(ec.need) + " bytes");
    if (reinterpret_cast<uintptr_t>(workspace_d) % kAlign) return fail(SURR_E_INVALID_ARG, "workspace must be 256-byte aligned");
    return evaluate_launch(ec, probs_d, speedup_d, n, n_bins, n_budgets, static_cast<char*>(workspace_d),
                           bin_d, brier_d, crps_d, summary_d, stream);
}

surrogate_status surrogate_evaluate_noalloc(const float* probs_d, const float* speedup_d, int32_t n,
                                            int32_t n_bins, const double* bin_values_h,
                                            const double* bin_edges_h, const double* budgets_h,
                                            int32_t n_budgets, int32_t* bin_d, float* brier_d,
                                            float* crps_d, double* summary_d, hipStream_t stream) {
    EvalCall ec;
    surrogate_status st = evaluate_args(probs_d, speedup_d, n, n_bins, bin_values_h, bin_edges_h,
                                        budgets_h, n_budgets, summary_d, &ec);
    if (st != SURR_OK) return st;
    if (ec.need > kScratchBytes)
        return fail(SURR_E_WORKSPACE, "the call needs " + std::to_string(ec.need) +
                                          " bytes of scratch; the fixed scratch holds " +
                                          std::to_string(kScratchBytes));
    char* scratch_d = nullptr;
    st = device_scratch(&scratch_d);
    if (st != SURR_OK) return st;
    return evaluate_launch(ec, probs_d, speedup_d, n, n_bins, n_budgets, scratch_d, bin_d, brier_d,
                           crps_d, summary_d, stream);
}

surrogate_status surrogate_device_status(surrogate_model* m, hipStream_t stream) {
    if (!m) return fail(SURR_E_INVALID_ARG, "null argument");
    int32_t flag = 0;
    SURR_HIP(hipStreamSynchronize(stream));
    SURR_HIP(hipMemcpy(&flag, m->err_flag, 4, hipMemcpyDeviceToHost));
    if (flag) {
        SURR_HIP(hipMemset(m->err_flag, 0, 4));
        return fail(SURR_E_TOKEN_RANGE, "a token id outside [0, vocab) was read as id 0");
    }
    return SURR_OK;
}

surrogate_status surrogate_profile_enable(surrogate_model* m, int32_t enable) {
    if (!m) return fail(SURR_E_INVALID_ARG, "null argument");
    m->profiling = enable != 0;
    return SURR_OK;
}

surrogate_status surrogate_profile_collect(surrogate_model* m, double* ms_out, int64_t* launches_out) {
    if (!m || !ms_out || !launches_out) return fail(SURR_E_INVALID_ARG, "null argument");
    for (int p = 0; p < SURR_N_PHASES; ++p) {
        ms_out[p] = 0.0;
        launches_out[p] = 0;
    }
    for (const auto& r : m->rec) {
        float ms = 0.f;
        SURR_HIP(hipEventSynchronize(m->ev_pool[r.second + 1]));
        SURR_HIP(hipEventElapsedTime(&ms, m->ev_pool[r.second], m->ev_pool[r.second + 1]));
        ms_out[r.first] += ms;
        launches_out[r.first] += 1;
    }
    m->rec.clear();
    m->ev_used = 0;
    return SURR_OK;
}

const char* surrogate_status_string(surrogate_status s) {
    switch (s) {
        case SURR_OK: return "ok";
        case SURR_E_INVALID_ARG: return "invalid argument";
        case SURR_E_SHAPE: return "unsupported shape or length";
        case SURR_E_TOKEN_RANGE: return "token id out of range";
        case SURR_E_OOM: return "out of memory";
        case SURR_E_HIP: return "HIP runtime error";
        case SURR_E_WEIGHTS: return "weights do not match the config, or a malformed weight file";
        case SURR_E_IO: return "weight file unreadable";
        case SURR_E_WORKSPACE: return "workspace too small";
    }
    return "unknown status";
}

const char* surrogate_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
