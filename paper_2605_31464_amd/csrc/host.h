// Host-only parts of the runtime: configuration checks, tensor shapes, the weight-file
// header, and the per-call plan of a ragged batch.  Nothing here calls HIP, so the same
// source builds into the library and, with the host compiler's sanitizers, into a CPU
// check program.
#pragma once

#include <cstdint>
#include <string>
#include <utility>
#include <vector>

#include "surrogate.h"

namespace surr {
namespace host {

// ---------------------------------------------------------------- configuration
bool valid_config(const surrogate_config* c, std::string* why);

// Shape and element type of tensor `idx` of the pointer list surrogate_load_weights takes
// (embed; per layer attn_norm, w_q, w_k, w_v, w_o, mlp_norm, w_gate, w_up, w_down;
// final_norm; lm_head).
void tensor_shape(const surrogate_config* c, int idx, int64_t* rows, int64_t* cols, int32_t* dt);

// ---------------------------------------------------------------- weight file
// Layout (little-endian):
//   bytes [0, 8)        the magic "SURRWGT1"
//   bytes [8, 16)       uint64 H, the length of the JSON header
//   bytes [16, 16 + H)  the JSON header (ASCII)
//   tensor blobs at the offsets the header gives, each a multiple of 4096, in the file
//   order below, without overlap; bf16 tensors hold raw 16-bit patterns, f32 IEEE floats.
// Header: {"format": "surrogate-weights", "version": 1,
//          "config": {"n_layers": .., "d_model": .., "n_q_heads": .., "n_kv_heads": ..,
//                     "head_dim": .., "d_ff": .., "vocab": .., "max_pos": ..,
//                     "rope_base": .., "rms_eps": .., "dtype": "bf16" | "f32"},
//          "tensors": [{"name": .., "dtype": .., "shape": [rows, cols], "offset": ..}, ..]}
// File order: embed [V, d]; per layer l: layers.l.attn_norm [d], layers.l.w_qkv
// [d_q + 2 d_kv, d] (rows: q heads, then k heads, then v heads), layers.l.w_o [d, d_q],
// layers.l.mlp_norm [d], layers.l.w_gate [d_ff, d], layers.l.w_up [d_ff, d],
// layers.l.w_down [d, d_ff]; final_norm [d]; lm_head [V, d].  Norms are f32 with shape [d];
// matrices have the config's dtype.
constexpr uint64_t kFileAlign = 4096;
constexpr uint64_t kMaxHeaderBytes = 64ull << 20;
extern const char kFileMagic[8];

struct FileTensor {
    std::string name;
    int32_t dtype = 0;
    int64_t rows = 0, cols = 0;  // norms: rows = 1
    uint64_t offset = 0, bytes = 0;
};

struct WeightFile {
    surrogate_config cfg{};
    std::vector<FileTensor> tensors;  // in file order
};

int32_t file_tensor_count(int32_t n_layers);  // 3 + 7 n_layers
void file_tensor_spec(const surrogate_config& c, int idx, std::string* name, int32_t* dtype,
                      int64_t* rows, int64_t* cols);

// Parse and check a weight file whose first n bytes are `data` (n may be the whole file)
// and whose size is file_size.  On success every tensor lies inside the file.
bool parse_weight_file(const unsigned char* data, uint64_t n, uint64_t file_size, WeightFile* out,
                       std::string* why);

// A read-only mapping of a whole file (POSIX mmap); size 0 maps nothing.
struct MappedFile {
    const unsigned char* data = nullptr;
    uint64_t size = 0;
};
bool map_file(const char* path, MappedFile* out, std::string* why);
void unmap_file(MappedFile* f);

// ---------------------------------------------------------------- batch plan
struct Int2 {
    int32_t x, y;
};

struct PlanArgs {
    const int32_t* lengths = nullptr;  // [batch], host
    int32_t batch = 0;
    int64_t row_stride = 0;
    int32_t max_pos = 0;
    int32_t q_tile = 128;     // query rows per attention work item
    const int32_t* plen = nullptr;  // [batch] tokens already cached before each prompt (0: none)
    const int32_t* room = nullptr;  // [batch] tokens its cache entry can still take (appends)
    bool build = false;       // building a prefix cache: a prefix leaves room for one token
    bool append = false;      // prompts extend cache entries
    bool prefix = false;      // prompts continue cached prefixes
    bool dec_path = false;    // one-token continuations take the split-key decode attention
    int32_t dec_slice = 256;  // keys per slice of that attention
};

struct Plan {
    int64_t T = 0;  // total tokens
    int32_t max_len = 0;
    std::vector<int32_t> cu, last, pos_last, vt_off;  // [batch + 1], [batch], [batch], [batch + 1]
    std::vector<Int2> work, work_last;  // (prompt, query tile), longest key range first
    std::vector<int32_t> dprompt, dfirst;  // decode-attention prompts, first slice item of each
    std::vector<Int2> ditems;              // (decode prompt index, key slice)
};

// Checks the lengths (SURR_E_SHAPE with a message in *why) and builds the plan.
surrogate_status plan_batch(const PlanArgs& a, Plan* p, std::string* why);

}  // namespace host
}  // namespace surr
