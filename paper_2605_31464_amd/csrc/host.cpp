// Host-only parts of the runtime (see host.h).
#include "host.h"

#include <algorithm>
#include <cerrno>
#include <climits>
#include <cmath>
#include <cstdlib>
#include <cstring>

#include <fcntl.h>
#include <sys/mman.h>
#include <sys/stat.h>
#include <unistd.h>

namespace surr {
namespace host {

// ---------------------------------------------------------------- configuration
bool valid_config(const surrogate_config* c, std::string* why) {
    auto bad = [&](const char* m) { *why = m; return false; };
    if (c->dtype != SURR_F32 && c->dtype != SURR_BF16) return bad("dtype must be SURR_F32 or SURR_BF16");
    if (c->n_layers < 1 || c->d_model < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1 ||
        c->d_ff < 1 || c->vocab < 1 || c->max_pos < 1)
        return bad("sizes must be positive");
    if (c->n_q_heads % c->n_kv_heads) return bad("n_q_heads must be a multiple of n_kv_heads");
    if (!(c->rope_base > 0.f) || !(c->rms_eps >= 0.f) || !std::isfinite(c->rope_base) ||
        !std::isfinite(c->rms_eps))
        return bad("rope_base > 0 and rms_eps >= 0 required (finite)");
    const int64_t dq = (int64_t)c->n_q_heads * c->head_dim;
    if (c->dtype == SURR_BF16) {
        if (c->head_dim != 64 && c->head_dim != 128) return bad("bf16 needs head_dim 64 or 128");
        if (c->d_model % 64 || dq % 64 || c->d_ff % 64) return bad("bf16 needs d_model, d_q, d_ff multiples of 64");
    } else {
        if (c->head_dim != 32 && c->head_dim != 64 && c->head_dim != 128)
            return bad("f32 needs head_dim 32, 64 or 128");
        if (c->d_model % 32 || dq % 32 || c->d_ff % 32) return bad("f32 needs d_model, d_q, d_ff multiples of 32");
    }
    if (c->vocab % 32) return bad("vocab must be a multiple of 32");
    if ((int64_t)c->max_pos * c->vocab <= 0) return bad("overflow");
    return true;
}

void tensor_shape(const surrogate_config* c, int idx, int64_t* rows, int64_t* cols, int32_t* dt) {
    const int64_t d = c->d_model, dq = (int64_t)c->n_q_heads * c->head_dim,
                  dkv = (int64_t)c->n_kv_heads * c->head_dim, ff = c->d_ff, V = c->vocab;
    const int last = 1 + 9 * c->n_layers;
    *dt = c->dtype;
    if (idx == 0 || idx == last + 1) { *rows = V; *cols = d; return; }
    if (idx == last) { *rows = 1; *cols = d; *dt = SURR_F32; return; }
    switch ((idx - 1) % 9) {
        case 0: case 5: *rows = 1; *cols = d; *dt = SURR_F32; return;
        case 1: *rows = dq; *cols = d; return;
        case 2: case 3: *rows = dkv; *cols = d; return;
        case 4: *rows = d; *cols = dq; return;
        case 6: case 7: *rows = ff; *cols = d; return;
        default: *rows = d; *cols = ff; return;
    }
}

// ---------------------------------------------------------------- JSON (header subset)
namespace {

struct Json {
    enum Kind { Null, Bool, Num, Str, Arr, Obj } kind = Null;
    bool b = false;
    double num = 0.0;
    std::string str;
    std::vector<Json> arr;
    std::vector<std::pair<std::string, Json>> obj;

    const Json* get(const char* key) const {
        if (kind != Obj) return nullptr;
        for (const auto& kv : obj)
            if (kv.first == key) return &kv.second;
        return nullptr;
    }
};

// Recursive descent over [p, end): objects, arrays, ASCII strings (the usual escapes, \u
// only below 0x80), numbers, true/false/null.  Nesting is bounded, every read is bounds
// checked, and duplicate object keys are rejected.
class JsonParser {
  public:
    JsonParser(const char* p, const char* end, std::string* why) : p_(p), end_(end), why_(why) {}

    bool document(Json* out) {
        if (!value(out, 0)) return false;
        ws();
        if (p_ != end_) return err("trailing bytes after the JSON header");
        return true;
    }

  private:
    const char* p_;
    const char* end_;
    std::string* why_;

    bool err(const char* m) {
        *why_ = m;
        return false;
    }
    void ws() {
        while (p_ < end_ && (*p_ == ' ' || *p_ == '\t' || *p_ == '\n' || *p_ == '\r')) ++p_;
    }
    bool lit(const char* s) {
        const size_t n = std::strlen(s);
        if ((size_t)(end_ - p_) < n || std::memcmp(p_, s, n) != 0) return err("bad JSON literal");
        p_ += n;
        return true;
    }
    bool string(std::string* out) {
        if (p_ >= end_ || *p_ != '"') return err("expected a JSON string");
        ++p_;
        out->clear();
        while (true) {
            if (p_ >= end_) return err("unterminated JSON string");
            const unsigned char ch = (unsigned char)*p_++;
            if (ch == '"') return true;
            if (ch < 0x20 || ch >= 0x80) return err("JSON header strings must be printable ASCII");
            if (ch != '\\') {
                out->push_back((char)ch);
                continue;
            }
            if (p_ >= end_) return err("unterminated JSON escape");
            const char e = *p_++;
            switch (e) {
                case '"': out->push_back('"'); break;
                case '\\': out->push_back('\\'); break;
                case '/': out->push_back('/'); break;
                case 'b': out->push_back('\b'); break;
                case 'f': out->push_back('\f'); break;
                case 'n': out->push_back('\n'); break;
                case 'r': out->push_back('\r'); break;
                case 't': out->push_back('\t'); break;
                case 'u': {
                    if (end_ - p_ < 4) return err("short \\u escape");
                    unsigned v = 0;
                    for (int i = 0; i < 4; ++i) {
                        const char h = *p_++;
                        v <<= 4;
                        if (h >= '0' && h <= '9') v |= (unsigned)(h - '0');
                        else if (h >= 'a' && h <= 'f') v |= (unsigned)(h - 'a' + 10);
                        else if (h >= 'A' && h <= 'F') v |= (unsigned)(h - 'A' + 10);
                        else return err("bad \\u escape");
                    }
                    if (v >= 0x80 || v < 0x20) return err("\\u escapes must be printable ASCII");
                    out->push_back((char)v);
                    break;
                }
                default: return err("bad JSON escape");
            }
        }
    }
    bool number(double* out) {
        const char* s = p_;
        if (p_ < end_ && *p_ == '-') ++p_;
        const char* digits = p_;
        while (p_ < end_ && *p_ >= '0' && *p_ <= '9') ++p_;
        if (p_ == digits) return err("bad JSON number");
        if (p_ < end_ && *p_ == '.') {
            ++p_;
            const char* f = p_;
            while (p_ < end_ && *p_ >= '0' && *p_ <= '9') ++p_;
            if (p_ == f) return err("bad JSON number");
        }
        if (p_ < end_ && (*p_ == 'e' || *p_ == 'E')) {
            ++p_;
            if (p_ < end_ && (*p_ == '+' || *p_ == '-')) ++p_;
            const char* x = p_;
            while (p_ < end_ && *p_ >= '0' && *p_ <= '9') ++p_;
            if (p_ == x) return err("bad JSON number");
        }
        if (p_ - s > 64) return err("JSON number too long");
        char buf[72];
        std::memcpy(buf, s, (size_t)(p_ - s));
        buf[p_ - s] = '\0';
        char* stop = nullptr;
        *out = std::strtod(buf, &stop);
        if (stop != buf + (p_ - s) || !std::isfinite(*out)) return err("bad JSON number");
        return true;
    }
    bool value(Json* out, int depth) {
        if (depth > 8) return err("JSON header nested too deeply");
        ws();
        if (p_ >= end_) return err("truncated JSON header");
        const char c = *p_;
        if (c == '{') {
            ++p_;
            out->kind = Json::Obj;
            ws();
            if (p_ < end_ && *p_ == '}') { ++p_; return true; }
            while (true) {
                ws();
                std::string key;
                if (!string(&key)) return false;
                if (out->get(key.c_str())) return err("duplicate key in the JSON header");
                ws();
                if (p_ >= end_ || *p_ != ':') return err("expected ':' in a JSON object");
                ++p_;
                out->obj.emplace_back(std::move(key), Json());
                if (!value(&out->obj.back().second, depth + 1)) return false;
                ws();
                if (p_ < end_ && *p_ == ',') { ++p_; continue; }
                if (p_ < end_ && *p_ == '}') { ++p_; return true; }
                return err("expected ',' or '}' in a JSON object");
            }
        }
        if (c == '[') {
            ++p_;
            out->kind = Json::Arr;
            ws();
            if (p_ < end_ && *p_ == ']') { ++p_; return true; }
            while (true) {
                out->arr.emplace_back();
                if (!value(&out->arr.back(), depth + 1)) return false;
                ws();
                if (p_ < end_ && *p_ == ',') { ++p_; continue; }
                if (p_ < end_ && *p_ == ']') { ++p_; return true; }
                return err("expected ',' or ']' in a JSON array");
            }
        }
        if (c == '"') {
            out->kind = Json::Str;
            return string(&out->str);
        }
        if (c == 't') { out->kind = Json::Bool; out->b = true; return lit("true"); }
        if (c == 'f') { out->kind = Json::Bool; out->b = false; return lit("false"); }
        if (c == 'n') { out->kind = Json::Null; return lit("null"); }
        out->kind = Json::Num;
        return number(&out->num);
    }
};

// A non-negative integer field below 2^53 (exact in a double).
bool as_count(const Json* j, uint64_t* out) {
    if (!j || j->kind != Json::Num || !(j->num >= 0.0) || j->num >= 9007199254740992.0 ||
        j->num != std::floor(j->num))
        return false;
    *out = (uint64_t)j->num;
    return true;
}

bool as_int32(const Json* j, int32_t* out) {
    uint64_t v = 0;
    if (!as_count(j, &v) || v > (uint64_t)INT32_MAX) return false;
    *out = (int32_t)v;
    return true;
}

bool as_dtype(const Json* j, int32_t* out) {
    if (!j || j->kind != Json::Str) return false;
    if (j->str == "bf16") { *out = SURR_BF16; return true; }
    if (j->str == "f32") { *out = SURR_F32; return true; }
    return false;
}

}  // namespace

const char kFileMagic[8] = {'S', 'U', 'R', 'R', 'W', 'G', 'T', '1'};

int32_t file_tensor_count(int32_t n_layers) { return 3 + 7 * n_layers; }

void file_tensor_spec(const surrogate_config& c, int idx, std::string* name, int32_t* dtype,
                      int64_t* rows, int64_t* cols) {
    const int64_t d = c.d_model, dq = (int64_t)c.n_q_heads * c.head_dim,
                  dkv = (int64_t)c.n_kv_heads * c.head_dim, ff = c.d_ff, V = c.vocab;
    const int last = 1 + 7 * c.n_layers;
    *dtype = c.dtype;
    if (idx == 0) { *name = "embed"; *rows = V; *cols = d; return; }
    if (idx == last) { *name = "final_norm"; *rows = 1; *cols = d; *dtype = SURR_F32; return; }
    if (idx == last + 1) { *name = "lm_head"; *rows = V; *cols = d; return; }
    const int l = (idx - 1) / 7;
    const std::string p = "layers." + std::to_string(l) + ".";
    switch ((idx - 1) % 7) {
        case 0: *name = p + "attn_norm"; *rows = 1; *cols = d; *dtype = SURR_F32; return;
        case 1: *name = p + "w_qkv"; *rows = dq + 2 * dkv; *cols = d; return;
        case 2: *name = p + "w_o"; *rows = d; *cols = dq; return;
        case 3: *name = p + "mlp_norm"; *rows = 1; *cols = d; *dtype = SURR_F32; return;
        case 4: *name = p + "w_gate"; *rows = ff; *cols = d; return;
        case 5: *name = p + "w_up"; *rows = ff; *cols = d; return;
        default: *name = p + "w_down"; *rows = d; *cols = ff; return;
    }
}

bool parse_weight_file(const unsigned char* data, uint64_t n, uint64_t file_size, WeightFile* out,
                       std::string* why) {
    auto bad = [&](const std::string& m) { *why = m; return false; };
    if (!data || n > file_size) return bad("bad buffer");
    if (n < 16) return bad("file shorter than its 16-byte preamble");
    if (std::memcmp(data, kFileMagic, 8) != 0) return bad("not a surrogate weight file (magic)");
    uint64_t H = 0;
    for (int i = 7; i >= 0; --i) H = (H << 8) | data[8 + i];
    if (H < 2 || H > kMaxHeaderBytes) return bad("header length out of range");
    if (H > n - 16) return bad("file truncated inside the JSON header");
    const char* js = reinterpret_cast<const char*>(data + 16);
    Json root;
    {
        std::string jwhy;
        JsonParser jp(js, js + H, &jwhy);
        if (!jp.document(&root)) return bad("JSON header: " + jwhy);
    }
    if (root.kind != Json::Obj) return bad("JSON header must be an object");
    const Json* fmt = root.get("format");
    if (!fmt || fmt->kind != Json::Str || fmt->str != "surrogate-weights") return bad("format must be \"surrogate-weights\"");
    uint64_t ver = 0;
    if (!as_count(root.get("version"), &ver) || ver != 1) return bad("version must be 1");
    const Json* cj = root.get("config");
    if (!cj || cj->kind != Json::Obj) return bad("missing config object");
    surrogate_config c{};
    struct { const char* key; int32_t* dst; } ints[] = {
        {"n_layers", &c.n_layers}, {"d_model", &c.d_model}, {"n_q_heads", &c.n_q_heads},
        {"n_kv_heads", &c.n_kv_heads}, {"head_dim", &c.head_dim}, {"d_ff", &c.d_ff},
        {"vocab", &c.vocab}, {"max_pos", &c.max_pos}};
    for (auto& f : ints)
        if (!as_int32(cj->get(f.key), f.dst)) return bad(std::string("config.") + f.key + " must be an integer in [0, 2^31)");
    const Json* rb = cj->get("rope_base");
    const Json* re = cj->get("rms_eps");
    if (!rb || rb->kind != Json::Num || !re || re->kind != Json::Num) return bad("config.rope_base and config.rms_eps must be numbers");
    c.rope_base = (float)rb->num;
    c.rms_eps = (float)re->num;
    if (!as_dtype(cj->get("dtype"), &c.dtype)) return bad("config.dtype must be \"bf16\" or \"f32\"");
    if (cj->obj.size() != 11) return bad("config has fields other than the 11 of surrogate_config");
    std::string cwhy;
    if (!valid_config(&c, &cwhy)) return bad("config: " + cwhy);
    if (c.n_layers > (INT32_MAX - 3) / 9) return bad("config: too many layers");

    const Json* tj = root.get("tensors");
    if (!tj || tj->kind != Json::Arr) return bad("missing tensors array");
    const int32_t nt = file_tensor_count(c.n_layers);
    if ((int64_t)tj->arr.size() != nt) return bad("expected " + std::to_string(nt) + " tensors");
    WeightFile wf;
    wf.cfg = c;
    wf.tensors.resize(nt);
    uint64_t end_prev = 16 + H;
    for (int i = 0; i < nt; ++i) {
        const Json& t = tj->arr[i];
        FileTensor& ft = wf.tensors[i];
        int32_t want_dt = 0;
        file_tensor_spec(c, i, &ft.name, &want_dt, &ft.rows, &ft.cols);
        const std::string at = "tensor " + std::to_string(i) + " (" + ft.name + ")";
        if (t.kind != Json::Obj || t.obj.size() != 4) return bad(at + ": needs exactly name, dtype, shape, offset");
        const Json* nm = t.get("name");
        if (!nm || nm->kind != Json::Str || nm->str != ft.name) return bad(at + ": wrong name or order");
        if (!as_dtype(t.get("dtype"), &ft.dtype) || ft.dtype != want_dt) return bad(at + ": wrong dtype");
        const Json* sh = t.get("shape");
        const bool norm = ft.rows == 1;
        if (!sh || sh->kind != Json::Arr || sh->arr.size() != (norm ? 1u : 2u)) return bad(at + ": wrong shape rank");
        uint64_t r = 0, cc = 0;
        if (norm) {
            if (!as_count(&sh->arr[0], &cc) || cc != (uint64_t)ft.cols) return bad(at + ": wrong shape");
        } else if (!as_count(&sh->arr[0], &r) || !as_count(&sh->arr[1], &cc) || r != (uint64_t)ft.rows ||
                   cc != (uint64_t)ft.cols) {
            return bad(at + ": wrong shape");
        }
        if (!as_count(t.get("offset"), &ft.offset)) return bad(at + ": offset must be an integer");
        if (ft.offset % kFileAlign) return bad(at + ": offset not a multiple of 4096");
        if (ft.offset < end_prev) return bad(at + ": overlaps the header or the previous tensor");
        ft.bytes = (uint64_t)ft.rows * (uint64_t)ft.cols * (ft.dtype == SURR_BF16 ? 2u : 4u);
        if (ft.offset > file_size || ft.bytes > file_size - ft.offset) return bad(at + ": extends past the end of the file");
        end_prev = ft.offset + ft.bytes;
    }
    *out = std::move(wf);
    return true;
}

bool map_file(const char* path, MappedFile* out, std::string* why) {
    *out = MappedFile{};
    const int fd = ::open(path, O_RDONLY | O_CLOEXEC);
    if (fd < 0) {
        *why = std::string("cannot open ") + path + ": " + std::strerror(errno);
        return false;
    }
    struct stat st;
    if (::fstat(fd, &st) != 0 || !S_ISREG(st.st_mode)) {
        *why = std::string(path) + " is not a readable regular file";
        ::close(fd);
        return false;
    }
    out->size = (uint64_t)st.st_size;
    if (out->size > 0) {
        void* p = ::mmap(nullptr, (size_t)out->size, PROT_READ, MAP_PRIVATE, fd, 0);
        if (p == MAP_FAILED) {
            *why = std::string("cannot map ") + path + ": " + std::strerror(errno);
            ::close(fd);
            *out = MappedFile{};
            return false;
        }
        out->data = static_cast<const unsigned char*>(p);
    }
    ::close(fd);  // the mapping stays valid
    return true;
}

void unmap_file(MappedFile* f) {
    if (f->data) ::munmap(const_cast<unsigned char*>(f->data), (size_t)f->size);
    *f = MappedFile{};
}

// ---------------------------------------------------------------- batch plan
surrogate_status plan_batch(const PlanArgs& a, Plan* p, std::string* why) {
    if (a.batch < 1) { *why = "batch must be >= 1"; return SURR_E_INVALID_ARG; }
    if (a.row_stride < 1) { *why = "row_stride must be >= 1"; return SURR_E_INVALID_ARG; }
    if (a.q_tile < 1 || a.dec_slice < 1) { *why = "bad tile sizes"; return SURR_E_INVALID_ARG; }
    const int B = a.batch;
    auto plen = [&](int b) { return a.plen ? a.plen[b] : 0; };
    auto room = [&](int b) { return a.room ? a.room[b] : INT32_MAX; };
    // a prompt's positions run to prefix length + length - 1 < max_pos; a prefix being
    // built leaves room for at least one continuing token
    int64_t T = 0;
    int32_t max_len = 0;
    for (int b = 0; b < B; ++b) {
        const int64_t cap = std::min<int64_t>(std::min<int64_t>(a.row_stride, room(b)),
                                              (int64_t)a.max_pos - plen(b) - (a.build ? 1 : 0));
        if (a.lengths[b] < 1 || a.lengths[b] > cap) {
            *why = "length of prompt " + std::to_string(b) +
                   (a.build ? " outside [1, min(row_stride, max_pos - 1)]"
                    : a.append ? " outside [1, min(row_stride, max_pos - length, capacity - length)]"
                    : a.prefix ? " outside [1, min(row_stride, max_pos - prefix length)]"
                               : " outside [1, min(row_stride, max_pos)]");
            return SURR_E_SHAPE;
        }
        max_len = std::max(max_len, a.lengths[b]);
        T += a.lengths[b];
    }
    if (T + 64 * (int64_t)B > INT32_MAX) {
        *why = "total tokens plus 64 per prompt exceed 2^31 - 1";
        return SURR_E_SHAPE;
    }
    p->T = T;
    p->max_len = max_len;
    p->cu.assign(B + 1, 0);
    p->last.assign(B, 0);
    p->pos_last.assign(B, 0);
    p->vt_off.assign(B + 1, 0);
    for (int b = 0; b < B; ++b) {
        p->cu[b + 1] = p->cu[b] + a.lengths[b];
        p->last[b] = p->cu[b + 1] - 1;
        p->pos_last[b] = plen(b) + a.lengths[b] - 1;  // the position the embedding gives that row
        p->vt_off[b + 1] = p->vt_off[b] + (a.lengths[b] + 63) / 64 * 64;
    }
    // One-token continuations of cached sequences (decode steps) take the split-key decode
    // attention; every other prompt takes the tiled kernel.  The choice depends on the
    // prompt alone, so a row's result does not depend on the batch.
    p->dprompt.clear();
    p->dfirst.assign(1, 0);
    p->ditems.clear();
    p->work.clear();
    p->work_last.clear();
    const int qt = a.q_tile;
    for (int b = 0; b < B; ++b) {
        if (a.dec_path && a.lengths[b] == 1) {
            const int ns = (plen(b) + 1 + a.dec_slice - 1) / a.dec_slice;
            for (int s = 0; s < ns; ++s) p->ditems.push_back({(int32_t)p->dprompt.size(), s});
            p->dprompt.push_back(b);
            p->dfirst.push_back((int32_t)p->ditems.size());
            continue;
        }
        for (int t = 0; (int64_t)t * qt < a.lengths[b]; ++t) p->work.push_back({b, t});
        p->work_last.push_back({b, (a.lengths[b] - 1) / qt});
    }
    // Longest key range first (a cached prefix counts in whole tiles), so the big causal
    // tiles start early; stable for a deterministic order.
    auto kv_len = [&](const Int2& it) {
        return (int64_t)(plen(it.x) + 63) / 64 * 64 + std::min<int64_t>(a.lengths[it.x], (int64_t)(it.y + 1) * qt);
    };
    std::stable_sort(p->work.begin(), p->work.end(),
                     [&](const Int2& x, const Int2& y) { return kv_len(x) > kv_len(y); });
    return SURR_OK;
}

}  // namespace host
}  // namespace surr
