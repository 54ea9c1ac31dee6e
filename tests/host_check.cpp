// CPU check of the runtime's host code (paper_2605_31464_amd/csrc/host.cpp), built by
// tests/test_host_sanitized.py with AddressSanitizer and UndefinedBehaviorSanitizer:
//  - the batch planner against a direct restatement of what it must produce, on random
//    batches (prefixes, appends, decode steps, length errors);
//  - the configuration checks on random configurations;
//  - the weight-file parser on valid files (argv) and on randomly corrupted copies of them,
//    which must be rejected or, if accepted, keep every tensor inside the file.
// Prints "host check ok" and exits 0, or prints the first failure and exits 1.
#include <algorithm>
#include <climits>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <fstream>
#include <random>
#include <string>
#include <vector>

#include "host.h"

using namespace surr::host;

namespace {

int g_fail = 0;

#define CHECK(cond, ...)                                 \
    do {                                                 \
        if (!(cond)) {                                   \
            std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
            std::fprintf(stderr, __VA_ARGS__);           \
            std::fprintf(stderr, "\n");                  \
            g_fail = 1;                                  \
            return;                                      \
        }                                                \
    } while (0)

void check_plan_case(std::mt19937_64& rng) {
    std::uniform_int_distribution<int> U(0, 1 << 30);
    PlanArgs a;
    const int B = 1 + U(rng) % 40;
    a.batch = B;
    a.max_pos = 64 + U(rng) % 4000;
    a.row_stride = 1 + U(rng) % 5000;
    a.q_tile = (U(rng) & 1) ? 128 : 64;
    a.dec_slice = 256;
    const int mode = U(rng) % 4;  // plain, prefix, append, build
    a.prefix = mode == 1 || mode == 2;
    a.append = mode == 2;
    a.build = mode == 3;
    a.dec_path = a.append && (U(rng) & 1);
    std::vector<int32_t> len(B), plen(B, 0), room(B, INT32_MAX);
    const bool make_bad = U(rng) % 5 == 0;
    for (int b = 0; b < B; ++b) {
        if (a.prefix) plen[b] = U(rng) % (a.max_pos / 2 + 1);
        if (a.append) room[b] = U(rng) % 3000;
        const int64_t cap = std::min<int64_t>(std::min<int64_t>(a.row_stride, room[b]),
                                              (int64_t)a.max_pos - plen[b] - (a.build ? 1 : 0));
        const bool one = a.dec_path && (U(rng) % 3 == 0);
        if (cap >= 1) len[b] = one ? 1 : 1 + U(rng) % (int)std::min<int64_t>(cap, 900);
        else len[b] = 1;  // no valid length exists: an error is expected
        if (make_bad && U(rng) % 7 == 0) len[b] = (U(rng) & 1) ? 0 : (int32_t)std::min<int64_t>(cap + 1 + U(rng) % 5, INT32_MAX);
    }
    a.lengths = len.data();
    a.plen = plen.data();
    a.room = room.data();

    int first_bad = -1;
    for (int b = 0; b < B && first_bad < 0; ++b) {
        const int64_t cap = std::min<int64_t>(std::min<int64_t>(a.row_stride, room[b]),
                                              (int64_t)a.max_pos - plen[b] - (a.build ? 1 : 0));
        if (len[b] < 1 || len[b] > cap) first_bad = b;
    }
    Plan p;
    std::string why;
    const surrogate_status st = plan_batch(a, &p, &why);
    if (first_bad >= 0) {
        CHECK(st == SURR_E_SHAPE, "expected a length error, got %d", (int)st);
        CHECK(why.find("prompt " + std::to_string(first_bad) + " ") != std::string::npos,
              "error names the wrong prompt: %s (want %d)", why.c_str(), first_bad);
        return;
    }
    CHECK(st == SURR_OK, "plan failed: %s", why.c_str());
    int64_t T = 0;
    for (int b = 0; b < B; ++b) T += len[b];
    CHECK(p.T == T, "T %lld != %lld", (long long)p.T, (long long)T);
    CHECK((int)p.cu.size() == B + 1 && p.cu[0] == 0, "cu size");
    for (int b = 0; b < B; ++b) {
        CHECK(p.cu[b + 1] - p.cu[b] == len[b], "cu step");
        CHECK(p.last[b] == p.cu[b + 1] - 1, "last row");
        CHECK(p.pos_last[b] == plen[b] + len[b] - 1, "last position");
        CHECK(p.vt_off[b + 1] - p.vt_off[b] == (len[b] + 63) / 64 * 64, "V^T block");
    }
    CHECK(p.max_len == *std::max_element(len.begin(), len.end()), "max_len");
    // decode prompts and their key slices, in prompt order
    std::vector<int> dec, rest;
    for (int b = 0; b < B; ++b) (a.dec_path && len[b] == 1 ? dec : rest).push_back(b);
    CHECK(p.dprompt == std::vector<int32_t>(dec.begin(), dec.end()), "decode prompts");
    CHECK((int)p.dfirst.size() == (int)dec.size() + 1 && p.dfirst[0] == 0, "decode firsts");
    size_t k = 0;
    for (size_t i = 0; i < dec.size(); ++i) {
        const int ns = (plen[dec[i]] + 1 + 255) / 256;
        CHECK(p.dfirst[i + 1] - p.dfirst[i] == ns, "slices of decode prompt %d", dec[i]);
        for (int s = 0; s < ns; ++s, ++k)
            CHECK(p.ditems[k].x == (int)i && p.ditems[k].y == s, "decode item");
    }
    CHECK(k == p.ditems.size(), "decode item count");
    // every (prompt, query tile) exactly once, longest key range first, ties in order
    std::vector<Int2> want;
    for (int b : rest)
        for (int t = 0; (int64_t)t * a.q_tile < len[b]; ++t) want.push_back({b, t});
    CHECK(p.work.size() == want.size(), "work items %zu != %zu", p.work.size(), want.size());
    auto kv = [&](const Int2& it) {
        return (int64_t)(plen[it.x] + 63) / 64 * 64 + std::min<int64_t>(len[it.x], (int64_t)(it.y + 1) * a.q_tile);
    };
    for (size_t i = 1; i < p.work.size(); ++i) {
        const int64_t k0 = kv(p.work[i - 1]), k1 = kv(p.work[i]);
        CHECK(k0 >= k1, "work list not longest first");
        if (k0 == k1)
            CHECK(p.work[i - 1].x < p.work[i].x ||
                  (p.work[i - 1].x == p.work[i].x && p.work[i - 1].y < p.work[i].y), "unstable order");
    }
    auto key = [](const Int2& v) { return ((int64_t)v.x << 32) | (uint32_t)v.y; };
    std::vector<int64_t> got_k, want_k;
    for (auto& v : p.work) got_k.push_back(key(v));
    for (auto& v : want) want_k.push_back(key(v));
    std::sort(got_k.begin(), got_k.end());
    std::sort(want_k.begin(), want_k.end());
    CHECK(got_k == want_k, "work items differ from the (prompt, tile) set");
    CHECK(p.work_last.size() == rest.size(), "last-row items");
    for (size_t i = 0; i < rest.size(); ++i)
        CHECK(p.work_last[i].x == rest[i] && p.work_last[i].y == (len[rest[i]] - 1) / a.q_tile, "last-row item");
}

void check_configs(std::mt19937_64& rng) {
    surrogate_config c7{28, 3584, 28, 4, 128, 18944, 131072, 8192, 10000.f, 1e-6f, SURR_BF16};
    std::string why;
    CHECK(valid_config(&c7, &why), "7B shape rejected: %s", why.c_str());
    surrogate_config bad = c7;
    bad.head_dim = 48;
    CHECK(!valid_config(&bad, &why), "head_dim 48 accepted");
    bad = c7;
    bad.n_kv_heads = 0;
    CHECK(!valid_config(&bad, &why), "zero kv heads accepted");
    bad = c7;
    bad.rope_base = 1.0f / 0.0f;
    CHECK(!valid_config(&bad, &why), "infinite rope base accepted");
    std::uniform_int_distribution<int> U(INT_MIN, INT_MAX);
    for (int i = 0; i < 20000; ++i) {
        surrogate_config c{};
        int32_t* f[] = {&c.n_layers, &c.d_model, &c.n_q_heads, &c.n_kv_heads, &c.head_dim, &c.d_ff,
                        &c.vocab, &c.max_pos};
        for (int32_t* x : f) *x = (i & 1) ? U(rng) : U(rng) % 300;
        c.dtype = U(rng) % 3;
        c.rope_base = (float)(U(rng) % 20000);
        c.rms_eps = 1e-6f;
        if (valid_config(&c, &why))
            for (int t = 0; t < 3 + 9 * std::min(c.n_layers, 3); ++t) {
                int64_t r, cc;
                int32_t dt;
                tensor_shape(&c, t, &r, &cc, &dt);
                CHECK(r >= 1 && cc >= 1, "tensor shape");
            }
    }
}

std::vector<unsigned char> read_file(const char* path) {
    std::ifstream f(path, std::ios::binary);
    return std::vector<unsigned char>((std::istreambuf_iterator<char>(f)), std::istreambuf_iterator<char>());
}

void check_parsed(const WeightFile& wf, uint64_t size) {
    uint64_t end = 0;
    for (const FileTensor& t : wf.tensors) {
        CHECK(t.offset % kFileAlign == 0, "misaligned tensor accepted");
        CHECK(t.offset >= end, "overlap accepted");
        CHECK(t.offset <= size && t.bytes <= size - t.offset, "tensor past the end accepted");
        end = t.offset + t.bytes;
    }
}

void check_file(const char* path, std::mt19937_64& rng, int rounds) {
    const std::vector<unsigned char> good = read_file(path);
    CHECK(good.size() > 16, "%s: empty", path);
    WeightFile wf;
    std::string why;
    CHECK(parse_weight_file(good.data(), good.size(), good.size(), &wf, &why), "%s: %s", path, why.c_str());
    check_parsed(wf, good.size());
    uint64_t H = 0;
    for (int i = 7; i >= 0; --i) H = (H << 8) | good[8 + i];
    // The parser reads the preamble and the header; the tensors matter only through the
    // file size.  Each round corrupts an exact-size heap copy of the first 16 + H bytes
    // (so a read past them is caught) and passes a file size of its own.
    const uint64_t head = 16 + H;
    std::uniform_int_distribution<uint64_t> U(0, UINT64_MAX);
    for (int r = 0; r < rounds; ++r) {
        std::vector<unsigned char> b(good.begin(), good.begin() + (ptrdiff_t)head);
        uint64_t size = good.size();
        const int kind = (int)(U(rng) % 5);
        if (kind == 0) {  // flip bytes of the header
            const int n = 1 + (int)(U(rng) % 8);
            for (int i = 0; i < n; ++i) b[16 + U(rng) % H] ^= (unsigned char)(1 + U(rng) % 255);
        } else if (kind == 1) {  // printable substitutions (keeps the JSON lexically plausible)
            const char alphabet[] = "0123456789-+.eE\"{}[],: tfn";
            const int n = 1 + (int)(U(rng) % 4);
            for (int i = 0; i < n; ++i) b[16 + U(rng) % H] = (unsigned char)alphabet[U(rng) % (sizeof(alphabet) - 1)];
        } else if (kind == 2) {  // the file truncated anywhere
            size = U(rng) % good.size();
            b.resize((size_t)std::min<uint64_t>(size, head));
        } else if (kind == 3) {  // another header length
            const uint64_t h2 = (U(rng) & 1) ? U(rng) : U(rng) % (H + 64);
            for (int i = 0; i < 8; ++i) b[8 + i] = (unsigned char)(h2 >> (8 * i));
        } else {  // a header length that ends inside the real header
            const uint64_t h2 = U(rng) % H;
            for (int i = 0; i < 8; ++i) b[8 + i] = (unsigned char)(h2 >> (8 * i));
        }
        WeightFile w2;
        std::string why2;
        unsigned char* copy = static_cast<unsigned char*>(std::malloc(b.size() ? b.size() : 1));
        if (!b.empty()) std::memcpy(copy, b.data(), b.size());
        const bool ok = parse_weight_file(copy, b.size(), size, &w2, &why2);
        std::free(copy);
        if (ok) check_parsed(w2, size);
        if (g_fail) return;
    }
}

}  // namespace

int main(int argc, char** argv) {
    std::mt19937_64 rng(12345);
    for (int i = 0; i < 20000 && !g_fail; ++i) check_plan_case(rng);
    if (!g_fail) check_configs(rng);
    for (int i = 1; i < argc && !g_fail; ++i) check_file(argv[i], rng, 3000);
    if (g_fail) return 1;
    std::printf("host check ok: 20000 plans, 20000 configs, %d weight files x 3000 corruptions\n",
                argc - 1);
    return 0;
}
