// Host-side checks of libmtp's argument validation, buffer sizing, weight
// layout and KV page planning, built with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code (device code is compiled
// as usual and never launched: every call below returns before any kernel
// or HIP memory operation).  Run by tests/test_abi_sanitize.py on the CPU;
// prints "abi sanitize ok" and exits 0, or names the failing check.
#include <algorithm>
#include <cstdint>
#include <utility>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "../include/mtp.h"

static int failures = 0;
#define CHECK(cond)                                                        \
    do {                                                                   \
        if (!(cond)) {                                                     \
            std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
            ++failures;                                                    \
        }                                                                  \
    } while (0)

// The 12-layer d1024 bf16 decoder with 8 heads, as a batch of `batch`.
static mtp_config valle(int batch) {
    mtp_config c{};
    c.n_layers = 12; c.d_model = 1024; c.n_heads = 16; c.d_ff = 4096; c.vocab = 1025; c.eos_id = 1024;
    c.n_phone = 512; c.max_pos = 4096; c.k_heads = 8; c.topk_max = 32; c.max_batch = batch; c.max_prompt = 450;
    c.max_new = 750; c.eos_min = 600; c.page_size = 16; c.num_pages = 0; c.dtype = MTP_DTYPE_BF16; c.flags = 0;
    return c;
}

// Device-looking pointers: 256-byte aligned, never dereferenced by the calls below.
static void* fake(uintptr_t k) { return reinterpret_cast<void*>(k << 20); }

int main() {
    // ---- sizes: valid configs of every workload shape, and their monotonicity
    {
        mtp_sizes s1{}, s32{};
        mtp_config c1 = valle(1), c32 = valle(32);
        CHECK(mtp_query_sizes(&c1, &s1) == MTP_OK);
        CHECK(mtp_query_sizes(&c32, &s32) == MTP_OK);
        CHECK(s1.weights_bytes == s32.weights_bytes);
        CHECK(s32.kv_bytes > s1.kv_bytes && s32.workspace_bytes > s1.workspace_bytes);
        CHECK(s1.logq_bytes == 1025ull * 1025 * 4);
        mtp_config nar = valle(8);
        nar.flags = MTP_FLAG_NAR; nar.k_heads = 7; nar.max_prompt = 1200; nar.max_new = 1;
        mtp_sizes sn{};
        CHECK(mtp_query_sizes(&nar, &sn) == MTP_OK);
        CHECK(sn.logq_bytes == 0);
        mtp_config tiny = valle(1);
        tiny.n_layers = 2; tiny.d_model = 256; tiny.n_heads = 4; tiny.d_ff = 1024; tiny.k_heads = 2;
        tiny.dtype = MTP_DTYPE_F32; tiny.max_prompt = 32; tiny.max_new = 64; tiny.eos_min = 64;
        CHECK(mtp_query_sizes(&tiny, &s1) == MTP_OK);
    }
    // ---- every rejected field, and NULL outputs
    {
        mtp_sizes s{};
        struct Bad { int off; int32_t v; } bad[] = {
            {offsetof(mtp_config, n_layers), 0},   {offsetof(mtp_config, d_model), 1000},
            {offsetof(mtp_config, n_heads), 15},   {offsetof(mtp_config, d_ff), 100},
            {offsetof(mtp_config, vocab), 1},      {offsetof(mtp_config, vocab), 5000},
            {offsetof(mtp_config, eos_id), 1025},  {offsetof(mtp_config, k_heads), 9},
            {offsetof(mtp_config, topk_max), 33},  {offsetof(mtp_config, max_batch), 0},
            {offsetof(mtp_config, max_new), 5000}, {offsetof(mtp_config, page_size), 8},
            {offsetof(mtp_config, page_size), 32}, {offsetof(mtp_config, num_pages), -1},
            {offsetof(mtp_config, dtype), 7},      {offsetof(mtp_config, flags), 64},
            {offsetof(mtp_config, max_prompt), 0}, {offsetof(mtp_config, n_phone), 0},
        };
        for (const Bad& b : bad) {
            mtp_config c = valle(1);
            std::memcpy(reinterpret_cast<char*>(&c) + b.off, &b.v, sizeof(int32_t));
            CHECK(mtp_query_sizes(&c, &s) == MTP_EINVAL);
        }
        mtp_config c = valle(1);
        CHECK(mtp_query_sizes(nullptr, &s) == MTP_EINVAL);
        CHECK(mtp_query_sizes(&c, nullptr) == MTP_EINVAL);
    }
    // ---- weight layout: aligned, disjoint, inside the buffer
    {
        mtp_config c = valle(1);
        mtp_sizes s{};
        CHECK(mtp_query_sizes(&c, &s) == MTP_OK);
        std::vector<std::pair<uint64_t, uint64_t>> spans;
        for (int t = 0; t < MTP_T_COUNT; ++t) {
            const int layers = (t >= MTP_T_LN1_G && t <= MTP_T_B_2) ? c.n_layers : 1;
            for (int l = 0; l < layers; ++l) {
                uint64_t off = 0, n = 0;
                CHECK(mtp_weight_offset(&c, t, l, &off, &n) == MTP_OK);
                CHECK(off % 256 == 0);
                const bool mat = t == MTP_T_EMB_PHONE || t == MTP_T_EMB_AC || t == MTP_T_POS || t == MTP_T_W_QKV ||
                                 t == MTP_T_W_O || t == MTP_T_W_1 || t == MTP_T_W_2 || t == MTP_T_W_HEADS;
                spans.emplace_back(off, off + n * (mat ? 2 : 4));
                CHECK(spans.back().second <= s.weights_bytes);
            }
        }
        std::sort(spans.begin(), spans.end());
        for (size_t i = 1; i < spans.size(); ++i) CHECK(spans[i - 1].second <= spans[i].first);
        uint64_t off = 0, n = 0;
        CHECK(mtp_weight_offset(&c, MTP_T_COUNT, 0, &off, &n) == MTP_EINVAL);
        CHECK(mtp_weight_offset(&c, -1, 0, &off, &n) == MTP_EINVAL);
        CHECK(mtp_weight_offset(&c, MTP_T_W_QKV, 12, &off, &n) == MTP_EINVAL);
    }
    // ---- context: buffer checks, calls out of order, prompt validation and
    //      KV page planning (all refused before any HIP call)
    {
        mtp_config c = valle(2);
        c.num_pages = 40;   // a small pool: two prompts + budgets do not fit
        mtp_buffers b{fake(1), static_cast<const float*>(fake(2)), fake(3), fake(4)};
        mtp_ctx* ctx = nullptr;
        mtp_buffers mis = b;
        mis.workspace = reinterpret_cast<char*>(fake(4)) + 64;
        CHECK(mtp_create(&c, &mis, nullptr, &ctx) == MTP_EINVAL && ctx == nullptr);
        mtp_buffers nul = b;
        nul.kv_pool = nullptr;
        CHECK(mtp_create(&c, &nul, nullptr, &ctx) == MTP_EINVAL);
        CHECK(mtp_create(&c, &b, nullptr, &ctx) == MTP_OK && ctx != nullptr);
        int32_t tok[64] = {0}, cnt[2] = {0, 0};
        float lg[16] = {0};
        CHECK(mtp_decode_step(ctx, 4, 4, tok, cnt) == MTP_ESTATE);
        CHECK(mtp_decode_step_async(ctx, 4, 4, nullptr, nullptr) == MTP_ESTATE);
        CHECK(mtp_force_tokens(ctx, tok, cnt) == MTP_ESTATE);
        CHECK(mtp_get_logits(ctx, lg) == MTP_ESTATE);
        CHECK(mtp_get_uniforms(ctx, lg) == MTP_ESTATE);
        CHECK(mtp_get_seq_state(ctx, cnt, nullptr, nullptr, nullptr) == MTP_ESTATE);
        double us = 0;
        CHECK(mtp_profile_replay(ctx, 0, 1, nullptr, 0, &us) == MTP_EINVAL);
        CHECK(mtp_profile_replay(ctx, MTP_KCLASS_GEMM_QKV, 1, fake(5), 100, &us) == MTP_EINVAL);
        CHECK(mtp_profile_replay(ctx, MTP_KCLASS_GEMM_QKV, 1, nullptr, 0, &us) == MTP_ESTATE);
        CHECK(mtp_set_selection(ctx, 2, 0) == MTP_EINVAL);
        CHECK(mtp_set_selection(ctx, MTP_LATTICE_UNION, 1) == MTP_OK);
        CHECK(mtp_set_sampling(ctx, MTP_SELECT_SAMPLE, 0.f, 1) == MTP_EINVAL);
        CHECK(mtp_set_sampling(ctx, MTP_SELECT_SAMPLE, 1e-39f, 1) == MTP_EINVAL);   // reciprocal overflows
        CHECK(mtp_set_sampling(ctx, MTP_SELECT_SAMPLE, 0.7f, 1) == MTP_OK);
        CHECK(mtp_set_sampling(ctx, 5, 1.f, 1) == MTP_EINVAL);
        CHECK(mtp_nar_run(ctx) == MTP_EINVAL);            // not a NAR context
        std::vector<int32_t> phon(300, 5), ac(900, 7);
        int32_t pl[3] = {100, 100, 100}, al[3] = {225, 225, 225};
        CHECK(mtp_prefill(ctx, 3, phon.data(), pl, ac.data(), al) == MTP_EINVAL);   // batch above max_batch
        CHECK(mtp_prefill(ctx, 0, phon.data(), pl, ac.data(), al) == MTP_EINVAL);
        int32_t al_long[2] = {400, 225};
        CHECK(mtp_prefill(ctx, 2, phon.data(), pl, ac.data(), al_long) == MTP_EINVAL);  // prompt above max_prompt
        int32_t zero[2] = {0, 0};
        CHECK(mtp_prefill(ctx, 2, phon.data(), zero, ac.data(), zero) == MTP_EINVAL);   // empty prompts
        ac[10] = 1024;                                                                   // EOS is not a prompt token
        CHECK(mtp_prefill(ctx, 2, phon.data(), pl, ac.data(), al) == MTP_EINVAL);
        ac[10] = 7;
        phon[3] = 512;
        CHECK(mtp_prefill(ctx, 2, phon.data(), pl, ac.data(), al) == MTP_EINVAL);
        phon[3] = 5;
        CHECK(mtp_prefill(ctx, 2, phon.data(), pl, ac.data(), al) == MTP_ENOMEM);       // 2 x 69 pages > 40
        CHECK(mtp_prefill(ctx, 2, nullptr, pl, ac.data(), al) == MTP_EINVAL);
        CHECK(std::strlen(mtp_last_error(ctx)) > 0);
        CHECK(mtp_reset(ctx) == MTP_OK);
        mtp_destroy(ctx);
        CHECK(std::strcmp(mtp_last_error(nullptr), "NULL context") == 0);
        for (int code = 1; code >= -5; --code) CHECK(mtp_strerror(code) != nullptr);
    }
    // ---- NAR context: preparation checks
    {
        mtp_config c = valle(2);
        c.flags = MTP_FLAG_NAR; c.k_heads = 7; c.max_prompt = 1200; c.max_new = 1;
        mtp_buffers b{fake(1), nullptr, fake(3), fake(4)};
        mtp_ctx* ctx = nullptr;
        CHECK(mtp_create(&c, &b, nullptr, &ctx) == MTP_OK);
        std::vector<int32_t> phon(100, 1), prompt(8 * 225, 3), a1(750, 9);
        int32_t pl[1] = {100}, ql[1] = {225}, tl[1] = {750}, tl_long[1] = {1000};
        CHECK(mtp_nar_prepare(ctx, 1, phon.data(), pl, prompt.data(), ql, a1.data(), tl_long) == MTP_EINVAL);
        prompt[5] = 1024;
        CHECK(mtp_nar_prepare(ctx, 1, phon.data(), pl, prompt.data(), ql, a1.data(), tl) == MTP_EINVAL);
        CHECK(mtp_nar_run(ctx) == MTP_ESTATE);
        int32_t codes[8];
        CHECK(mtp_nar_get_codes(ctx, codes) == MTP_ESTATE);
        CHECK(mtp_prefill(ctx, 1, phon.data(), pl, a1.data(), ql) == MTP_EINVAL);     // not an AR context
        mtp_destroy(ctx);
    }
    // ---- transition-table estimation: sizes and refusals before any launch
    {
        uint64_t bytes = 0, prev = 0;
        for (int64_t n = 0; n <= (int64_t)20 << 20; n += (int64_t)1 << 20) {
            CHECK(mtp_q_workspace_size(n, n / 297, 1025, &bytes) == MTP_OK);
            CHECK(bytes >= prev && bytes >= (uint64_t)n * 4);
            prev = bytes;
        }
        CHECK(mtp_q_workspace_size(-1, 0, 1025, &bytes) == MTP_EINVAL);
        CHECK(mtp_q_workspace_size(10, 1, 0, &bytes) == MTP_EINVAL);
        CHECK(mtp_q_workspace_size(10, 1, 9000, &bytes) == MTP_EINVAL);
        const int32_t* tk = static_cast<const int32_t*>(fake(6));
        const int64_t* of = static_cast<const int64_t*>(fake(7));
        uint32_t* counts = static_cast<uint32_t*>(fake(8));
        uint64_t* status = static_cast<uint64_t*>(fake(9));
        CHECK(mtp_q_count(tk, 100, of, 2, 1025, 1025, 0, counts, status, fake(10), 1 << 20, nullptr) == MTP_EINVAL);
        CHECK(mtp_q_count(tk, 100, of, 2, 1025, 1024, 4, counts, status, fake(10), 1 << 20, nullptr) == MTP_EINVAL);
        CHECK(mtp_q_count(tk + 1, 100, of, 2, 1025, 1024, 0, counts, status, fake(10), 1 << 20, nullptr) == MTP_EINVAL);
        CHECK(mtp_q_count(tk, 100, of, 2, 1025, 1024, 0, counts, status, nullptr, 1 << 20, nullptr) == MTP_EINVAL);
        CHECK(mtp_q_count(tk, 100, of, 2, 1025, 1024, 0, counts, status, fake(10), 1024, nullptr) == MTP_ENOMEM);
        CHECK(mtp_q_count_noalloc(tk, (int64_t)12 << 20, of, 40000, 1025, 1024, 0, counts, status, nullptr) ==
              MTP_ENOMEM);
        CHECK(mtp_q_count_noalloc(nullptr, 100, of, 2, 1025, 1024, 0, counts, status, nullptr) == MTP_EINVAL);
        CHECK(mtp_q_normalize(counts, 1025, -1.f, static_cast<float*>(fake(11)), nullptr) == MTP_EINVAL);
        CHECK(mtp_q_normalize(counts, 0, 1.f, static_cast<float*>(fake(11)), nullptr) == MTP_EINVAL);
    }
    if (failures) {
        std::fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    std::printf("abi sanitize ok\n");
    return 0;
}
