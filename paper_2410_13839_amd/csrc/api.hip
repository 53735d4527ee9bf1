// libmtp: C ABI and host runtime of the MTP + Viterbi decode path.
//
// The context holds only host bookkeeping: the device layout of the
// caller's buffers, the KV page assignment, the launch plan of a decode step
// and the hipGraph instances that replay it.  Every step of the computation
// runs in the kernels of gemm.hip, attention.hip, rowops.hip and select.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <map>
#include <new>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/mtp.h"
#include "common.h"
#include "launch.h"

using namespace mtp;

namespace {

uint64_t align256(uint64_t x) { return (x + 255) & ~uint64_t(255); }

bool is_matrix(int t) {
    return t == MTP_T_EMB_PHONE || t == MTP_T_EMB_AC || t == MTP_T_POS || t == MTP_T_W_QKV || t == MTP_T_W_O ||
           t == MTP_T_W_1 || t == MTP_T_W_2 || t == MTP_T_W_HEADS;
}
bool is_layer_tensor(int t) { return t >= MTP_T_LN1_G && t <= MTP_T_B_2; }

bool is_nar(const mtp_config& c) { return (c.flags & MTP_FLAG_NAR) != 0; }

// The NAR module has one codebook table per codec layer (k_heads + 1 of
// them, vocab - 1 codes each), one head and one stage vector per predicted
// layer; the AR decoder has one codec table (vocab entries) and no stage
// vectors.
uint64_t tensor_numel(const mtp_config& c, int t) {
    const uint64_t d = c.d_model, f = c.d_ff, v = c.vocab;
    const uint64_t hv = is_nar(c) ? v - 1 : v;      // rows per head
    switch (t) {
    case MTP_T_EMB_PHONE: return (uint64_t)c.n_phone * d;
    case MTP_T_EMB_AC: return is_nar(c) ? (uint64_t)(c.k_heads + 1) * (v - 1) * d : v * d;
    case MTP_T_POS: return (uint64_t)c.max_pos * d;
    case MTP_T_LN1_G: case MTP_T_LN1_B: case MTP_T_B_O: case MTP_T_LN2_G: case MTP_T_LN2_B: case MTP_T_B_2:
    case MTP_T_LNF_G: case MTP_T_LNF_B: return d;
    case MTP_T_W_QKV: return 3 * d * d;
    case MTP_T_B_QKV: return 3 * d;
    case MTP_T_W_O: return d * d;
    case MTP_T_W_1: return f * d;
    case MTP_T_B_1: return f;
    case MTP_T_W_2: return d * f;
    case MTP_T_W_HEADS: return (uint64_t)c.k_heads * hv * d;
    case MTP_T_B_HEADS: return (uint64_t)c.k_heads * hv;
    case MTP_T_STAGE: return is_nar(c) ? (uint64_t)c.k_heads * d : 0;
    }
    return 0;
}

// bf16 Linear weights are stored in MFMA fragment order with the rows padded
// to a multiple of 16 (layout in mtp.h).
bool is_tiled(const mtp_config& c, int t) {
    return c.dtype == MTP_DTYPE_BF16 &&
           (t == MTP_T_W_QKV || t == MTP_T_W_O || t == MTP_T_W_1 || t == MTP_T_W_2 || t == MTP_T_W_HEADS);
}

uint64_t tensor_cols(const mtp_config& c, int t) { return t == MTP_T_W_2 ? (uint64_t)c.d_ff : (uint64_t)c.d_model; }

uint64_t tensor_bytes(const mtp_config& c, int t) {
    if (is_tiled(c, t)) {
        const uint64_t K = tensor_cols(c, t), N = tensor_numel(c, t) / K;
        return (N + 15) / 16 * 16 * K * 2;
    }
    return tensor_numel(c, t) * (is_matrix(t) ? (c.dtype == MTP_DTYPE_BF16 ? 2 : 4) : 4);
}

// Offsets of every tensor in packing order; returns total bytes.
uint64_t weight_layout(const mtp_config& c, std::vector<uint64_t>* glob, std::vector<uint64_t>* lay) {
    uint64_t off = 0;
    if (glob) glob->assign(MTP_T_COUNT, 0);
    if (lay) lay->assign((size_t)c.n_layers * MTP_T_COUNT, 0);
    for (int t = MTP_T_EMB_PHONE; t <= MTP_T_POS; ++t) {
        if (glob) (*glob)[t] = off;
        off = align256(off + tensor_bytes(c, t));
    }
    for (int l = 0; l < c.n_layers; ++l)
        for (int t = MTP_T_LN1_G; t <= MTP_T_B_2; ++t) {
            if (lay) (*lay)[(size_t)l * MTP_T_COUNT + t] = off;
            off = align256(off + tensor_bytes(c, t));
        }
    for (int t = MTP_T_LNF_G; t <= MTP_T_STAGE; ++t) {
        if (glob) (*glob)[t] = off;
        off = align256(off + tensor_bytes(c, t));
    }
    return off;
}

int validate(const mtp_config* c, std::string* why) {
    auto bad = [&](const char* m) { if (why) *why = m; return MTP_EINVAL; };
    if (!c) return bad("config is NULL");
    if (c->n_layers < 1 || c->n_layers > 256) return bad("n_layers out of range");
    if (c->d_model < 64 || c->d_model % 256 != 0 || c->d_model > 2048) return bad("d_model must be a multiple of 256 in 256..2048");
    if (c->n_heads * MTP_HEAD_DIM != c->d_model) return bad("d_model / n_heads must be 64");
    if (c->d_ff < 64 || c->d_ff % 256 != 0) return bad("d_ff must be a positive multiple of 256");
    if (c->vocab < 2 || c->vocab > 64 * 17) return bad("vocab out of range (2..1088)");
    if (c->eos_id < 0 || c->eos_id >= c->vocab) return bad("eos_id out of range");
    if (c->n_phone < 1) return bad("n_phone must be positive");
    if (c->k_heads < 1 || c->k_heads > MTP_MAX_HEADS_K) return bad("k_heads must be in 1..8");
    if (c->topk_max < 1 || c->topk_max > MTP_MAX_TOPK || c->topk_max >= c->vocab) return bad("topk_max must be in 1..32 and below vocab");
    if (c->max_batch < 1 || c->max_batch > 4096) return bad("max_batch out of range");
    if (c->max_prompt < 1) return bad("max_prompt must be positive");
    if (c->max_new < 1) return bad("max_new must be positive");
    if ((int64_t)c->max_prompt + c->max_new > c->max_pos) return bad("max_prompt + max_new exceeds max_pos");
    if ((int64_t)c->max_prompt + c->max_new > 16384) return bad("max_prompt + max_new exceeds 16384");
    // 16-key pages: one 16-key MFMA tile per page in the attention kernels
    // and the transposed V block of a page is one 16-byte operand per dimension
    if (c->page_size != 16) return bad("page_size must be 16");
    if (c->num_pages < 0) return bad("num_pages must be >= 0");
    if (c->dtype != MTP_DTYPE_F32 && c->dtype != MTP_DTYPE_BF16) return bad("unknown dtype");
    if ((c->flags & ~(MTP_FLAG_NO_GRAPH | MTP_FLAG_NAR)) != 0) return bad("unknown flags");
    if ((c->flags & MTP_FLAG_NAR) && c->k_heads > 7) return bad("a NAR module predicts at most 7 layers (k_heads <= 7)");
    return MTP_OK;
}

struct WsLayout {
    uint64_t rows, ids, tiles, last_row, state, btab, h, q, qh, u, attn, ffn, part, apart, kvnew, fsync, ffs, hz, z, logits,
        cand, ehat,
        u_states, u_m, u_ehat, u_delta, u_psi, smp_cfg, smp_u, codes, tgt_rows, nar_logits,
        delta, psi, slots, out_tok, out_cnt, hist, total;
    int64_t m_pre, m_dec, m_max, max_tiles, max_splits, maxp, num_pages;
    int act_bytes;
};

WsLayout ws_layout(const mtp_config& c) {
    WsLayout w{};
    const int64_t B = c.max_batch, d = c.d_model, F = c.d_ff, KH = c.k_heads, V = c.vocab, TK = c.topk_max;
    const int64_t H = c.n_heads;
    w.act_bytes = c.dtype == MTP_DTYPE_BF16 ? 2 : 4;
    w.m_pre = B * c.max_prompt;
    w.m_dec = B * KH;
    w.m_max = std::max(w.m_pre, w.m_dec);
    w.max_tiles = w.m_pre / MTP_ATTN_QT + B + 1;
    const int64_t max_ctx = (int64_t)c.max_prompt + (is_nar(c) ? 0 : c.max_new);
    w.max_splits = (max_ctx + 63) / 64;
    // the fused QKV + attention front of small batches writes one word per
    // workgroup of a head (up to 16) whatever the context
    const bool front = c.dtype == MTP_DTYPE_BF16 && w.m_dec <= 8 && d <= 1024 && !is_nar(c);
    if (front) w.max_splits = std::max<int64_t>(w.max_splits, 16);
    w.maxp = (max_ctx + c.page_size - 1) / c.page_size;
    w.num_pages = c.num_pages > 0 ? c.num_pages : B * w.maxp;
    uint64_t o = 0;
    auto take = [&](uint64_t bytes) { uint64_t r = o; o = align256(o + bytes); return r; };
    w.rows = take(w.m_max * sizeof(RowInfo));
    w.ids = take(w.m_pre * 4);
    w.tiles = take(w.max_tiles * 8);
    w.last_row = take(B * 4);
    w.state = take(B * sizeof(SeqState));
    w.btab = take(B * w.maxp * 4);
    w.h = take(w.m_max * d * 4);
    w.q = take(w.m_max * d * 4);
    // bf16 activations may be stored in fragment order: rows padded to 16
    const int64_t m_act = (w.m_max + 15) / 16 * 16;
    w.u = take(m_act * d * w.act_bytes);
    w.attn = take(m_act * d * w.act_bytes);
    w.ffn = take(m_act * F * w.act_bytes);
    // split-K partials: up to 4 splits of a prefill-sized GEMM, 8 of a decode one
    w.part = take(std::max(w.m_pre * 4, w.m_dec * (int64_t)MTP_SPLITK_MAX) * d * 4);
    w.apart = take(B * H * w.max_splits * MTP_ATTN_QT * 68 * 4);
    w.kvnew = take(front ? 2 * w.m_dec * d * 2 : 0);   // the pending rows' keys and values (bf16)
    // the chained front (qkv_front): its bf16 queries, and its hand-off
    // words (three sets of one flag per QKV column tile, a wait-overrun
    // count and the dealing check's 8 masks)
    const bool chain = c.dtype == MTP_DTYPE_BF16 && !is_nar(c);
    w.qh = take(chain ? w.m_dec * d * 2 : 0);
    w.fsync = take(chain ? (3 * (3 * d / 16) + 1 + 8) * 4 : 0);
    // the chained FFN (ffn_chain): three sets of 16 hidden rows, then a
    // wait-overrun count
    w.ffs = take(chain ? 3 * 16 * F * 2 + 4 : 0);
    w.hz = take(B * d * 4);
    w.z = take((B + 15) / 16 * 16 * d * w.act_bytes);
    w.logits = take(B * KH * V * 4);
    w.cand = take(B * KH * TK * 4);
    w.ehat = take(B * KH * TK * 4);
    w.delta = take(B * KH * TK * 4);
    w.psi = take(B * KH * TK * 4);
    w.slots = take(B * KH * 4);
    w.u_states = take(B * 64 * 4);                // union lattice (K * top_k <= 64 states)
    w.u_m = take(B * 4);
    w.u_ehat = take(B * MTP_MAX_HEADS_K * 64 * 4);
    w.u_delta = take(B * MTP_MAX_HEADS_K * 64 * 4);
    w.u_psi = take(B * MTP_MAX_HEADS_K * 64 * 4);
    w.smp_cfg = take(sizeof(SampleCfg));
    w.smp_u = take(B * MTP_MAX_HEADS_K * 4);
    w.out_tok = take(B * KH * 4);
    w.out_cnt = take(B * 4);
    w.hist = take(B * (int64_t)c.max_new * 4);
    const bool nar = is_nar(c);
    w.codes = take(nar ? w.m_pre * 8 * 4 : 0);                         // NAR: codec codes per row
    w.tgt_rows = take(nar ? w.m_pre * 4 : 0);                         // NAR: rows of the target positions
    w.nar_logits = take(nar ? (uint64_t)KH * w.m_pre * (V - 1) * 4 : 0);   // NAR: every stage's logits
    w.total = o;
    return w;
}

uint64_t kv_bytes(const mtp_config& c, const WsLayout& w) {
    return (uint64_t)c.n_layers * w.num_pages * 2 * c.n_heads * c.page_size * MTP_HEAD_DIM * (c.dtype == MTP_DTYPE_BF16 ? 2 : 4);
}

}  // namespace

struct mtp_ctx {
    mtp_config cfg;
    mtp_buffers buf;
    hipStream_t stream;
    WsLayout ws;
    std::vector<uint64_t> wglob, wlay;
    std::string err;
    // sequence bookkeeping
    bool prefilled = false;
    int B = 0;
    int q_pad = 0;               // pending rows per sequence for the next step
    int last_K = 0, last_topk = 0, last_lattice = 0, last_sample = 0;
    int split_len = 64, n_splits = 1;
    // how a small batch's layers start: 0 QKV and attention launches, 1 one
    // qkv_attn launch (on request), 2 one qkv_front launch
    int front = 0;
    int xcd_deal = -1;           // workgroups j and j + 8 share an XCD: -1 not yet checked, 0 no, 1 yes
    int front_spin = 100000;     // polls before a front hand-off wait gives up (MTP_FRONT_SPIN)
    // small batches: FFN1 and FFN2 in one launch (ffn_chain); -1 until the
    // first step that can use it fills the row sets with the sentinel
    int ffn_chain = 0;
    int ffn_ready = -1;
    int lattice = MTP_LATTICE_OWN, anchored = 0;   // selection options (mtp_set_selection)
    int sample = 0;              // mtp_set_sampling: draw the path instead of the best one
    SampleCfg h_smp{0, 1.0f, 0}; // copied to the workspace before the next step when dirty
    bool smp_dirty = true;
    int64_t plan_ctx = 0;        // longest prompt + budget of the batch (sizes the split plan)
    // NAR module
    bool nar_ready = false, nar_ran = false;
    int nar_rows = 0, nar_tiles = 0;
    std::vector<int32_t> h_codes, h_tgt, h_tlen;
    std::vector<int32_t> h_ids, h_last, h_btab;
    std::vector<RowInfo> h_rows;
    std::vector<int2> h_tiles;
    std::vector<SeqState> h_state;
    int n_pre_rows = 0, n_pre_tiles = 0;
    // graphs keyed by (K, top_k, q_pad, batch, split_len, n_splits, lattice, anchored, sampling, front)
    using StepKey = std::tuple<int, int, int, int, int, int, int, int, int, int, int>;
    std::map<StepKey, hipGraphExec_t> graphs;
    // every launch of each kernel class in the step of a key (arguments
    // captured by value), for replay timing
    using Launch = std::function<hipError_t(hipStream_t)>;
    struct StepLaunches { std::vector<Launch> cls[MTP_KCLASS_FFN_CHAIN + 1]; };
    std::map<StepKey, StepLaunches> step_launches;
    StepLaunches* recording = nullptr;
    StepKey last_key{};
    bool has_last = false;

    char* W() const { return (char*)buf.weights; }
    char* WS() const { return (char*)buf.workspace; }
    template <typename T> T* ws_ptr(uint64_t off) const { return reinterpret_cast<T*>(WS() + off); }
    const void* wt(int t) const { return W() + wglob[t]; }
    const void* lt(int l, int t) const { return W() + wlay[(size_t)l * MTP_T_COUNT + t]; }
    KVView kv(int layer) const {
        KVView v;
        v.pool = buf.kv_pool;
        v.block_table = ws_ptr<int32_t>(ws.btab);
        v.max_pages_per_seq = (int32_t)ws.maxp;
        v.num_pages = (int32_t)ws.num_pages;
        v.page_size = cfg.page_size;
        int sh = 0;
        while ((1 << sh) < cfg.page_size) ++sh;
        v.page_shift = sh;
        v.n_heads = cfg.n_heads;
        v.layer = layer;
        return v;
    }
};

namespace {

int hip_fail(mtp_ctx* c, hipError_t e, const char* where) {
    c->err = std::string(where) + ": " + hipGetErrorString(e);
    return MTP_EHIP;
}
#define HIPCHK(ctx, expr, where)                                  \
    do {                                                          \
        hipError_t _e = (expr);                                   \
        if (_e != hipSuccess) return hip_fail((ctx), _e, (where)); \
    } while (0)

int pick_splits(const mtp_ctx* c, int M, int N, int K) {
    if (c->cfg.dtype != MTP_DTYPE_BF16) return 1;
    const int64_t cap_rows = std::max(c->ws.m_pre * 4, c->ws.m_dec * (int64_t)MTP_SPLITK_MAX);
    const int gran = gemm_split_granule(1, M);
    const int tiles = gemm_tiles(M, N);
    int s = 1;
    while (s < MTP_SPLITK_MAX && tiles * s < 256 && K % (gran * s * 2) == 0 && (int64_t)M * s * 2 <= cap_rows) s *= 2;
    return s;
}

// Launch through `f` and, while a step is being recorded, keep it under class `kclass`.
hipError_t launch_rec(mtp_ctx* c, int kclass, std::function<hipError_t(hipStream_t)> f) {
    hipError_t e = f(c->stream);
    if (kclass > 0 && kclass <= MTP_KCLASS_FFN_CHAIN && c->recording) c->recording->cls[kclass].push_back(std::move(f));
    return e;
}

AttnDecArgs dec_attn_args(mtp_ctx* c, int l, int qt) {
    AttnDecArgs a{};
    a.dtype = c->cfg.dtype; a.B = c->B; a.Q = c->q_pad; a.qt = qt; a.st = c->ws_ptr<SeqState>(c->ws.state);
    a.q = c->ws_ptr<float>(c->ws.q); a.ldq = c->cfg.d_model; a.kv = c->kv(l);
    a.split_len = c->split_len; a.n_splits = c->n_splits; a.out = c->WS() + c->ws.attn; a.ldo = c->cfg.d_model;
    a.part = c->ws_ptr<float>(c->ws.apart); a.merge = 1;
    return a;
}

// Decode attention of layer l: MFMA kernel for bf16 caches, VALU kernel for
// fp32 caches.  With merge_launch, split partials are merged by a separate
// launch; otherwise the consumer merges them.
hipError_t decode_attention(mtp_ctx* c, int l, int qt, bool merge_launch, bool packed = false) {
    AttnDecArgs da = dec_attn_args(c, l, qt);
    da.merge = merge_launch ? 1 : 0;
    da.packed = packed ? 1 : 0;
    if (c->cfg.dtype != MTP_DTYPE_BF16)
        return launch_rec(c, MTP_KCLASS_ATTENTION, [da](hipStream_t s) { return attention_decode(s, da); });
    AttnMfmaArgs m{};
    m.mode = 0; m.n_tiles = c->B; m.Q = c->q_pad; m.qt = qt; m.st = da.st;
    m.q = da.q; m.ldq = da.ldq; m.kv = da.kv; m.split_len = da.split_len; m.n_splits = da.n_splits;
    m.out = (bf16_t*)da.out; m.ldo = da.ldo; m.part = da.part; m.packed = da.packed;
    hipError_t e = launch_rec(c, MTP_KCLASS_ATTENTION, [m](hipStream_t s) { return attention_mfma(s, m); });
    if (e != hipSuccess || !merge_launch) return e;
    return attention_decode_merge(c->stream, da);
}

// Whether the out-projection prologue merges the attention split partials
// itself (small batches) instead of a separate merge launch.
bool prologue_merge(const mtp_ctx* c, int rows) {
    return c->n_splits >= 2 && c->n_splits <= gemv_merge_max_splits(rows, c->cfg.d_model);
}

// One layer of the fused small-M decode trunk (bf16, B*Q <= 16 rows).  The
// out-projection and FFN2 leave four split-K partial sums, the first of which
// also carries the residual input and the bias; the next LayerNorm consumer
// (FFN1, the next layer's QKV, the heads) sums them into its input rows and
// writes the completed residual rows back to h for the next projection.
int run_layer_fused(mtp_ctx* c, int l, int rows, int qt) {
    const mtp_config& cf = c->cfg;
    const int d = cf.d_model, F = cf.d_ff;
    float* h = c->ws_ptr<float>(c->ws.h);
    float* part = c->ws_ptr<float>(c->ws.part);
    // FFN2's partials: past the out-projection's when the two FFN products
    // share a launch (the out-projection's are read in it)
    float* part2 = c->ffn_chain ? part + (size_t)4 * rows * d : part;
    GemvArgs g{};
    g.epi = EPI_QKV; g.M = rows; g.N = 3 * d; g.K = d;
    g.W = (const bf16_t*)c->lt(l, MTP_T_W_QKV); g.ldh = d; g.h_out = h;
    if (l == 0) {
        g.xmode = 2;
        g.emb = (const bf16_t*)c->wt(MTP_T_EMB_AC); g.pos = (const bf16_t*)c->wt(MTP_T_POS);
    } else {
        g.xmode = 1; g.part = part2; g.part_rows = rows; g.part_on = 1;
    }
    g.g = (const float*)c->lt(l, MTP_T_LN1_G); g.beta = (const float*)c->lt(l, MTP_T_LN1_B);
    g.st = c->ws_ptr<SeqState>(c->ws.state); g.Q = c->q_pad;
    g.bias = (const float*)c->lt(l, MTP_T_B_QKV); g.q = c->ws_ptr<float>(c->ws.q); g.kv = c->kv(l); g.d = d;
    bf16_t* kvnew = c->ws_ptr<bf16_t>(c->ws.kvnew);
    bool pm;
    if (c->front == 1) {
        // LN1 + QKV + attention over the cached keys in one launch; the
        // out-projection merges the splits and the chunk's own keys
        g.apart = c->ws_ptr<float>(c->ws.apart); g.qt = qt; g.split_len = c->split_len; g.n_splits = c->n_splits;
        g.kvnew = kvnew;
        HIPCHK(c, launch_rec(c, MTP_KCLASS_QKV_ATTN, [g](hipStream_t s) { return qkv_attn(s, g); }), "qkv + attention");
        pm = true;
    } else if (c->front == 2) {
        // LN1 + QKV, then the decode attention of each head as soon as its
        // columns are stored, in one launch
        pm = prologue_merge(c, rows);
        AttnDecArgs da = dec_attn_args(c, l, qt);
        AttnMfmaArgs m{};
        m.mode = 0; m.n_tiles = c->B; m.Q = c->q_pad; m.qt = qt; m.st = da.st;
        m.q = da.q; m.ldq = da.ldq; m.kv = da.kv; m.split_len = da.split_len; m.n_splits = da.n_splits;
        m.out = (bf16_t*)da.out; m.ldo = da.ldo; m.part = da.part; m.packed = 0;
        m.qh = g.qh = c->ws_ptr<bf16_t>(c->ws.qh);
        // flag sets: consecutive launches (layer order, then the next step's
        // layer 0) alternate sets 0 and 1; with an odd layer count the last
        // layer takes set 2
        const int L = cf.n_layers, nf = 3 * (d / 16);
        auto set_of = [L](int i) { return (L % 2 == 1 && i == L - 1) ? 2 : i % 2; };
        FrontSync fs{};
        unsigned* fw = c->ws_ptr<unsigned>(c->ws.fsync);
        fs.flags = fw + set_of(l) * nf; fs.next_flags = fw + set_of((l + 1) % L) * nf; fs.err = fw + 3 * nf;
        fs.tiles_per_mat = d / 16; fs.per_head = c->B * c->n_splits; fs.spin = c->front_spin;
        HIPCHK(c, launch_rec(c, MTP_KCLASS_QKV_FRONT, [g, m, fs](hipStream_t s) { return qkv_front(s, g, m, fs); }),
               "qkv + attention front");
    } else {
        HIPCHK(c, launch_rec(c, MTP_KCLASS_GEMM_QKV, [g](hipStream_t s) { return gemv(s, g); }), "qkv gemv");
        pm = prologue_merge(c, rows);
        HIPCHK(c, decode_attention(c, l, qt, !pm), "decode attention");
    }

    g = GemvArgs{};
    g.epi = EPI_PARTIAL; g.xmode = c->front == 1 ? 5 : pm ? 4 : 0; g.M = rows; g.N = d; g.K = d;
    g.W = (const bf16_t*)c->lt(l, MTP_T_W_O); g.x = (const bf16_t*)(c->WS() + c->ws.attn); g.ldx = d;
    g.st = c->ws_ptr<SeqState>(c->ws.state); g.Q = c->q_pad;
    g.apart = c->ws_ptr<float>(c->ws.apart); g.qt = qt; g.split_len = c->split_len; g.n_splits = c->n_splits;
    g.q = c->ws_ptr<float>(c->ws.q); g.kvnew = kvnew;
    g.h = h; g.ldh = d; g.bias = (const float*)c->lt(l, MTP_T_B_O); g.part_out = part;
    HIPCHK(c, launch_rec(c, MTP_KCLASS_GEMM_OPROJ, [g](hipStream_t s) { return gemv(s, g); }), "out-proj gemv");

    g = GemvArgs{};
    g.epi = EPI_GELU; g.xmode = 1; g.M = rows; g.N = F; g.K = d; g.ldh = d;
    g.W = (const bf16_t*)c->lt(l, MTP_T_W_1); g.part = part; g.part_rows = rows; g.part_on = 1; g.h_out = h;
    g.g = (const float*)c->lt(l, MTP_T_LN2_G); g.beta = (const float*)c->lt(l, MTP_T_LN2_B);
    g.bias = (const float*)c->lt(l, MTP_T_B_1); g.out = c->WS() + c->ws.ffn; g.ldo = F;
    GemvArgs g2{};
    g2.epi = EPI_PARTIAL; g2.xmode = 0; g2.M = rows; g2.N = d; g2.K = F;
    g2.W = (const bf16_t*)c->lt(l, MTP_T_W_2); g2.ldx = F;
    g2.h = h; g2.ldh = d; g2.bias = (const float*)c->lt(l, MTP_T_B_2); g2.part_out = part2;
    if (c->ffn_chain) {
        // row sets: consecutive launches (layer order, then the next step's
        // layer 0) alternate sets 0 and 1; with an odd layer count the last
        // layer takes set 2
        const int L = cf.n_layers;
        auto set_of = [L](int i) { return (L % 2 == 1 && i == L - 1) ? 2 : i % 2; };
        bf16_t* sets = c->ws_ptr<bf16_t>(c->ws.ffs);
        const size_t per_set = (size_t)16 * F;
        g.out = sets + set_of(l) * per_set;
        g2.x = (const bf16_t*)g.out; g2.part = part; g2.part_rows = rows;
        FfnSync fs{};
        fs.next = sets + set_of((l + 1) % L) * per_set;
        fs.err = reinterpret_cast<unsigned*>(sets + 3 * per_set);
        fs.spin = c->front_spin;
        HIPCHK(c, launch_rec(c, MTP_KCLASS_FFN_CHAIN, [g, g2, fs](hipStream_t s) { return ffn_chain(s, g, g2, fs); }),
               "ffn chain");
        return MTP_OK;
    }
    HIPCHK(c, launch_rec(c, MTP_KCLASS_GEMM_FFN1, [g](hipStream_t s) { return gemv(s, g); }), "ffn1 gemv");
    g2.x = (const bf16_t*)(c->WS() + c->ws.ffn);
    HIPCHK(c, launch_rec(c, MTP_KCLASS_GEMM_FFN2, [g2](hipStream_t s) { return gemv(s, g2); }), "ffn2 gemv");
    return MTP_OK;
}

// One trunk layer over `rows` rows whose row/tile metadata is already on the device.
int run_layer(mtp_ctx* c, int l, int rows, int n_tiles, int qt, int split_len, int n_splits, bool decode,
              bool bidir = false) {
    const mtp_config& cf = c->cfg;
    const int d = cf.d_model, F = cf.d_ff, dt = cf.dtype;
    hipStream_t st = c->stream;
    const int ab = c->ws.act_bytes;
    // bf16 activations travel between kernels in MFMA fragment order
    const int pk = dt == MTP_DTYPE_BF16 ? 1 : 0;
    GemmArgs g{};
    g.dtype = dt;
    // LN1 output u -> q, K/V cache
    g.epi = EPI_QKV; g.X = c->WS() + c->ws.u; g.ldx = d; g.M = rows; g.xpk = pk;
    g.W = c->lt(l, MTP_T_W_QKV); g.N = 3 * d; g.K = d; g.splits = 1;
    g.bias = (const float*)c->lt(l, MTP_T_B_QKV);
    g.q = c->ws_ptr<float>(c->ws.q); g.rows = c->ws_ptr<RowInfo>(c->ws.rows); g.kv = c->kv(l); g.d = d;
    HIPCHK(c, launch_rec(c, decode ? MTP_KCLASS_GEMM_QKV : 0, [g](hipStream_t s) { return gemm(s, g); }), "qkv gemm");
    // attention
    if (decode) {
        HIPCHK(c, decode_attention(c, l, qt, true, pk != 0), "decode attention");
    } else if (dt == MTP_DTYPE_BF16) {
        AttnMfmaArgs m{};
        m.mode = 1; m.n_tiles = n_tiles; m.Q = 0; m.qt = MTP_PREFILL_ROWS; m.st = c->ws_ptr<SeqState>(c->ws.state);
        m.tiles = c->ws_ptr<int2>(c->ws.tiles); m.rows = c->ws_ptr<RowInfo>(c->ws.rows);
        m.q = c->ws_ptr<float>(c->ws.q); m.ldq = d; m.kv = c->kv(l); m.split_len = 1 << 30; m.n_splits = 1;
        m.out = (bf16_t*)(c->WS() + c->ws.attn); m.ldo = d; m.part = nullptr; m.bidir = bidir ? 1 : 0;
        m.packed = pk;
        HIPCHK(c, attention_mfma(st, m), "prefill attention");
    } else {
        AttnArgs a{};
        a.dtype = dt; a.q = c->ws_ptr<float>(c->ws.q); a.ldq = d; a.rows = c->ws_ptr<RowInfo>(c->ws.rows);
        a.tiles = c->ws_ptr<int2>(c->ws.tiles); a.n_tiles = n_tiles; a.qt = qt; a.kv = c->kv(l);
        a.split_len = split_len; a.n_splits = n_splits; a.out = c->WS() + c->ws.attn; a.ldo = d;
        a.part = c->ws_ptr<float>(c->ws.apart);
        a.bidir = bidir ? 1 : 0; a.st = c->ws_ptr<SeqState>(c->ws.state);
        HIPCHK(c, attention(st, a), "attention");
    }
    // Prefill / NAR rows on the large-M kernel: the out-projection and FFN2
    // add their product and bias into the residual stream in their epilogue
    // (no K split: the split partials and the separate residual pass would
    // move three times the bytes), then a LayerNorm pass writes the next
    // product's rows.
    if (!decode && pk && gemm_resid_in_place(rows, d)) {
        float* h = c->ws_ptr<float>(c->ws.h);
        g = GemmArgs{};
        g.dtype = dt; g.epi = EPI_RESID; g.X = c->WS() + c->ws.attn; g.ldx = d; g.M = rows; g.xpk = pk;
        g.W = c->lt(l, MTP_T_W_O); g.N = d; g.K = d; g.splits = 1;
        g.bias = (const float*)c->lt(l, MTP_T_B_O); g.out = h; g.ldo = d;
        HIPCHK(c, gemm(st, g), "out-proj gemm");
        RowsLnArgs ln{};
        ln.dtype = dt; ln.n_rows = rows; ln.d = d; ln.h = h; ln.packed = pk; ln.u = c->WS() + c->ws.u;
        ln.ln_g = (const float*)c->lt(l, MTP_T_LN2_G); ln.ln_b = (const float*)c->lt(l, MTP_T_LN2_B);
        HIPCHK(c, rows_ln(st, ln), "ln2");
        g = GemmArgs{};
        g.dtype = dt; g.epi = EPI_GELU; g.X = c->WS() + c->ws.u; g.ldx = d; g.M = rows; g.xpk = pk; g.opk = pk;
        g.W = c->lt(l, MTP_T_W_1); g.N = F; g.K = d; g.splits = 1;
        g.bias = (const float*)c->lt(l, MTP_T_B_1); g.out = c->WS() + c->ws.ffn; g.ldo = F;
        HIPCHK(c, gemm(st, g), "ffn1 gemm");
        g = GemmArgs{};
        g.dtype = dt; g.epi = EPI_RESID; g.X = c->WS() + c->ws.ffn; g.ldx = F; g.M = rows; g.xpk = pk;
        g.W = c->lt(l, MTP_T_W_2); g.N = d; g.K = F; g.splits = 1;
        g.bias = (const float*)c->lt(l, MTP_T_B_2); g.out = h; g.ldo = d;
        HIPCHK(c, gemm(st, g), "ffn2 gemm");
        if (l + 1 < cf.n_layers) {
            ln.ln_g = (const float*)c->lt(l + 1, MTP_T_LN1_G); ln.ln_b = (const float*)c->lt(l + 1, MTP_T_LN1_B);
            HIPCHK(c, rows_ln(st, ln), "ln1");
        }
        return MTP_OK;
    }
    // out projection -> partials, residual + LN2
    const size_t sstride = (size_t)rows * d;
    g = GemmArgs{};
    g.dtype = dt; g.epi = EPI_PARTIAL; g.X = c->WS() + c->ws.attn; g.ldx = d; g.M = rows; g.xpk = pk;
    g.W = c->lt(l, MTP_T_W_O); g.N = d; g.K = d; g.splits = pick_splits(c, rows, d, d);
    g.out = c->WS() + c->ws.part; g.ldo = d; g.split_stride = sstride;
    HIPCHK(c, launch_rec(c, decode ? MTP_KCLASS_GEMM_OPROJ : 0, [g](hipStream_t s) { return gemm(s, g); }),
           "out-proj gemm");
    ResidArgs r{};
    r.dtype = dt; r.n_rows = rows; r.d = d; r.h = c->ws_ptr<float>(c->ws.h); r.part = c->ws_ptr<float>(c->ws.part);
    r.n_split = g.splits; r.split_stride = sstride; r.bias = (const float*)c->lt(l, MTP_T_B_O);
    r.ln_g = (const float*)c->lt(l, MTP_T_LN2_G); r.ln_b = (const float*)c->lt(l, MTP_T_LN2_B); r.u = c->WS() + c->ws.u;
    r.packed = pk;
    HIPCHK(c, launch_rec(c, decode ? MTP_KCLASS_RESID_LN : 0, [r](hipStream_t s) { return resid_ln(s, r); }),
           "resid+ln2");
    // FFN1 + GELU
    g = GemmArgs{};
    g.dtype = dt; g.epi = EPI_GELU; g.X = c->WS() + c->ws.u; g.ldx = d; g.M = rows; g.xpk = pk; g.opk = pk;
    g.W = c->lt(l, MTP_T_W_1); g.N = F; g.K = d; g.splits = 1;
    g.bias = (const float*)c->lt(l, MTP_T_B_1); g.out = c->WS() + c->ws.ffn; g.ldo = F;
    HIPCHK(c, launch_rec(c, decode ? MTP_KCLASS_GEMM_FFN1 : 0, [g](hipStream_t s) { return gemm(s, g); }), "ffn1 gemm");
    // FFN2 -> partials, residual + next LN1
    g = GemmArgs{};
    g.dtype = dt; g.epi = EPI_PARTIAL; g.X = c->WS() + c->ws.ffn; g.ldx = F; g.M = rows; g.xpk = pk;
    g.W = c->lt(l, MTP_T_W_2); g.N = d; g.K = F; g.splits = pick_splits(c, rows, d, F);
    g.out = c->WS() + c->ws.part; g.ldo = d; g.split_stride = sstride;
    HIPCHK(c, launch_rec(c, decode ? MTP_KCLASS_GEMM_FFN2 : 0, [g](hipStream_t s) { return gemm(s, g); }), "ffn2 gemm");
    r = ResidArgs{};
    r.dtype = dt; r.n_rows = rows; r.d = d; r.h = c->ws_ptr<float>(c->ws.h); r.part = c->ws_ptr<float>(c->ws.part);
    r.n_split = g.splits; r.split_stride = sstride; r.bias = (const float*)c->lt(l, MTP_T_B_2);
    if (l + 1 < cf.n_layers) {
        r.ln_g = (const float*)c->lt(l + 1, MTP_T_LN1_G); r.ln_b = (const float*)c->lt(l + 1, MTP_T_LN1_B);
        r.u = c->WS() + c->ws.u;
    }
    r.packed = pk;
    HIPCHK(c, launch_rec(c, decode ? MTP_KCLASS_RESID_LN : 0, [r](hipStream_t s) { return resid_ln(s, r); }),
           "resid+ln1");
    (void)ab;
    return MTP_OK;
}

int enqueue_step(mtp_ctx* c, int K, int top_k) {
    const mtp_config& cf = c->cfg;
    const int d = cf.d_model, dt = cf.dtype, B = c->B, Q = c->q_pad, V = cf.vocab;
    hipStream_t st = c->stream;
    const bool small = dt == MTP_DTYPE_BF16 && B * Q <= 16;
    int qt = 1;
    while (qt < Q) qt <<= 1;
    bool fin_part = false;                       // the heads' input is the last FFN2's partials
    if (Q > 0 && small) {
        for (int l = 0; l < cf.n_layers; ++l) {
            int rc = run_layer_fused(c, l, B * Q, qt);
            if (rc) return rc;
        }
        fin_part = true;
    } else if (Q > 0) {
        const int rows = B * Q;
        EmbedArgs e{};
        e.dtype = dt; e.mode = 0; e.n_rows = rows; e.Q = Q; e.st = c->ws_ptr<SeqState>(c->ws.state);
        e.ids = nullptr; e.rows = c->ws_ptr<RowInfo>(c->ws.rows); e.tiles = c->ws_ptr<int2>(c->ws.tiles);
        e.emb_phone = c->wt(MTP_T_EMB_PHONE); e.emb_ac = c->wt(MTP_T_EMB_AC); e.pos = c->wt(MTP_T_POS);
        e.ln_g = (const float*)c->lt(0, MTP_T_LN1_G); e.ln_b = (const float*)c->lt(0, MTP_T_LN1_B);
        e.d = d; e.h = c->ws_ptr<float>(c->ws.h); e.u = c->WS() + c->ws.u;
        e.packed = dt == MTP_DTYPE_BF16 ? 1 : 0;   // fragment order, as in run_layer
        HIPCHK(c, embed_ln(st, e), "embed");
        for (int l = 0; l < cf.n_layers; ++l) {
            int rc = run_layer(c, l, rows, B, qt, c->split_len, c->n_splits, true);
            if (rc) return rc;
        }
    }
    // the fused small-batch layers leave the last FFN2 as split-K partials,
    // which only the heads' LayerNorm prologue completes (B <= B * Q <= 16)
    if (dt == MTP_DTYPE_BF16 && (B <= 4 || fin_part)) {
        GemvArgs g{};
        g.epi = EPI_LOGITS; g.xmode = 3; g.M = B; g.N = K * V; g.K = d;
        g.W = (const bf16_t*)c->wt(MTP_T_W_HEADS); g.h = c->ws_ptr<float>(c->ws.h); g.ldh = d;
        g.part = c->ws_ptr<float>(c->ws.part) + (c->ffn_chain ? (size_t)4 * B * Q * d : 0);
        g.part_rows = B * Q; g.part_on = fin_part ? 1 : 0;
        g.hz = c->ws_ptr<float>(c->ws.hz); g.st = c->ws_ptr<SeqState>(c->ws.state); g.Q = Q;
        g.g = (const float*)c->wt(MTP_T_LNF_G); g.beta = (const float*)c->wt(MTP_T_LNF_B);
        g.bias = (const float*)c->wt(MTP_T_B_HEADS); g.out = c->WS() + c->ws.logits; g.ldo = K * V;
        HIPCHK(c, launch_rec(c, MTP_KCLASS_HEADS, [g](hipStream_t s) { return gemv(s, g); }), "heads gemv");
    } else {
        FinalArgs f{};
        f.dtype = dt; f.B = B; f.d = d; f.mode = 0; f.Q = Q; f.st = c->ws_ptr<SeqState>(c->ws.state);
        f.h = c->ws_ptr<float>(c->ws.h); f.hz = c->ws_ptr<float>(c->ws.hz);
        f.ln_g = (const float*)c->wt(MTP_T_LNF_G); f.ln_b = (const float*)c->wt(MTP_T_LNF_B); f.z = c->WS() + c->ws.z;
        f.packed = dt == MTP_DTYPE_BF16 ? 1 : 0;
        HIPCHK(c, final_ln(st, f), "final ln");
        GemmArgs g{};
        g.dtype = dt; g.epi = EPI_LOGITS; g.X = c->WS() + c->ws.z; g.ldx = d; g.M = B; g.xpk = f.packed;
        g.W = c->wt(MTP_T_W_HEADS); g.N = K * V; g.K = d; g.splits = 1;
        g.bias = (const float*)c->wt(MTP_T_B_HEADS); g.out = c->WS() + c->ws.logits; g.ldo = K * V;
        HIPCHK(c, launch_rec(c, MTP_KCLASS_HEADS, [g](hipStream_t s) { return gemm(s, g); }), "heads gemm");
    }
    SelectArgs s{};
    s.B = B; s.K = K; s.top_k = top_k; s.V = V; s.eos_id = cf.eos_id; s.eos_min = cf.eos_min; s.max_new = cf.max_new;
    s.Q = Q; s.logits = c->ws_ptr<float>(c->ws.logits); s.ld_logits = K * V; s.logq = c->buf.logq;
    s.st = c->ws_ptr<SeqState>(c->ws.state);
    s.cand = c->ws_ptr<int32_t>(c->ws.cand); s.ehat = c->ws_ptr<float>(c->ws.ehat); s.delta = c->ws_ptr<float>(c->ws.delta);
    s.psi = c->ws_ptr<int32_t>(c->ws.psi); s.slots = c->ws_ptr<int32_t>(c->ws.slots);
    s.out_tokens = c->ws_ptr<int32_t>(c->ws.out_tok); s.out_count = c->ws_ptr<int32_t>(c->ws.out_cnt);
    s.hist = c->ws_ptr<int32_t>(c->ws.hist); s.hist_ld = cf.max_new;
    s.lattice = c->lattice; s.anchored = c->anchored;
    s.u_states = c->ws_ptr<int32_t>(c->ws.u_states); s.u_m = c->ws_ptr<int32_t>(c->ws.u_m);
    s.u_ehat = c->ws_ptr<float>(c->ws.u_ehat); s.u_delta = c->ws_ptr<float>(c->ws.u_delta);
    s.u_psi = c->ws_ptr<int32_t>(c->ws.u_psi);
    s.sample = c->sample;
    s.smp = c->ws_ptr<SampleCfg>(c->ws.smp_cfg);
    s.smp_u = c->ws_ptr<float>(c->ws.smp_u);
    HIPCHK(c, launch_rec(c, MTP_KCLASS_SELECT, [s](hipStream_t q) { return select_fused(q, s); }), "select");
    return MTP_OK;
}

// Decode attention split plan for a step with Q pending rows per sequence,
// fixed per (batch, Q) so one captured graph serves every such step.  Small
// batches split the keys into short ranges so that they spread over many CUs
// (one CU streams only ~25 GB/s from HBM) and the out-projection merges the
// partials of its own heads; larger batches aim at ~192 (sequence, head,
// split) workgroups (one split once the batch's heads alone reach that, so
// no merge launch) and merge in a separate launch otherwise.
int plan_splits(mtp_ctx* c, int Q) {
    const mtp_config& cf = c->cfg;
    const int64_t max_ctx = std::max<int64_t>(c->plan_ctx, 1);
    const int64_t B = std::max(c->B, 1);
    const int64_t rows = B * std::max(Q, 1);
    const int merge_max =
        (cf.dtype == MTP_DTYPE_BF16 && rows <= 16) ? gemv_merge_max_splits((int)rows, cf.d_model) : 0;
    // small batches, on request: QKV and the attention over the cached keys
    // in one launch with G workgroups (key splits) per head.  Not the
    // default: every workgroup streams its head's 128 KB of query weights,
    // so the launch takes about as long as the two it replaces (10.7 vs
    // 5.97 + 5.13 us at batch 1, K = 4) and the out-projection's merge of
    // the chunk's own keys adds ~1 us (323 vs 312 us per step)
    c->front = 0;
    // small batches: FFN1 and FFN2 in one launch, whose FFN2 workgroups wait
    // for their K range of the hidden rows (at least two layers: consecutive
    // launches use different row sets)
    c->ffn_chain = 0;
    if (cf.dtype == MTP_DTYPE_BF16 && Q > 0 && !(cf.flags & MTP_FLAG_NAR) && rows <= 16 && cf.n_layers >= 2 &&
        ffn_chain_ok((int)rows, cf.d_model, cf.d_ff)) {
        const char* env = getenv("MTP_FFN_CHAIN");
        if (!(env && atoi(env) == 0) && c->ffn_ready != 0) {
            if (c->ffn_ready < 0) {
                // once per context, outside any capture: every row set
                // starts as the sentinel, the overrun count at zero
                char* fb = c->WS() + c->ws.ffs;
                const size_t sets = (size_t)3 * 16 * cf.d_ff * 2;
                HIPCHK(c, hipMemsetAsync(fb, 0xFF, sets, c->stream), "ffn row sets");
                HIPCHK(c, hipMemsetAsync(fb + sets, 0, 4, c->stream), "ffn row sets");
                c->ffn_ready = 1;
            }
            c->ffn_chain = 1;
        }
    }
    if (cf.dtype == MTP_DTYPE_BF16 && Q > 0 && !(cf.flags & MTP_FLAG_NAR)) {
        int G = 0;
        if (const char* env = getenv("MTP_QKV_ATTN")) G = atoi(env);
        if ((G == 8 || G == 16) && G <= c->ws.max_splits && G <= merge_max &&
            qkv_attn_ok((int)rows, cf.d_model, cf.n_heads, max_ctx, G)) {
            c->front = 1;
            c->split_len = qkv_attn_split_len(max_ctx, G);
            c->n_splits = G;
            return MTP_OK;
        }
    }
    // small batches: QKV and the decode attention in one launch whose
    // attention workgroups wait for their own head's columns (qkv_front).
    // Keys per split: 256 (one 16-key group per wave of 16), or 512 when
    // that keeps the splits within what the out-projection merges (at 256,
    // batch 1, K = 4: 244.7 us per step against 263.8 at 512, K = 8: 296.4
    // against 299.8, although 256 puts a few more workgroups in the launch
    // than there are CUs at the longest contexts).  At least two layers:
    // consecutive launches alternate their hand-off flag sets.
    const char* fenv = getenv("MTP_FRONT");
    if (cf.dtype == MTP_DTYPE_BF16 && Q > 0 && !(cf.flags & MTP_FLAG_NAR) && rows <= 16 && cf.n_layers >= 2 &&
        !(fenv && atoi(fenv) == 0)) {
        const int hpx = cf.n_heads / 8;
        int pick = 0;
        for (int sl2 : {256, 512}) {
            const int64_t n = (max_ctx + sl2 - 1) / sl2;
            if (n <= c->ws.max_splits && (n == 1 || n <= merge_max) &&
                qkv_front_ok((int)rows, cf.d_model, cf.n_heads, (int)B, sl2, (int)n)) {
                pick = sl2;
                break;
            }
        }
        if (fenv && (atoi(fenv) == 256 || atoi(fenv) == 512)) {
            const int sl2 = atoi(fenv);
            const int64_t n = (max_ctx + sl2 - 1) / sl2;
            pick = (n <= c->ws.max_splits && (n == 1 || n <= merge_max) &&
                    qkv_front_ok((int)rows, cf.d_model, cf.n_heads, (int)B, sl2, (int)n)) ? sl2 : 0;
        }
        if (pick && c->xcd_deal < 0) {
            // once per context, outside any capture: the hand-off words
            // start at zero, and the front needs workgroups j and j + 8 of
            // a launch on one XCD (the dispatcher deals them in turn from
            // where the previous launch stopped)
            unsigned* fw = c->ws_ptr<unsigned>(c->ws.fsync);
            unsigned* masks = fw + 3 * (3 * cf.d_model / 16) + 1;
            const size_t fbytes = (size_t)(3 * (3 * cf.d_model / 16) + 1 + 8) * 4;
            unsigned h_masks[8];
            HIPCHK(c, hipMemsetAsync(fw, 0, fbytes, c->stream), "front hand-off words");
            const int64_t n = (max_ctx + pick - 1) / pick;
            HIPCHK(c, xcd_deal_check(c->stream, masks, (int)(8 * hpx * (12 + B * n))), "dealing check");
            HIPCHK(c, hipMemcpyAsync(h_masks, masks, sizeof(h_masks), hipMemcpyDeviceToHost, c->stream),
                   "dealing check");
            HIPCHK(c, hipStreamSynchronize(c->stream), "dealing check");
            unsigned seen = 0;
            bool ok = true;
            for (unsigned m : h_masks) {
                ok = ok && m != 0 && (m & (m - 1)) == 0 && (seen & m) == 0;
                seen |= m;
            }
            c->xcd_deal = ok ? 1 : 0;
        }
        if (pick && c->xcd_deal == 1) {
            c->front = 2;
            c->split_len = pick;
            c->n_splits = (int)((max_ctx + pick - 1) / pick);
            return MTP_OK;
        }
    }
    int64_t sl;
    if (merge_max >= 2) {
        sl = std::max<int64_t>(128, ((max_ctx + merge_max - 1) / merge_max + 63) / 64 * 64);
    } else {
        const int64_t bh = B * cf.n_heads;
        const int64_t want = std::max<int64_t>(1, (192 + bh - 1) / bh);
        sl = (max_ctx + want - 1) / want;
        sl = std::max<int64_t>(64, (sl + 63) / 64 * 64);
    }
    if (const char* env = getenv("MTP_SPLIT_LEN")) {
        const int64_t v = atoll(env);
        if (v >= 32 && v % 32 == 0) sl = v;
    }
    sl = std::max<int64_t>(sl, ((max_ctx + 63) / 64 + 63) / 64 * 64);   // at most 64 splits
    const int64_t n = (max_ctx + sl - 1) / sl;
    if (n > 64 || n > c->ws.max_splits) { c->err = "attention split plan exceeds workspace"; return MTP_ENOMEM; }
    c->split_len = (int)sl;
    c->n_splits = (int)n;
    return MTP_OK;
}

int step_common(mtp_ctx* c, int K, int top_k) {
    if (!c) return MTP_EINVAL;
    if (!c->prefilled) { c->err = "decode step before prefill"; return MTP_ESTATE; }
    if (K < 1 || K > c->cfg.k_heads) { c->err = "K must be in 1..k_heads"; return MTP_EINVAL; }
    if (top_k < 1 || top_k > c->cfg.topk_max) { c->err = "top_k must be in 1..topk_max"; return MTP_EINVAL; }
    const bool use_graph = !(c->cfg.flags & MTP_FLAG_NO_GRAPH) && c->stream != nullptr;
    {
        const int rc0 = plan_splits(c, c->q_pad);
        if (rc0) return rc0;
    }
    if (c->lattice == MTP_LATTICE_UNION && K * top_k > 64) { c->err = "union lattice needs K * top_k <= 64"; return MTP_EINVAL; }
    if (c->sample && c->smp_dirty) {
        // stream-ordered before this step's launches (never inside a capture)
        // (waits for the copy, so that a later mtp_set_sampling cannot
        // change the source under it; only after a change of settings)
        HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.smp_cfg, &c->h_smp, sizeof(SampleCfg), hipMemcpyHostToDevice, c->stream),
               "sampling configuration");
        HIPCHK(c, hipStreamSynchronize(c->stream), "sampling configuration");
        c->smp_dirty = false;
    }
    const auto key = std::make_tuple(K, top_k, c->q_pad, c->B, c->split_len, c->n_splits, c->lattice, c->anchored,
                                     c->sample, c->front, c->ffn_chain);
    auto record = [&]() {
        mtp_ctx::StepLaunches& sl = c->step_launches[key];
        for (auto& v : sl.cls) v.clear();
        c->recording = &sl;
        const int r = enqueue_step(c, K, top_k);
        c->recording = nullptr;
        return r;
    };
    c->has_last = false;
    int rc;
    if (!use_graph) {
        rc = record();
    } else {
        auto it = c->graphs.find(key);
        if (it == c->graphs.end()) {
            hipGraph_t graph;
            HIPCHK(c, hipStreamBeginCapture(c->stream, hipStreamCaptureModeRelaxed), "begin capture");
            rc = record();
            hipError_t e = hipStreamEndCapture(c->stream, &graph);
            if (rc) { if (e == hipSuccess) (void)hipGraphDestroy(graph); return rc; }
            if (e != hipSuccess) return hip_fail(c, e, "end capture");
            hipGraphExec_t exec;
            e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
            (void)hipGraphDestroy(graph);
            if (e != hipSuccess) return hip_fail(c, e, "graph instantiate");
            it = c->graphs.emplace(key, exec).first;
        }
        HIPCHK(c, hipGraphLaunch(it->second, c->stream), "graph launch");
        rc = MTP_OK;
    }
    if (rc == MTP_OK) {
        c->q_pad = K;
        c->last_K = K;
        c->last_topk = top_k;
        c->last_lattice = c->lattice;
        c->last_sample = c->sample;
        c->last_key = key;
        c->has_last = true;
    }
    return rc;
}

}  // namespace

extern "C" {

const char* mtp_strerror(int code) {
    switch (code) {
    case MTP_OK: return "ok";
    case MTP_EINVAL: return "invalid argument";
    case MTP_ENOMEM: return "KV page pool or workspace too small";
    case MTP_ESTATE: return "call out of order";
    case MTP_EHIP: return "HIP runtime error";
    case MTP_ETIMEOUT: return "a bounded device-side wait ran out";
    }
    return "unknown error";
}

int mtp_query_sizes(const mtp_config* cfg, mtp_sizes* out) {
    if (!out) return MTP_EINVAL;
    int rc = validate(cfg, nullptr);
    if (rc) return rc;
    WsLayout w = ws_layout(*cfg);
    out->weights_bytes = weight_layout(*cfg, nullptr, nullptr);
    out->logq_bytes = is_nar(*cfg) ? 0 : (uint64_t)cfg->vocab * cfg->vocab * 4;
    out->kv_bytes = kv_bytes(*cfg, w);
    out->workspace_bytes = w.total;
    return MTP_OK;
}

int mtp_weight_offset(const mtp_config* cfg, int tensor, int layer, uint64_t* offset_bytes, uint64_t* numel) {
    int rc = validate(cfg, nullptr);
    if (rc) return rc;
    if (tensor < 0 || tensor >= MTP_T_COUNT) return MTP_EINVAL;
    std::vector<uint64_t> g, l;
    weight_layout(*cfg, &g, &l);
    uint64_t off;
    if (is_layer_tensor(tensor)) {
        if (layer < 0 || layer >= cfg->n_layers) return MTP_EINVAL;
        off = l[(size_t)layer * MTP_T_COUNT + tensor];
    } else {
        off = g[tensor];
    }
    if (offset_bytes) *offset_bytes = off;
    if (numel) *numel = tensor_numel(*cfg, tensor);
    return MTP_OK;
}

int mtp_create(const mtp_config* cfg, const mtp_buffers* bufs, void* hip_stream, mtp_ctx** out) {
    if (!out || !bufs) return MTP_EINVAL;
    *out = nullptr;
    int rc = validate(cfg, nullptr);
    if (rc) return rc;
    if (!bufs->weights || (!bufs->logq && !is_nar(*cfg)) || !bufs->kv_pool || !bufs->workspace) return MTP_EINVAL;
    auto aligned = [](const void* p) { return ((uintptr_t)p & 255) == 0; };
    if (!aligned(bufs->weights) || !aligned(bufs->logq) || !aligned(bufs->kv_pool) || !aligned(bufs->workspace))
        return MTP_EINVAL;
    mtp_ctx* c = new (std::nothrow) mtp_ctx();
    if (!c) return MTP_ENOMEM;
    c->cfg = *cfg;
    c->buf = *bufs;
    if (const char* env = getenv("MTP_FRONT_SPIN")) c->front_spin = std::max(0, atoi(env));
    c->stream = (hipStream_t)hip_stream;
    c->ws = ws_layout(*cfg);
    weight_layout(*cfg, &c->wglob, &c->wlay);
    *out = c;
    return MTP_OK;
}

int mtp_prefill(mtp_ctx* c, int B, const int32_t* phon, const int32_t* phon_len, const int32_t* ac,
                const int32_t* ac_len) {
    if (!c) return MTP_EINVAL;
    if (is_nar(c->cfg)) { c->err = "a NAR context has no AR prefill"; return MTP_EINVAL; }
    const mtp_config& cf = c->cfg;
    if (B < 1 || B > cf.max_batch) { c->err = "batch out of range"; return MTP_EINVAL; }
    if (!phon_len || !ac_len || !ac) { c->err = "NULL prompt array"; return MTP_EINVAL; }
    int64_t n_phon = 0, n_ac = 0;
    for (int b = 0; b < B; ++b) {
        if (phon_len[b] < 0 || ac_len[b] < 0 || phon_len[b] + ac_len[b] < 1 || phon_len[b] + ac_len[b] > cf.max_prompt) {
            c->err = "prompt length out of range";
            return MTP_EINVAL;
        }
        n_phon += phon_len[b];
        n_ac += ac_len[b];
    }
    if (n_phon > 0 && !phon) { c->err = "NULL phoneme array"; return MTP_EINVAL; }
    for (int64_t i = 0; i < n_phon; ++i)
        if (phon[i] < 0 || phon[i] >= cf.n_phone) { c->err = "phoneme id out of range"; return MTP_EINVAL; }
    for (int64_t i = 0; i < n_ac; ++i)
        if (ac[i] < 0 || ac[i] >= cf.vocab - 1) { c->err = "acoustic id out of range"; return MTP_EINVAL; }
    // KV pages: each sequence reserves prompt + max_new positions; pages are
    // handed out round-robin from the top of the pool so that consecutive
    // pages of a sequence are not adjacent in memory.
    const int64_t maxp = c->ws.maxp;
    std::vector<int> need(B);
    int64_t total_pages = 0;
    for (int b = 0; b < B; ++b) {
        need[b] = (int)((phon_len[b] + ac_len[b] + (int64_t)cf.max_new + cf.page_size - 1) / cf.page_size);
        total_pages += need[b];
    }
    if (total_pages > c->ws.num_pages) { c->err = "KV page pool exhausted"; return MTP_ENOMEM; }
    c->h_btab.assign((size_t)B * maxp, 0);
    int next = (int)c->ws.num_pages - 1;
    for (int p = 0; p < maxp; ++p)
        for (int b = 0; b < B; ++b)
            if (p < need[b]) c->h_btab[(size_t)b * maxp + p] = next--;
    // packed rows and attention tiles
    c->h_ids.clear(); c->h_rows.clear(); c->h_tiles.clear(); c->h_last.assign(B, 0); c->h_state.assign(B, SeqState{});
    int64_t op = 0, oa = 0;
    for (int b = 0; b < B; ++b) {
        const int len = phon_len[b] + ac_len[b];
        const int row0 = (int)c->h_ids.size();
        for (int i = 0; i < phon_len[b]; ++i) c->h_ids.push_back(phon[op++]);
        for (int i = 0; i < ac_len[b]; ++i) c->h_ids.push_back(ac[oa++]);
        for (int i = 0; i < len; ++i) c->h_rows.push_back(RowInfo{b, i});
        const int trows = (cf.dtype == MTP_DTYPE_BF16) ? MTP_PREFILL_ROWS : MTP_ATTN_QT;
        for (int i0 = 0; i0 < len; i0 += trows) c->h_tiles.push_back(make_int2(row0 + i0, std::min(trows, len - i0)));
        c->h_last[b] = row0 + len - 1;
        SeqState s{};
        s.ctx_len = len; s.pend_len = 0; s.gen = 0; s.done = 0; s.phon_len = phon_len[b]; s.prompt_len = len;
        s.last_tok = ac_len[b] > 0 ? ac[oa - 1] : -1;     // the acoustic prompt's last codec token
        c->h_state[b] = s;
    }
    const int rows = (int)c->h_ids.size();
    const int n_tiles = (int)c->h_tiles.size();
    hipStream_t st = c->stream;
    HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.ids, c->h_ids.data(), rows * 4, hipMemcpyHostToDevice, st), "upload ids");
    HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.rows, c->h_rows.data(), rows * sizeof(RowInfo), hipMemcpyHostToDevice, st), "upload rows");
    HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.tiles, c->h_tiles.data(), n_tiles * sizeof(int2), hipMemcpyHostToDevice, st), "upload tiles");
    HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.last_row, c->h_last.data(), B * 4, hipMemcpyHostToDevice, st), "upload last rows");
    HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.state, c->h_state.data(), B * sizeof(SeqState), hipMemcpyHostToDevice, st), "upload state");
    HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.btab, c->h_btab.data(), c->h_btab.size() * 4, hipMemcpyHostToDevice, st), "upload block table");
    HIPCHK(c, hipStreamSynchronize(st), "prefill upload sync");

    const int d = cf.d_model, dt = cf.dtype;
    EmbedArgs e{};
    e.dtype = dt; e.mode = 1; e.n_rows = rows; e.Q = 0; e.st = c->ws_ptr<SeqState>(c->ws.state);
    e.ids = c->ws_ptr<int32_t>(c->ws.ids); e.rows = c->ws_ptr<RowInfo>(c->ws.rows); e.tiles = c->ws_ptr<int2>(c->ws.tiles);
    e.emb_phone = c->wt(MTP_T_EMB_PHONE); e.emb_ac = c->wt(MTP_T_EMB_AC); e.pos = c->wt(MTP_T_POS);
    e.ln_g = (const float*)c->lt(0, MTP_T_LN1_G); e.ln_b = (const float*)c->lt(0, MTP_T_LN1_B);
    e.d = d; e.h = c->ws_ptr<float>(c->ws.h); e.u = c->WS() + c->ws.u;
    e.packed = dt == MTP_DTYPE_BF16 ? 1 : 0;
    HIPCHK(c, embed_ln(st, e), "prefill embed");
    for (int l = 0; l < cf.n_layers; ++l) {
        int rc = run_layer(c, l, rows, n_tiles, MTP_ATTN_QT, 1 << 30, 1, false);
        if (rc) return rc;
    }
    FinalArgs f{};
    f.dtype = dt; f.B = B; f.d = d; f.mode = 1; f.Q = 0; f.st = c->ws_ptr<SeqState>(c->ws.state);
    f.last_row = c->ws_ptr<int32_t>(c->ws.last_row); f.h = c->ws_ptr<float>(c->ws.h); f.hz = c->ws_ptr<float>(c->ws.hz);
    f.z = nullptr;
    HIPCHK(c, final_ln(st, f), "prefill last rows");

    int64_t max_ctx = 0;
    for (int b = 0; b < B; ++b) max_ctx = std::max<int64_t>(max_ctx, phon_len[b] + ac_len[b] + (int64_t)cf.max_new);
    c->plan_ctx = max_ctx;
    c->B = B;
    {
        const int rc = plan_splits(c, 0);
        if (rc) return rc;
    }
    c->q_pad = 0;
    c->prefilled = true;
    c->n_pre_rows = rows;
    c->n_pre_tiles = n_tiles;
    return MTP_OK;
}

int mtp_decode_step_async(mtp_ctx* c, int K, int top_k, int32_t* d_tokens, int32_t* d_count) {
    int rc = step_common(c, K, top_k);
    if (rc) return rc;
    if (d_tokens)
        HIPCHK(c, hipMemcpyAsync(d_tokens, c->WS() + c->ws.out_tok, (size_t)c->B * K * 4, hipMemcpyDeviceToDevice, c->stream), "copy tokens");
    if (d_count)
        HIPCHK(c, hipMemcpyAsync(d_count, c->WS() + c->ws.out_cnt, (size_t)c->B * 4, hipMemcpyDeviceToDevice, c->stream), "copy counts");
    return MTP_OK;
}

int mtp_decode_step(mtp_ctx* c, int K, int top_k, int32_t* out_tokens, int32_t* out_count) {
    if (!out_tokens || !out_count) { if (c) c->err = "NULL output"; return MTP_EINVAL; }
    int rc = step_common(c, K, top_k);
    if (rc) return rc;
    HIPCHK(c, hipMemcpyAsync(out_tokens, c->WS() + c->ws.out_tok, (size_t)c->B * K * 4, hipMemcpyDeviceToHost, c->stream), "tokens to host");
    HIPCHK(c, hipMemcpyAsync(out_count, c->WS() + c->ws.out_cnt, (size_t)c->B * 4, hipMemcpyDeviceToHost, c->stream), "counts to host");
    unsigned waits_out[2] = {0, 0};
    // (each word exists, zeroed, once its launch has been planned)
    unsigned* werr = c->xcd_deal == 1 ? c->ws_ptr<unsigned>(c->ws.fsync) + 3 * (3 * c->cfg.d_model / 16) : nullptr;
    unsigned* ferr = c->ffn_ready == 1
                         ? reinterpret_cast<unsigned*>(c->ws_ptr<bf16_t>(c->ws.ffs) + (size_t)3 * 16 * c->cfg.d_ff)
                         : nullptr;
    if (werr)
        HIPCHK(c, hipMemcpyAsync(&waits_out[0], werr, 4, hipMemcpyDeviceToHost, c->stream), "front wait count");
    if (ferr)
        HIPCHK(c, hipMemcpyAsync(&waits_out[1], ferr, 4, hipMemcpyDeviceToHost, c->stream), "ffn wait count");
    HIPCHK(c, hipStreamSynchronize(c->stream), "step sync");
    if (waits_out[0] || waits_out[1]) {
        // a one-launch front or FFN went on with data it could not see
        // complete: the tokens and the sequences' state are not those of
        // the model.  The context keeps separate launches from now on.
        if (waits_out[0]) {
            HIPCHK(c, hipMemsetAsync(werr, 0, 4, c->stream), "front wait count");
            c->xcd_deal = 0;
        }
        if (waits_out[1]) {
            HIPCHK(c, hipMemsetAsync(ferr, 0, 4, c->stream), "ffn wait count");
            c->ffn_ready = 0;
        }
        HIPCHK(c, hipStreamSynchronize(c->stream), "wait counts");
        c->prefilled = false;
        c->err = waits_out[0] ? "a decode front's hand-off wait ran out: this step's tokens and the sequence state "
                                "are invalid; prefill again"
                              : "a chained FFN's wait ran out: this step's tokens and the sequence state are "
                                "invalid; prefill again";
        return MTP_ETIMEOUT;
    }
    return MTP_OK;
}

int mtp_get_logits(mtp_ctx* c, float* logits) {
    if (!c) return MTP_EINVAL;
    if (!c->last_K) { c->err = "no decode step yet"; return MTP_ESTATE; }
    if (logits)
        HIPCHK(c, hipMemcpyAsync(logits, c->WS() + c->ws.logits, (size_t)c->B * c->last_K * c->cfg.vocab * 4, hipMemcpyDeviceToHost, c->stream), "logits to host");
    HIPCHK(c, hipStreamSynchronize(c->stream), "sync");
    return MTP_OK;
}

int mtp_get_lattice(mtp_ctx* c, int32_t* cand, float* ehat, float* delta, int32_t* psi, int32_t* slots) {
    if (!c) return MTP_EINVAL;
    if (!c->last_K) { c->err = "no decode step yet"; return MTP_ESTATE; }
    const size_t n = (size_t)c->B * c->last_K * c->last_topk * 4;
    hipStream_t st = c->stream;
    if (cand) HIPCHK(c, hipMemcpyAsync(cand, c->WS() + c->ws.cand, n, hipMemcpyDeviceToHost, st), "cand");
    if (ehat) HIPCHK(c, hipMemcpyAsync(ehat, c->WS() + c->ws.ehat, n, hipMemcpyDeviceToHost, st), "ehat");
    if (delta) HIPCHK(c, hipMemcpyAsync(delta, c->WS() + c->ws.delta, n, hipMemcpyDeviceToHost, st), "delta");
    if (psi) HIPCHK(c, hipMemcpyAsync(psi, c->WS() + c->ws.psi, n, hipMemcpyDeviceToHost, st), "psi");
    if (slots) HIPCHK(c, hipMemcpyAsync(slots, c->WS() + c->ws.slots, (size_t)c->B * c->last_K * 4, hipMemcpyDeviceToHost, st), "slots");
    HIPCHK(c, hipStreamSynchronize(st), "sync");
    return MTP_OK;
}

int mtp_force_tokens(mtp_ctx* c, const int32_t* tokens, const int32_t* count) {
    if (!c) return MTP_EINVAL;
    if (is_nar(c->cfg)) { c->err = "a NAR context has no decode steps"; return MTP_EINVAL; }
    if (!c->prefilled || !c->last_K) { c->err = "no decode step to force since the last prefill"; return MTP_ESTATE; }
    if (!tokens || !count) { c->err = "NULL token or count array"; return MTP_EINVAL; }
    const mtp_config& cf = c->cfg;
    const int B = c->B, K = c->last_K;
    hipStream_t st = c->stream;
    std::vector<SeqState> s(B);
    std::vector<int32_t> n_old(B);
    HIPCHK(c, hipMemcpyAsync(s.data(), c->WS() + c->ws.state, B * sizeof(SeqState), hipMemcpyDeviceToHost, st), "state to host");
    HIPCHK(c, hipMemcpyAsync(n_old.data(), c->WS() + c->ws.out_cnt, B * 4, hipMemcpyDeviceToHost, st), "counts to host");
    HIPCHK(c, hipStreamSynchronize(st), "sync");
    // validate everything before changing anything
    for (int b = 0; b < B; ++b) {
        const int n = count[b], g0 = s[b].gen - n_old[b];
        if (n_old[b] == 0) {
            if (n != 0) { c->err = "a sequence that had ended before the step takes count 0"; return MTP_EINVAL; }
            continue;
        }
        if (n < 1 || n > K || n > cf.max_new - g0) { c->err = "forced count out of range"; return MTP_EINVAL; }
        for (int i = 0; i < n; ++i) {
            const int32_t t = tokens[(size_t)b * K + i];
            if (t < 0 || t >= cf.vocab) { c->err = "forced token id out of range"; return MTP_EINVAL; }
            if (t == cf.eos_id && (i != n - 1 || g0 + i < cf.eos_min)) {
                c->err = "a forced EOS must be the last forced token and at a generated index >= eos_min";
                return MTP_EINVAL;
            }
        }
    }
    std::vector<int32_t> out_tok((size_t)B * K, -1), out_cnt(B);
    for (int b = 0; b < B; ++b) {
        const int n = count[b];
        out_cnt[b] = n;
        if (n_old[b] == 0) continue;
        const int g0 = s[b].gen - n_old[b];
        const int32_t* tb = tokens + (size_t)b * K;
        for (int i = 0; i < n; ++i) {
            out_tok[(size_t)b * K + i] = tb[i];
            s[b].pend_ids[i] = tb[i];
        }
        const bool done = tb[n - 1] == cf.eos_id || g0 + n >= cf.max_new;
        s[b].gen = g0 + n;
        s[b].done = done ? 1 : 0;
        s[b].pend_len = done ? 0 : n;
        s[b].last_tok = tb[n - 1];
        HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.hist + ((size_t)b * cf.max_new + g0) * 4, tb, (size_t)n * 4,
                                 hipMemcpyHostToDevice, st), "history");
    }
    HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.state, s.data(), B * sizeof(SeqState), hipMemcpyHostToDevice, st), "state");
    HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.out_tok, out_tok.data(), out_tok.size() * 4, hipMemcpyHostToDevice, st), "tokens");
    HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.out_cnt, out_cnt.data(), B * 4, hipMemcpyHostToDevice, st), "counts");
    HIPCHK(c, hipStreamSynchronize(st), "sync");
    return MTP_OK;
}

int mtp_set_selection(mtp_ctx* c, int lattice, int anchored) {
    if (!c) return MTP_EINVAL;
    if (lattice != MTP_LATTICE_OWN && lattice != MTP_LATTICE_UNION) { c->err = "unknown lattice"; return MTP_EINVAL; }
    if (anchored != 0 && anchored != 1) { c->err = "anchored must be 0 or 1"; return MTP_EINVAL; }
    c->lattice = lattice;
    c->anchored = anchored;
    return MTP_OK;
}

int mtp_get_union_lattice(mtp_ctx* c, int32_t* m, int32_t* states, float* ehat, float* delta, int32_t* psi,
                          int32_t* slots) {
    if (!c) return MTP_EINVAL;
    if (!c->last_K) { c->err = "no decode step yet"; return MTP_ESTATE; }
    if (c->last_lattice != MTP_LATTICE_UNION) { c->err = "the last step did not use the union lattice"; return MTP_ESTATE; }
    const size_t B = c->B, n = B * MTP_MAX_HEADS_K * 64 * 4;
    hipStream_t st = c->stream;
    if (m) HIPCHK(c, hipMemcpyAsync(m, c->WS() + c->ws.u_m, B * 4, hipMemcpyDeviceToHost, st), "m");
    if (states) HIPCHK(c, hipMemcpyAsync(states, c->WS() + c->ws.u_states, B * 64 * 4, hipMemcpyDeviceToHost, st), "states");
    if (ehat) HIPCHK(c, hipMemcpyAsync(ehat, c->WS() + c->ws.u_ehat, n, hipMemcpyDeviceToHost, st), "ehat");
    if (delta) HIPCHK(c, hipMemcpyAsync(delta, c->WS() + c->ws.u_delta, n, hipMemcpyDeviceToHost, st), "delta");
    if (psi) HIPCHK(c, hipMemcpyAsync(psi, c->WS() + c->ws.u_psi, n, hipMemcpyDeviceToHost, st), "psi");
    if (slots) HIPCHK(c, hipMemcpyAsync(slots, c->WS() + c->ws.slots, B * c->last_K * 4, hipMemcpyDeviceToHost, st), "slots");
    HIPCHK(c, hipStreamSynchronize(st), "sync");
    return MTP_OK;
}

int mtp_set_sampling(mtp_ctx* c, int mode, float temperature, uint64_t seed) {
    if (!c) return MTP_EINVAL;
    if (mode != MTP_SELECT_BEST && mode != MTP_SELECT_SAMPLE) { c->err = "unknown selection mode"; return MTP_EINVAL; }
    if (mode == MTP_SELECT_SAMPLE) {
        const float inv = 1.0f / temperature;
        if (!(temperature > 0.f) || !std::isfinite(temperature) || !std::isfinite(inv)) {
            c->err = "temperature must be finite and positive";
            return MTP_EINVAL;
        }
        c->h_smp.seed = seed;
        c->h_smp.inv_tau = inv;
        c->smp_dirty = true;
    }
    c->sample = mode == MTP_SELECT_SAMPLE ? 1 : 0;
    return MTP_OK;
}

int mtp_get_uniforms(mtp_ctx* c, float* u) {
    if (!c || !u) return MTP_EINVAL;
    if (!c->last_K) { c->err = "no decode step yet"; return MTP_ESTATE; }
    if (!c->last_sample) { c->err = "the last step did not sample"; return MTP_ESTATE; }
    HIPCHK(c, hipMemcpyAsync(u, c->WS() + c->ws.smp_u, (size_t)c->B * MTP_MAX_HEADS_K * 4, hipMemcpyDeviceToHost, c->stream),
           "uniforms");
    HIPCHK(c, hipStreamSynchronize(c->stream), "sync");
    return MTP_OK;
}

// ---------------------------------------------------------------- NAR module
int mtp_nar_prepare(mtp_ctx* c, int B, const int32_t* phon, const int32_t* phon_len, const int32_t* prompt,
                    const int32_t* prompt_len, const int32_t* a1, const int32_t* target_len) {
    if (!c) return MTP_EINVAL;
    const mtp_config& cf = c->cfg;
    if (!is_nar(cf)) { c->err = "not a NAR context"; return MTP_EINVAL; }
    if (B < 1 || B > cf.max_batch) { c->err = "batch out of range"; return MTP_EINVAL; }
    if (!phon_len || !prompt_len || !target_len) { c->err = "NULL length array"; return MTP_EINVAL; }
    const int nq = cf.k_heads + 1, cb = cf.vocab - 1;
    int64_t n_ph = 0, n_pr = 0, n_tg = 0;
    for (int b = 0; b < B; ++b) {
        const int64_t len = (int64_t)phon_len[b] + prompt_len[b] + target_len[b];
        if (phon_len[b] < 0 || prompt_len[b] < 0 || target_len[b] < 0 || len < 1 || len > cf.max_prompt) {
            c->err = "utterance length out of range";
            return MTP_EINVAL;
        }
        n_ph += phon_len[b];
        n_pr += prompt_len[b];
        n_tg += target_len[b];
    }
    if ((n_ph > 0 && !phon) || (n_pr > 0 && !prompt) || (n_tg > 0 && !a1)) { c->err = "NULL input array"; return MTP_EINVAL; }
    for (int64_t i = 0; i < n_ph; ++i)
        if (phon[i] < 0 || phon[i] >= cf.n_phone) { c->err = "phoneme id out of range"; return MTP_EINVAL; }
    for (int64_t i = 0; i < n_pr * nq; ++i)
        if (prompt[i] < 0 || prompt[i] >= cb) { c->err = "prompt code out of range"; return MTP_EINVAL; }
    for (int64_t i = 0; i < n_tg; ++i)
        if (a1[i] < 0 || a1[i] >= cb) { c->err = "target code out of range"; return MTP_EINVAL; }
    const int64_t maxp = c->ws.maxp;
    std::vector<int> need(B);
    int64_t total_pages = 0;
    for (int b = 0; b < B; ++b) {
        need[b] = (int)((phon_len[b] + prompt_len[b] + (int64_t)target_len[b] + cf.page_size - 1) / cf.page_size);
        total_pages += need[b];
    }
    if (total_pages > c->ws.num_pages) { c->err = "KV page pool exhausted"; return MTP_ENOMEM; }
    c->h_btab.assign((size_t)B * maxp, 0);
    int next = (int)c->ws.num_pages - 1;
    for (int p = 0; p < maxp; ++p)
        for (int b = 0; b < B; ++b)
            if (p < need[b]) c->h_btab[(size_t)b * maxp + p] = next--;
    c->h_rows.clear(); c->h_tiles.clear(); c->h_codes.clear(); c->h_tgt.clear();
    c->h_state.assign(B, SeqState{});
    c->h_tlen.assign(target_len, target_len + B);
    int64_t oph = 0, opr = 0, otg = 0;
    const int trows = (cf.dtype == MTP_DTYPE_BF16) ? MTP_PREFILL_ROWS : MTP_ATTN_QT;
    for (int b = 0; b < B; ++b) {
        const int lp = phon_len[b], lq = prompt_len[b], lt = target_len[b], len = lp + lq + lt;
        const int row0 = (int)c->h_rows.size();
        for (int i = 0; i < len; ++i) c->h_rows.push_back(RowInfo{b, i});
        for (int i = 0; i < lp; ++i) {
            int32_t cr[8] = {phon[oph + i], 0, 0, 0, 0, 0, 0, 0};
            c->h_codes.insert(c->h_codes.end(), cr, cr + 8);
        }
        for (int t = 0; t < lq; ++t) {
            int32_t cr[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            for (int q = 0; q < nq; ++q) cr[q] = prompt[opr * nq + (int64_t)q * lq + t];
            c->h_codes.insert(c->h_codes.end(), cr, cr + 8);
        }
        for (int t = 0; t < lt; ++t) {
            int32_t cr[8] = {a1[otg + t], 0, 0, 0, 0, 0, 0, 0};
            c->h_codes.insert(c->h_codes.end(), cr, cr + 8);
            c->h_tgt.push_back(row0 + lp + lq + t);
        }
        oph += lp;
        opr += lq;
        otg += lt;
        for (int i0 = 0; i0 < len; i0 += trows) c->h_tiles.push_back(make_int2(row0 + i0, std::min(trows, len - i0)));
        SeqState s{};
        s.ctx_len = len; s.phon_len = lp; s.prompt_len = lp + lq; s.last_tok = -1; s.done = 1;
        c->h_state[b] = s;
    }
    const int rows = (int)c->h_rows.size(), n_tiles = (int)c->h_tiles.size();
    hipStream_t st = c->stream;
    HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.rows, c->h_rows.data(), rows * sizeof(RowInfo), hipMemcpyHostToDevice, st), "upload rows");
    HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.tiles, c->h_tiles.data(), n_tiles * sizeof(int2), hipMemcpyHostToDevice, st), "upload tiles");
    HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.state, c->h_state.data(), B * sizeof(SeqState), hipMemcpyHostToDevice, st), "upload state");
    HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.btab, c->h_btab.data(), c->h_btab.size() * 4, hipMemcpyHostToDevice, st), "upload block table");
    HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.codes, c->h_codes.data(), c->h_codes.size() * 4, hipMemcpyHostToDevice, st), "upload codes");
    if (!c->h_tgt.empty())
        HIPCHK(c, hipMemcpyAsync(c->WS() + c->ws.tgt_rows, c->h_tgt.data(), c->h_tgt.size() * 4, hipMemcpyHostToDevice, st), "upload target rows");
    HIPCHK(c, hipStreamSynchronize(st), "nar upload sync");
    c->B = B;
    c->nar_rows = rows;
    c->nar_tiles = n_tiles;
    c->nar_ready = true;
    c->nar_ran = false;
    return MTP_OK;
}

int mtp_nar_run(mtp_ctx* c) {
    if (!c) return MTP_EINVAL;
    const mtp_config& cf = c->cfg;
    if (!is_nar(cf)) { c->err = "not a NAR context"; return MTP_EINVAL; }
    if (!c->nar_ready) { c->err = "NAR run before prepare"; return MTP_ESTATE; }
    const int d = cf.d_model, dt = cf.dtype, cb = cf.vocab - 1, rows = c->nar_rows;
    const size_t esz = dt == MTP_DTYPE_BF16 ? 2 : 4;
    hipStream_t st = c->stream;
    for (int s = 0; s < cf.k_heads; ++s) {
        NarEmbedArgs e{};
        e.dtype = dt; e.n_rows = rows; e.d = d; e.stage = s; e.n_q = cf.k_heads + 1; e.cb = cb;
        e.st = c->ws_ptr<SeqState>(c->ws.state); e.rows = c->ws_ptr<RowInfo>(c->ws.rows);
        e.codes = c->ws_ptr<int32_t>(c->ws.codes);
        e.emb_phone = c->wt(MTP_T_EMB_PHONE); e.emb_codes = c->wt(MTP_T_EMB_AC); e.pos = c->wt(MTP_T_POS);
        e.stage_vec = (const float*)c->wt(MTP_T_STAGE);
        e.ln_g = (const float*)c->lt(0, MTP_T_LN1_G); e.ln_b = (const float*)c->lt(0, MTP_T_LN1_B);
        e.h = c->ws_ptr<float>(c->ws.h); e.u = c->WS() + c->ws.u;
        e.packed = dt == MTP_DTYPE_BF16 ? 1 : 0;
        HIPCHK(c, nar_embed_ln(st, e), "nar embed");
        for (int l = 0; l < cf.n_layers; ++l) {
            const int rc = run_layer(c, l, rows, c->nar_tiles, MTP_ATTN_QT, 1 << 30, 1, false, true);
            if (rc) return rc;
        }
        RowsLnArgs r{};
        r.dtype = dt; r.n_rows = rows; r.d = d; r.h = c->ws_ptr<float>(c->ws.h);
        r.ln_g = (const float*)c->wt(MTP_T_LNF_G); r.ln_b = (const float*)c->wt(MTP_T_LNF_B); r.u = c->WS() + c->ws.u;
        r.packed = dt == MTP_DTYPE_BF16 ? 1 : 0;
        HIPCHK(c, rows_ln(st, r), "nar final ln");
        float* lg = c->ws_ptr<float>(c->ws.nar_logits) + (size_t)s * c->ws.m_pre * cb;
        GemmArgs g{};
        g.dtype = dt; g.epi = EPI_LOGITS; g.X = c->WS() + c->ws.u; g.ldx = d; g.M = rows; g.xpk = r.packed;
        g.W = (const char*)c->wt(MTP_T_W_HEADS) + (size_t)s * cb * d * esz; g.N = cb; g.K = d; g.splits = 1;
        g.bias = (const float*)c->wt(MTP_T_B_HEADS) + (size_t)s * cb; g.out = lg; g.ldo = cb;
        HIPCHK(c, gemm(st, g), "nar head gemm");
        ArgmaxArgs am{};
        am.n = (int)c->h_tgt.size(); am.tgt_rows = c->ws_ptr<int32_t>(c->ws.tgt_rows); am.logits = lg; am.ld = cb;
        am.cb = cb; am.codes = c->ws_ptr<int32_t>(c->ws.codes); am.slot = s + 1;
        HIPCHK(c, rows_argmax(st, am), "nar argmax");
    }
    c->nar_ran = true;
    return MTP_OK;
}

int mtp_nar_get_codes(mtp_ctx* c, int32_t* codes) {
    if (!c || !codes) return MTP_EINVAL;
    if (!is_nar(c->cfg)) { c->err = "not a NAR context"; return MTP_EINVAL; }
    if (!c->nar_ran) { c->err = "no NAR run yet"; return MTP_ESTATE; }
    std::vector<int32_t> all((size_t)c->nar_rows * 8);
    HIPCHK(c, hipMemcpyAsync(all.data(), c->WS() + c->ws.codes, all.size() * 4, hipMemcpyDeviceToHost, c->stream), "codes to host");
    HIPCHK(c, hipStreamSynchronize(c->stream), "sync");
    const int k = c->cfg.k_heads;
    size_t o = 0, ti = 0;
    for (int b = 0; b < c->B; ++b) {
        const int lt = c->h_tlen[b];
        for (int s = 0; s < k; ++s)
            for (int t = 0; t < lt; ++t) codes[o + (size_t)s * lt + t] = all[(size_t)c->h_tgt[ti + t] * 8 + s + 1];
        o += (size_t)k * lt;
        ti += lt;
    }
    return MTP_OK;
}

int mtp_nar_get_logits(mtp_ctx* c, int stage, float* logits) {
    if (!c || !logits) return MTP_EINVAL;
    if (!is_nar(c->cfg)) { c->err = "not a NAR context"; return MTP_EINVAL; }
    if (stage < 0 || stage >= c->cfg.k_heads) { c->err = "stage out of range"; return MTP_EINVAL; }
    if (!c->nar_ran) { c->err = "no NAR run yet"; return MTP_ESTATE; }
    const int cb = c->cfg.vocab - 1;
    std::vector<float> all((size_t)c->nar_rows * cb);
    const char* src = c->WS() + c->ws.nar_logits + (size_t)stage * c->ws.m_pre * cb * 4;
    HIPCHK(c, hipMemcpyAsync(all.data(), src, all.size() * 4, hipMemcpyDeviceToHost, c->stream), "logits to host");
    HIPCHK(c, hipStreamSynchronize(c->stream), "sync");
    for (size_t i = 0; i < c->h_tgt.size(); ++i)
        std::memcpy(logits + i * cb, all.data() + (size_t)c->h_tgt[i] * cb, (size_t)cb * 4);
    return MTP_OK;
}

int mtp_get_seq_state(mtp_ctx* c, int32_t* ctx_len, int32_t* pend_len, int32_t* gen, int32_t* done) {
    if (!c) return MTP_EINVAL;
    if (!c->prefilled) { c->err = "no prefill yet"; return MTP_ESTATE; }
    std::vector<SeqState> s(c->B);
    HIPCHK(c, hipMemcpyAsync(s.data(), c->WS() + c->ws.state, c->B * sizeof(SeqState), hipMemcpyDeviceToHost, c->stream), "state to host");
    HIPCHK(c, hipStreamSynchronize(c->stream), "sync");
    for (int b = 0; b < c->B; ++b) {
        if (ctx_len) ctx_len[b] = s[b].ctx_len;
        if (pend_len) pend_len[b] = s[b].pend_len;
        if (gen) gen[b] = s[b].gen;
        if (done) done[b] = s[b].done;
    }
    return MTP_OK;
}

int mtp_get_tokens(mtp_ctx* c, int32_t* tokens) {
    if (!c || !tokens) return MTP_EINVAL;
    if (!c->prefilled) { c->err = "no prefill yet"; return MTP_ESTATE; }
    HIPCHK(c, hipMemcpyAsync(tokens, c->WS() + c->ws.hist, (size_t)c->B * c->cfg.max_new * 4, hipMemcpyDeviceToHost, c->stream), "history to host");
    HIPCHK(c, hipStreamSynchronize(c->stream), "sync");
    return MTP_OK;
}

int mtp_profile_replay(mtp_ctx* c, int kclass, int iters, void* flush_buf, uint64_t flush_bytes, double* avg_us) {
    if (!c || !avg_us || iters < 1) return MTP_EINVAL;
    if ((flush_buf == nullptr) != (flush_bytes == 0)) { c->err = "eviction buffer and size must be given together"; return MTP_EINVAL; }
    if (flush_buf && (flush_bytes < 1024 || flush_bytes % 16 || ((uintptr_t)flush_buf & 15))) {
        c->err = "eviction buffer must be 16-byte aligned and a multiple of 16 bytes, at least 1 KiB";
        return MTP_EINVAL;
    }
    const bool cold = flush_buf != nullptr;
    if (kclass < MTP_KCLASS_GEMM_FFN1 || kclass > MTP_KCLASS_FFN_CHAIN) { c->err = "unknown kernel class"; return MTP_EINVAL; }
    auto it = c->has_last ? c->step_launches.find(c->last_key) : c->step_launches.end();
    if (it == c->step_launches.end() || it->second.cls[kclass].empty()) {
        c->err = "the last decode step launched nothing of this kernel class";
        return MTP_ESTATE;
    }
    const std::vector<mtp_ctx::Launch>& v = it->second.cls[kclass];
    // from here on the residual stream and the cache rows of the next
    // positions no longer hold what the next step expects
    c->prefilled = false;
    hipEvent_t e0, e1;
    HIPCHK(c, hipEventCreate(&e0), "event");
    hipError_t e = hipEventCreate(&e1);
    if (e != hipSuccess) { (void)hipEventDestroy(e0); return hip_fail(c, e, "event"); }
    // a pass holds at least 12 launches, so that its one launch latency is
    // spread as thinly for the heads (one launch per step) as for the layers
    const size_t reps = (12 + v.size() - 1) / v.size();
    double total_ms = 0.0;
    for (int i = 0; i < iters && e == hipSuccess; ++i) {
        if (cold) e = cache_flush(c->stream, flush_buf, (size_t)flush_bytes);
        if (e == hipSuccess) e = hipEventRecord(e0, c->stream);
        for (size_t j = 0; j < v.size() * reps && e == hipSuccess; ++j) e = v[j % v.size()](c->stream);
        if (e == hipSuccess) e = hipEventRecord(e1, c->stream);
        if (e == hipSuccess) e = hipEventSynchronize(e1);
        float ms = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
        total_ms += ms;
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    if (e != hipSuccess) return hip_fail(c, e, "replay");
    *avg_us = 1000.0 * total_ms / ((double)iters * (double)(v.size() * reps));
    return MTP_OK;
}

int mtp_reset(mtp_ctx* c) {
    if (!c) return MTP_EINVAL;
    c->prefilled = false;
    c->B = 0;
    c->q_pad = 0;
    c->last_K = 0;
    return MTP_OK;
}

void mtp_destroy(mtp_ctx* c) {
    if (!c) return;
    if (c->stream) (void)hipStreamSynchronize(c->stream);
    for (auto& kv : c->graphs) (void)hipGraphExecDestroy(kv.second);
    delete c;
}

const char* mtp_last_error(const mtp_ctx* c) { return c ? c->err.c_str() : "NULL context"; }

}  // extern "C"
