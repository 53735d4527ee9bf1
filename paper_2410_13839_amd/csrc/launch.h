// Host-side launchers of the decode kernels (internal to libmtp).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace mtp {

enum EpiKind { EPI_QKV = 0, EPI_GELU = 1, EPI_PARTIAL = 2, EPI_LOGITS = 3, EPI_RESID = 4 };

struct GemmArgs {
    int dtype;            // 0 fp32, 1 bf16 (both X and W)
    int epi;              // EpiKind
    const void* X; int ldx; int M;
    const void* W; int N; int K;
    int splits;           // split-K factor (EPI_PARTIAL only)
    int xpk;              // bf16 X in MFMA fragment order (frag_off), M <= 256 only
    int opk;              // EPI_GELU: bf16 output in fragment order
    // epilogue operands
    const float* bias;
    void* out; int ldo; size_t split_stride;   // EPI_RESID: out = the fp32 residual stream
    float* q; const RowInfo* rows; KVView kv; int d;
};

hipError_t gemm(hipStream_t st, const GemmArgs& a);
int gemm_split_granule(int dtype, int M);
int gemm_tiles(int M, int N);
int gemm_resid_in_place(int M, int N);

struct AttnArgs {
    int dtype;                 // KV / output element type: 0 fp32, 1 bf16
    const float* q; int ldq;   // [rows][d]
    const RowInfo* rows;
    const int2* tiles;         // (row0, nrows) per tile
    int n_tiles;
    int qt;                    // rows per tile (1, 2, 4 or 8)
    KVView kv;
    int split_len;             // keys per split (multiple of 32)
    int n_splits;
    void* out; int ldo;        // [rows][d] attention output (act type)
    float* part;               // split partials when n_splits > 1
    int bidir;                 // 1: every row sees its sequence's ctx_len keys (no causal mask)
    const SeqState* st;        // sequence lengths when bidir
};
hipError_t attention(hipStream_t st, const AttnArgs& a);

// Decode attention: the pending chunk of each sequence (rows b*Q .. b*Q +
// pend_len - 1) over its cache in splits of split_len keys.  With several
// splits the partials are merged by attn_decode_merge when `merge` is set,
// otherwise by the consumer (out-projection prologue, GemvArgs xmode 4).
struct AttnDecArgs {
    int dtype;
    int B; int Q; int qt;
    const SeqState* st;
    const float* q; int ldq;
    KVView kv;
    int split_len; int n_splits;
    void* out; int ldo;
    float* part;               // [B][H][n_splits][qt][66]
    int merge;                 // 1: launch the merge kernel after the splits
    int packed;                // bf16 out in fragment order (frag_off, K = ldo)
};
hipError_t attention_decode(hipStream_t st, const AttnDecArgs& a);
// Only the merge of decode split partials (after attention_mfma).
hipError_t attention_decode_merge(hipStream_t st, const AttnDecArgs& a);

// MFMA attention for bf16 caches: mode 0 = decode (one tile per sequence, rows
// from the sequence state), mode 1 = prefill (tiles of up to 16 rows).
// Hand-off state of the fused decode front (qkv_front): one flag per QKV
// column tile, set by the tile once its columns are stored.  Consecutive
// launches use different flag sets: a launch clears the set of the next one
// (next_flags), whose last user has finished.  Zero before the first launch.
struct FrontSync {
    unsigned* flags;      // [3 * tiles_per_mat]: this launch's set
    unsigned* next_flags; // [3 * tiles_per_mat]: the next launch's set (cleared here)
    unsigned* err;        // hand-off waits that ran out (a bounded wait; none expected)
    int tiles_per_mat;    // d / 16
    int per_head;         // attention workgroups per head (batch x key splits)
    int spin;             // polls before a hand-off wait gives up (0: at once)
};

// Hand-off state of the chained FFN (ffn_chain): the FFN1 workgroups store
// the hidden rows of this launch's set (GemvArgs::out of FFN1, ::x of FFN2:
// [16][d_ff] bf16, which held the sentinel 0xFFFF everywhere when the launch
// began) and refill the next launch's set with the sentinel; the FFN2
// workgroups poll their K range of the rows until no sentinel is left.
struct FfnSync {
    bf16_t* next;         // [16][d_ff]: the next launch's set
    unsigned* err;        // polls that ran out (a bounded wait; none expected)
    int spin;             // polls before a wait gives up (0: at once)
};

struct AttnMfmaArgs {
    int mode;
    int n_tiles;
    int Q; int qt;
    const SeqState* st;
    const int2* tiles; const RowInfo* rows;
    const float* q; int ldq;
    const bf16_t* qh;          // decode inside the fused front: the queries as bf16 q / 8 ([rows][ldq])
    KVView kv;
    int split_len; int n_splits;
    bf16_t* out; int ldo;
    float* part;
    int bidir;                 // prefill mode: 1 = every row sees its sequence's ctx_len keys
    int packed;                // decode mode: out in fragment order (frag_off, K = ldo)
};
hipError_t attention_mfma(hipStream_t st, const AttnMfmaArgs& a);

// Small-M (<= 16 rows) bf16 projection with fused row work; see gemv.hip.
struct GemvArgs {
    int epi;                   // EPI_QKV, EPI_GELU, EPI_LOGITS (LayerNorm modes), EPI_PARTIAL (split-K x4)
    int xmode;                 // 0 bf16 rows, 1 LN(h + partials + bias), 2 embed + LN, 3 final LN (heads),
                               // 4 merged attention partials, 5 merged attention partials plus the
                               // pending chunk's own keys (EPI_PARTIAL only)
    int M, N, K;
    const bf16_t* W;
    const bf16_t* x; int ldx;                       // xmode 0
    const float* h; int ldh;                        // residual rows, row stride = d: the LayerNorm input of
                                                    // xmode 1, 3 when part_on is 0; EPI_PARTIAL: the residual
                                                    // input its first K range adds (with `bias`)
    const float* part; int part_rows;               // [4][part_rows][d] split-K partials whose sum is the
                                                    // LayerNorm input (xmode 1, 3 with part_on)
    int part_on;
    const float* g; const float* beta;              // LN gain / shift
    const SeqState* st; int Q;                      // xmode 2, 3, 4 and EPI_QKV
    const bf16_t* emb; const bf16_t* pos;           // xmode 2
    float* h_out;                                   // completed residual rows, written by workgroup 0 (may be NULL;
                                                    // must not alias h)
    const float* hz;                                // xmode 3: last prefill hidden state
    float* apart; int qt, split_len, n_splits;         // xmode 4, 5: attention split partials (written by qkv_attn)
    const float* bias;
    void* out; int ldo;                             // EPI_GELU / EPI_LOGITS output
    float* part_out;                                // EPI_PARTIAL output [4][M][N]
    float* q; KVView kv; int d;                     // EPI_QKV; xmode 5 reads q ([M][d] fp32)
    bf16_t* qh;                                     // EPI_QKV in qkv_front: queries stored here as bf16 q / 8
                                                    // instead of to q
    bf16_t* kvnew;                                  // [2][M][d]: the pending rows' keys, then values (bf16),
                                                    // written by qkv_attn, read by xmode 5
};
int gemv_merge_max_splits(int M, int d);

// LN1 + QKV projection + attention of the pending chunk over the cached keys
// in one launch (B * Q <= 8 rows, bf16, d <= 1024; see qkv_attn.hip).  Reads
// the GemvArgs of an EPI_QKV launch (xmode 1 or 2) plus apart / qt /
// split_len / n_splits (workgroups per head) and kvnew.
hipError_t qkv_attn(hipStream_t st, const GemvArgs& a);
// Whether qkv_attn serves `rows` decode rows of model width d, cached
// contexts of at most max_ctx keys, with n_splits workgroups per head.
bool qkv_attn_ok(int rows, int d, int n_heads, int64_t max_ctx, int n_splits);
// Keys per split (a multiple of 16) of qkv_attn for contexts of at most
// max_ctx keys over n_splits workgroups per head.
int qkv_attn_split_len(int64_t max_ctx, int n_splits);

// LN1 + QKV projection + decode attention in one launch (gemv.hip): the
// GemvArgs of an EPI_QKV launch (xmode 1 or 2, rows = batch x Q <= 16) and
// the AttnMfmaArgs of the decode attention over its q and cache (split_len
// 256 or 512, whose partials the out-projection merges when n_splits > 1),
// with the hand-off state fs (zero before the first launch; every launch
// leaves it zero).  Needs n_heads a multiple of 8, head dim 64, d <= 1024,
// and the dispatcher dealing workgroups j and j + 8 of a launch to one XCD
// (xcd_deal_check).
hipError_t qkv_front(hipStream_t st, const GemvArgs& a, const AttnMfmaArgs& p, const FrontSync& fs);
bool qkv_front_ok(int rows, int d, int n_heads, int batch, int split_len, int n_splits);
// LN2 + FFN1 + GELU, then FFN2 into four split-K partials, in one launch
// (gemv.hip): a1 the GemvArgs of the EPI_GELU launch (xmode 1, rows <= 16,
// d <= 1024) with a1.out the rows of this launch's set, a2 those of the
// EPI_PARTIAL launch (xmode 0, x = a1.out, ldx = d_ff) whose split-K
// partials go to a2.part_out, and whose first K range adds the bias and the
// residual input, the sum of the four partials of a2.part (a2.part_rows
// rows per split) that FFN1's LayerNorm also reads; a2.part_out must not be
// a2.part.  Every set starts filled with the sentinel (see FfnSync).
hipError_t ffn_chain(hipStream_t st, const GemvArgs& a1, const GemvArgs& a2, const FfnSync& fs);
bool ffn_chain_ok(int rows, int d, int d_ff);
// ORs into masks[r] (8 words) a bit per XCD that a workgroup j of a
// `grid`-workgroup launch with j % 8 == r ran on.
hipError_t xcd_deal_check(hipStream_t st, unsigned* masks, int grid);

// Reads `bytes` (a multiple of 16) of `buf` so that earlier data leaves the
// L2 and last-level caches (measurement only); writes a few words of `buf`.
hipError_t cache_flush(hipStream_t st, void* buf, size_t bytes);
hipError_t gemv(hipStream_t st, const GemvArgs& a);

// Row embedding (+ first LayerNorm).  mode 0: decode rows derived from the
// sequence state (Q rows per sequence); mode 1: prefill rows given by
// ids/rows.
struct EmbedArgs {
    int dtype;
    int mode;
    int n_rows;
    int Q;
    const SeqState* st;
    const int32_t* ids;
    RowInfo* rows;
    int2* tiles;
    const void* emb_phone; const void* emb_ac; const void* pos;
    const float* ln_g; const float* ln_b;
    int d;
    float* h;
    void* u;
    int packed;                // bf16 u in fragment order (frag_off, K = d)
};
hipError_t embed_ln(hipStream_t st, const EmbedArgs& a);

// h[r] += sum_s part[s][r] + bias; optionally u[r] = LN(h[r]).
struct ResidArgs {
    int dtype;
    int n_rows; int d;
    float* h;
    const float* part; int n_split; size_t split_stride;
    const float* bias;
    const float* ln_g; const float* ln_b;   // NULL: no LayerNorm
    void* u;
    int packed;                // bf16 u in fragment order (frag_off, K = d)
};
hipError_t resid_ln(hipStream_t st, const ResidArgs& a);

// hz[b] = h[src row of b]; z[b] = LN_f(hz[b]).
struct FinalArgs {
    int dtype;
    int B; int d;
    int mode;                  // 0 decode (Q rows per seq, last pending row), 1 prefill (last_row[])
    int Q;
    const SeqState* st;
    const int32_t* last_row;
    const float* h;
    float* hz;
    const float* ln_g; const float* ln_b;
    void* z;                   // NULL: copy only
    int packed;                // bf16 z in fragment order (frag_off, K = d)
};
hipError_t final_ln(hipStream_t st, const FinalArgs& a);

// NAR module input of one stage: row r (sequence ri.seq, position ri.pos) is
// the phoneme table at codes[r][0] (pos < phon_len), the sum of the n_q
// codebook tables at codes[r][0..n_q) (pos < prompt_len), or the sum of the
// tables 0..stage at codes[r][0..stage] (target); plus position and stage
// vectors; h = that row, u = LN1 of layer 0.
struct NarEmbedArgs {
    int dtype;
    int n_rows; int d;
    int stage; int n_q; int cb;        // predicted layer = stage + 2; codebook size
    const SeqState* st; const RowInfo* rows;
    const int32_t* codes;              // [rows][8]
    const void* emb_phone; const void* emb_codes; const void* pos;
    const float* stage_vec;            // [k_heads][d]
    const float* ln_g; const float* ln_b;
    float* h; void* u;
    int packed;                        // bf16 u in fragment order (frag_off, K = d)
};
hipError_t nar_embed_ln(hipStream_t st, const NarEmbedArgs& a);

// u[r] = LN(h[r]) for every row.
struct RowsLnArgs {
    int dtype; int n_rows; int d;
    const float* h; const float* ln_g; const float* ln_b;
    void* u;
    int packed;                        // bf16 u in fragment order (frag_off, K = d)
};
hipError_t rows_ln(hipStream_t st, const RowsLnArgs& a);

// codes[row][slot] = argmax (lowest index on ties) of logits[row][0..cb) for
// the rows listed in tgt_rows.
struct ArgmaxArgs {
    int n; const int32_t* tgt_rows;
    const float* logits; int ld; int cb;
    int32_t* codes; int slot;
};
hipError_t rows_argmax(hipStream_t st, const ArgmaxArgs& a);

// Sampling configuration, read by the selection kernel from device memory so
// that a captured step serves every seed and temperature.
struct SampleCfg {
    uint64_t seed;             // Philox key word 0
    float inv_tau;             // float32(1 / temperature)
    int32_t pad;
};

struct SelectArgs {
    int B; int K; int top_k; int V; int eos_id; int eos_min; int max_new;
    int Q;                     // pending rows per sequence this step (0 right after prefill)
    const float* logits;       // [B][ld_logits], head t at t*V
    int ld_logits;
    const float* logq;         // [V][V]
    SeqState* st;
    int32_t* cand; float* ehat; float* delta; int32_t* psi; int32_t* slots;  // [B][K][top_k] / [B][K]
    int32_t* out_tokens;       // [B][K]
    int32_t* out_count;        // [B]
    int32_t* hist; int hist_ld;  // [B][max_new]
    int lattice;               // 0 own top_k per position, 1 union of all heads' top_k
    int anchored;              // 1: delta_0 carries logQ[last emitted token][c]
    int32_t* u_states; int32_t* u_m;        // union lattice: [B][64] states, [B] count
    float* u_ehat; float* u_delta; int32_t* u_psi;   // [B][8][64]
    int sample;                // 0 best path (Viterbi), 1 path drawn from the lattice distribution
    const SampleCfg* smp;      // sampling seed and inverse temperature (device)
    float* smp_u;              // [B][8] the uniforms of the step, in draw order
};
// top_k of all K heads, Viterbi (or the sampled path) and accept in one
// launch (one workgroup per sequence).
hipError_t select_fused(hipStream_t st, const SelectArgs& a);

}  // namespace mtp
