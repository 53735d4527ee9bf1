/*
 * mtp.h -- C ABI of the MI355X (gfx950) decode path for multi-token
 * prediction with Viterbi-based speculative decoding.
 *
 * Paper: "Accelerating Codec-based Speech Synthesis with Multi-Token
 * Prediction and Speculative Decoding" (arXiv 2410.13839).
 *
 * The problem (Sec. 3.1, Eq. 1): given a phoneme prompt p and an acoustic
 * prompt (first-quantizer codec tokens), an autoregressive decoder-only
 * Transformer generates the first-quantizer token sequence.  Sec. 3.2: n
 * heads on the last hidden state predict the next n tokens in one step, and
 * the number of heads used can be chosen per call without retraining
 * (Fig. 1 caption).  Sec. 3.3 / Fig. 2: the n emitted tokens are the
 * best-scoring path, under a token-transition table Q and each head's
 * probabilities S_t, through each head's top_k candidates.
 *
 * One decode step = trunk forward of the pending tokens over the paged KV
 * cache -> final LayerNorm -> K head projections -> EOS mask + per-head
 * top_k -> Viterbi lattice -> accept.  All of it runs in HIP kernels on the
 * caller's stream.
 *
 * Conventions
 *  - Every call returns 0 on success or a negative MTP_E* code; no C++
 *    exception crosses this boundary.  mtp_last_error() gives the text of
 *    the last failure on a context.
 *  - The library allocates NO device memory at run time.  The caller
 *    allocates the four device buffers (sizes from mtp_query_sizes) and owns
 *    them; they must outlive the context.  The context owns only host
 *    bookkeeping.  The one fixed device array, the scratch of
 *    mtp_q_count_noalloc, is part of the library's code object.
 *  - All work is ordered on the one HIP stream given to mtp_create.  A
 *    context is not thread-safe.
 *  - Pointers documented "host" are plain host memory; "device" pointers
 *    are device memory on the current HIP device.
 */
#ifndef MTP_H
#define MTP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- error codes -------------------------------------------------------- */
#define MTP_OK       0
#define MTP_EINVAL  -1   /* bad argument, shape or limit                        */
#define MTP_ENOMEM  -2   /* KV page pool or workspace too small for the request */
#define MTP_ESTATE  -3   /* call out of order (e.g. decode before prefill)      */
#define MTP_EHIP    -4   /* a HIP runtime error; text in mtp_last_error         */
#define MTP_ETIMEOUT -5  /* a bounded device-side wait ran out (decode front);
                            the step's outputs and the sequence state are
                            invalid: prefill again                            */

/* ---- element types ------------------------------------------------------ */
#define MTP_DTYPE_F32   0   /* fp32 weights, activations and KV cache          */
#define MTP_DTYPE_BF16  1   /* bf16 weights / GEMM inputs / KV, fp32 accumulate */

/* ---- flags -------------------------------------------------------------- */
#define MTP_FLAG_NO_GRAPH  1   /* launch the decode step eagerly (no hipGraph replay) */
#define MTP_FLAG_NAR       2   /* the context holds the NAR module (mtp_nar_*), not the AR decoder */

/* Model and capacity description.  Head dimension is fixed at 64
 * (d_model / n_heads == 64). */
typedef struct mtp_config {
    int32_t n_layers;     /* Transformer blocks                                  */
    int32_t d_model;      /* hidden size, multiple of 64                          */
    int32_t n_heads;      /* attention heads, d_model / 64                        */
    int32_t d_ff;         /* FFN hidden size, multiple of 64                      */
    int32_t vocab;        /* codec vocabulary incl. EOS (1025)                    */
    int32_t eos_id;       /* EOS token id (1024)                                  */
    int32_t n_phone;      /* phoneme inventory size (512)                         */
    int32_t max_pos;      /* rows of the learned position table                   */
    int32_t k_heads;      /* prediction heads loaded, 1..8                        */
    int32_t topk_max;     /* largest top_k a decode step may ask for, 1..32       */
    int32_t max_batch;    /* sequences per prefill                                */
    int32_t max_prompt;   /* phonemes + acoustic tokens per sequence              */
    int32_t max_new;      /* generation budget per sequence (tokens)              */
    int32_t eos_min;      /* EOS masked while the generated index is < eos_min    */
    int32_t page_size;    /* tokens per KV page: 16 (MTP_EINVAL otherwise)        */
    int32_t num_pages;    /* pages in the pool; 0 = max_batch full sequences      */
    int32_t dtype;        /* MTP_DTYPE_*                                          */
    int32_t flags;        /* MTP_FLAG_*                                           */
} mtp_config;

/* Byte sizes of the caller-allocated device buffers. */
typedef struct mtp_sizes {
    uint64_t weights_bytes;    /* packed weights, layout from mtp_weight_offset  */
    uint64_t logq_bytes;       /* log Q, float32 [vocab][vocab]                  */
    uint64_t kv_bytes;         /* paged KV pool                                  */
    uint64_t workspace_bytes;  /* activations, lattice, per-sequence state       */
} mtp_sizes;

/* Device buffers (all device pointers, 256-byte aligned, caller-owned). */
typedef struct mtp_buffers {
    void*        weights;      /* packed weights                                  */
    const float* logq;         /* log Q: row = previous token, column = next token */
    void*        kv_pool;      /* KV pages; contents need no initialisation       */
    void*        workspace;    /* scratch + state; needs no initialisation        */
} mtp_buffers;

/* Weight tensors in packing order.  Matrices (_W_, tables) are stored in the
 * model dtype; vectors (biases, LayerNorm gain/shift) are always float32.
 * Per-layer tensors repeat for layer = 0 .. n_layers-1 in the order
 * MTP_T_LN1_G .. MTP_T_B_2.
 *
 * The tables (EMB_PHONE, EMB_AC, POS) and the fp32 model's Linear weights are
 * row-major [rows][d] / [out][in].  The bf16 model's Linear weights (W_QKV,
 * W_O, W_1, W_2, and W_HEADS read as one [k_heads * vocab][d] matrix) are
 * stored in MFMA fragment order so that every 16-row x 32-column fragment is
 * one contiguous 1 KB: with N rows (out) and K columns (in, a multiple of 32),
 * the rows are padded with zeros to a multiple of 16 and element (n, k) sits
 * at index
 *     ((n / 16) * (K / 32) + k / 32) * 512 + ((k % 32) / 8) * 128 + (n % 16) * 8 + k % 8,
 * so a tensor occupies ceil(N / 16) * 16 * K elements (mtp_weight_offset
 * still reports N * K). */
enum mtp_tensor {
    MTP_T_EMB_PHONE = 0,  /* [n_phone][d]                  */
    MTP_T_EMB_AC,         /* [vocab][d]                    */
    MTP_T_POS,            /* [max_pos][d]                  */
    MTP_T_LN1_G,          /* [d]   (per layer)             */
    MTP_T_LN1_B,          /* [d]                           */
    MTP_T_W_QKV,          /* [3d][d], rows q | k | v       */
    MTP_T_B_QKV,          /* [3d]                          */
    MTP_T_W_O,            /* [d][d]                        */
    MTP_T_B_O,            /* [d]                           */
    MTP_T_LN2_G,          /* [d]                           */
    MTP_T_LN2_B,          /* [d]                           */
    MTP_T_W_1,            /* [d_ff][d]                     */
    MTP_T_B_1,            /* [d_ff]                        */
    MTP_T_W_2,            /* [d][d_ff]                     */
    MTP_T_B_2,            /* [d]   (last per-layer tensor) */
    MTP_T_LNF_G,          /* [d]                           */
    MTP_T_LNF_B,          /* [d]                           */
    MTP_T_W_HEADS,        /* [k_heads][vocab][d]           */
    MTP_T_B_HEADS,        /* [k_heads][vocab]              */
    MTP_T_STAGE,          /* [k_heads][d] float32, NAR only (0 elements otherwise) */
    MTP_T_COUNT
};

/* NAR module (MTP_FLAG_NAR; Sec. 3.1, Eq. 2): the same config fields with
 * these meanings.  n_q = k_heads + 1 codec layers (k_heads <= 7), vocab - 1
 * codes per layer (vocab counts one extra entry, as for the AR's EOS; it is
 * not used).  EMB_AC holds the n_q codebook tables, [n_q][vocab - 1][d];
 * W_HEADS [k_heads][vocab - 1][d] and B_HEADS [k_heads][vocab - 1] are the
 * heads of layers 2..n_q; STAGE [k_heads][d] their stage vectors.
 * max_prompt bounds phonemes + prompt + target per utterance; max_new,
 * eos_min and topk_max are unused (they must still be valid); log Q is not
 * used (logq_bytes is 0 and buffers.logq may be NULL). */

typedef struct mtp_ctx mtp_ctx;

/* Fills *out with the buffer sizes a config needs.  Returns MTP_EINVAL for an
 * unsupported config (text via mtp_strerror only; there is no context). */
int mtp_query_sizes(const mtp_config* cfg, mtp_sizes* out);

/* Byte offset (from the start of the weights buffer) and element count of
 * one tensor; `layer` is ignored for non-layer tensors.  Every tensor starts
 * on a 256-byte boundary. */
int mtp_weight_offset(const mtp_config* cfg, int tensor, int layer,
                      uint64_t* offset_bytes, uint64_t* numel);

/* Creates a context over caller-owned device buffers.  `hip_stream` is a
 * hipStream_t (NULL = the null stream).  No device memory is allocated;
 * the KV pool and workspace are not read before prefill writes them. */
int mtp_create(const mtp_config* cfg, const mtp_buffers* bufs, void* hip_stream,
               mtp_ctx** out);

/* Prefill (Sec. 3.1: the AR module reads [phonemes; acoustic prompt] as one
 * sequence).  Host arrays: phon / ac are the B sequences' ids concatenated
 * (phon ids < n_phone, ac ids < vocab - 1), with per-sequence lengths
 * phon_len[B] and ac_len[B]; phon_len + ac_len must be in 1..max_prompt.
 * Resets all sequence state, reserves each sequence's KV pages for
 * prompt + max_new tokens (MTP_ENOMEM if the pool is too small), runs the
 * trunk over the prompts and keeps each last hidden state as the source of
 * the first decode step.  Returns after the work is enqueued and the host
 * inputs have been consumed. */
int mtp_prefill(mtp_ctx* ctx, int B, const int32_t* phon, const int32_t* phon_len,
                const int32_t* ac, const int32_t* ac_len);

/* One decode step with heads 1..K (1 <= K <= k_heads) and top_k candidates
 * per head (1 <= top_k <= topk_max).  Host outputs: out_tokens[B*K] gets
 * each sequence's emitted tokens (entries past its count are -1) and
 * out_count[B] the number emitted: K, fewer at the budget, up to and
 * including the first EOS (which ends the sequence), 0 once a sequence has
 * ended.  Blocks until the outputs are on the host.
 * Tuning override: the environment variable MTP_SPLIT_LEN, a multiple of
 * 32 from 32 up, sets the keys per decode-attention split of the steps
 * planned after it is set (raised where needed to keep at most 64 splits;
 * the library otherwise chooses it from the batch and the longest
 * context).  Results are the same up to floating-point rounding.
 * Default decode front for B * K <= 16 rows of a bf16 model with at least
 * two layers: LayerNorm, the QKV projection and the decode attention in one
 * launch, whose attention workgroups wait (bounded) for their own head's
 * QKV columns, stored by workgroups of the same launch on the same XCD; it
 * runs only if a check at the first such step finds that workgroups j and
 * j + 8 of a launch share an XCD, with 256 or 512 keys per split (the first
 * whose split count the out-projection can merge).  MTP_FRONT = 0 selects
 * separate QKV and attention launches, 256 or 512 forces that split length
 * (separate launches if it does not fit).  MTP_QKV_ATTN = 8 or 16 instead
 * runs, for B * K <= 8 rows, d_model <= 1024 and contexts of at most 256 *
 * that many keys, a front in which each of that many workgroups (key
 * splits) per head computes its own head's queries, the pending chunk's
 * attention to its own keys merged by the out-projection (slower on
 * MI355X).  Every front gives the same results up to rounding; the
 * variables are read when a step is planned.
 * Likewise, for B * K <= 16 rows of a bf16 model with at least two layers,
 * d_model <= 1024 and d_ff <= 4096 (multiples of 256 and 512), FFN1 and
 * FFN2 run as one launch whose FFN2 workgroups wait (bounded) for their K
 * range of the GELU rows; MTP_FFN_CHAIN = 0 selects two launches.
 * The waits of both one-launch kinds are bounded (MTP_FRONT_SPIN polls,
 * read by mtp_create; default 100000, tens of ms; 0 makes every wait give
 * up at once, which the tests use to reach this error path).  A wait that
 * ran out makes this call return MTP_ETIMEOUT: the tokens and the
 * sequence state of the step are invalid, the context needs mtp_prefill
 * again and uses separate launches for that kind from then on.  The counts
 * are read only here: mtp_decode_step_async does not report them, the
 * next mtp_decode_step does. */
int mtp_decode_step(mtp_ctx* ctx, int K, int top_k, int32_t* out_tokens, int32_t* out_count);

/* Same step, outputs written to DEVICE buffers d_tokens[B*K] and d_count[B]
 * on the context's stream, with no host synchronisation. */
int mtp_decode_step_async(mtp_ctx* ctx, int K, int top_k, int32_t* d_tokens, int32_t* d_count);

/* Parity hooks: copy the last decode step's intermediates to host memory
 * (synchronises the stream).  logits: float32 [B][K][vocab] before the EOS
 * mask.  cand: int32 [B][K][top_k] candidate ids (logit desc, id asc);
 * ehat: float32 emission scores l[c] - max l; delta: float32 Viterbi
 * scores; psi: int32 back-pointers (psi[.][0][.] = 0); slots: int32 [B][K]
 * chosen slot per position.  Any pointer may be NULL. */
int mtp_get_logits(mtp_ctx* ctx, float* logits);
int mtp_get_lattice(mtp_ctx* ctx, int32_t* cand, float* ehat, float* delta,
                    int32_t* psi, int32_t* slots);

/* Teacher forcing (Sec. 3.1, Eq. 1: each token is generated conditioned on
 * the given history).  Replaces the tokens the last decode step emitted with
 * the caller's, as if the step had selected them: host arrays tokens[B*K]
 * (K of that step; row b's first count[b] entries are used) and count[B].
 * A sequence the step ran (it emitted at least one token) takes 1 <= count[b]
 * <= min(K, max_new - generated count before the step); a sequence that had
 * ended before the step takes count[b] = 0.  Ids must be in [0, vocab); EOS
 * (eos_id) only as a sequence's last forced token and at a generated index
 * >= eos_min.  The forced tokens replace the step's outputs (the values
 * mtp_decode_step returned, the emitted history, the generated count, the
 * anchor token) and become the pending chunk of the next step; EOS or the
 * budget ends the sequence.  The step's logits and lattice are kept.  May be
 * called again for the same step.  Synchronises.  MTP_ESTATE unless a decode
 * step ran since the last prefill (and no profile replay since); MTP_EINVAL
 * for bad arguments, with nothing changed. */
int mtp_force_tokens(mtp_ctx* ctx, const int32_t* tokens, const int32_t* count);

/* Selection options for the following decode steps (paper Sec. 3.3, Fig. 2).
 * lattice MTP_LATTICE_OWN (default): position t's states are head t's own
 * top_k.  MTP_LATTICE_UNION: every position's states are the m <= K*top_k
 * distinct tokens of all heads' top_k in ascending id, scored at position t
 * by head t (e_t(c) = l_t[c] - max l_t, -inf for a masked EOS), with the
 * m x m sub-table of log Q (the paper's reduced transition matrix); steps
 * then need K * top_k <= 64 (MTP_EINVAL otherwise).  anchored = 1 adds
 * logQ[last emitted token][c] to the first position's scores (the acoustic
 * prompt's last token before any token was emitted; no term when there is
 * none).  Ties keep the lowest state index in both lattices.  MTP_EINVAL for
 * other values. */
#define MTP_LATTICE_OWN    0
#define MTP_LATTICE_UNION  1
int mtp_set_selection(mtp_ctx* ctx, int lattice, int anchored);

/* Path choice for the following decode steps.  MTP_SELECT_BEST (default):
 * the highest-scoring path (Viterbi, Sec. 3.3).  MTP_SELECT_SAMPLE: top_k
 * sampling inside the lattice (Fig. 2 caption) -- the path is drawn from the
 * distribution over the lattice's paths (either lattice, anchored or not)
 * proportional to prod_t exp(e_t(a_t) / temperature) * prod_{t>=1}
 * Q(a_{t-1}, a_t), by forward filtering, backward sampling: forward weights
 * alpha_t(j) = exp(e_t(j)/temperature) * sum_i alpha_{t-1}(i) Q(i, j), each
 * position rescaled by a power of two, then position K-1 drawn from
 * alpha_{K-1} and position t from alpha_t(i) Q(i, a_{t+1}).  One head gives
 * ordinary top_k sampling at that temperature.  Draw r of a step (r = K-1-t
 * for position t) of sequence b with generated count g uses word r % 4 of
 * the Philox4x64-10 block (Salmon et al., SC 2011) at counter (g, b, r / 4, 0)
 * with key (seed, 0), as u = (word >> 40) * 2^-24; the draw takes the first
 * state whose running weight sum exceeds u times the total.  The arithmetic
 * is IEEE float32 with one rounding per operation, products flushed to 0
 * below 2^-100 and a fixed exp evaluation, so it is reproducible bit for bit
 * on any IEEE float32 implementation.  In this mode the lattice hooks return
 * the rescaled forward weights in place of delta and -1 in psi.
 * temperature (sample mode only) must be finite and > 0 with a finite
 * reciprocal; MTP_EINVAL otherwise or for an unknown mode.  Takes effect at
 * the next step; every step uses the seed and temperature last set. */
#define MTP_SELECT_BEST    0
#define MTP_SELECT_SAMPLE  1
int mtp_set_sampling(mtp_ctx* ctx, int mode, float temperature, uint64_t seed);

/* The last step's uniforms, float32 [B][8] in draw order (entries r < K
 * valid), to host (synchronises); MTP_ESTATE unless the last step sampled. */
int mtp_get_uniforms(mtp_ctx* ctx, float* u);

/* The last step's union lattice (it must have used MTP_LATTICE_UNION, else
 * MTP_ESTATE), to host (synchronises): m int32 [B] state counts; states
 * int32 [B][64] (ascending ids, the first m valid); ehat, delta float32 and
 * psi int32 [B][8][64] (position t, state j; psi[.][0][.] = 0); slots int32
 * [B][K] chosen state index per position.  Any pointer may be NULL. */
int mtp_get_union_lattice(mtp_ctx* ctx, int32_t* m, int32_t* states, float* ehat,
                          float* delta, int32_t* psi, int32_t* slots);

/* Per-sequence state to host (synchronises): cached tokens, pending chunk
 * length, generated count and done flag, each int32 [B]; any may be NULL. */
int mtp_get_seq_state(mtp_ctx* ctx, int32_t* ctx_len, int32_t* pend_len,
                      int32_t* gen, int32_t* done);

/* Every token emitted since prefill, to host (synchronises): int32
 * [B][max_new]; entries at or past a sequence's generated count are
 * unspecified. */
int mtp_get_tokens(mtp_ctx* ctx, int32_t* tokens);

/* Kernel timing for measurement.  Replays the launches of kernel class
 * `kclass` (MTP_KCLASS_*) recorded for the most recent decode step (one per
 * layer, or one for the heads), in order, `iters` times on the context
 * stream; each pass is bracketed by two HIP events.  With a non-NULL
 * flush_buf (DEVICE memory owned by the caller, flush_bytes long, 16-byte
 * aligned, a multiple of 16 bytes and at least 1 KiB) each pass is preceded,
 * outside the events, by a read of that buffer; 512 MiB evicts the weights
 * from the L2 and last-level caches, as in a real step where the other
 * layers' weights pass through them between two launches of a class.  The
 * read may write one word into the buffer.  NULL and 0 time cache-warm
 * passes.  A pass repeats the recorded launches until it holds at least 12
 * (the heads' single launch is replayed 12 times, the later ones cache-warm).
 * Returns the average time per launch in microseconds (synchronises; one
 * launch latency per pass is included).  The replayed launches keep their
 * arguments and may overwrite the residual stream and the cache rows of the
 * next positions: the context needs mtp_prefill before the next decode step
 * (MTP_ESTATE otherwise).  MTP_ESTATE if the last step launched nothing of
 * the class; MTP_EINVAL for a bad class, iters < 1 or a bad buffer. */
#define MTP_KCLASS_GEMM_FFN1   1   /* LN2 -> x W_1^T -> GELU                  */
#define MTP_KCLASS_GEMM_FFN2   2   /* GELU out x W_2^T (residual partials)    */
#define MTP_KCLASS_GEMM_QKV    3   /* LN1 -> x W_qkv^T, K/V into the cache    */
#define MTP_KCLASS_ATTENTION   4   /* decode attention over the paged cache   */
#define MTP_KCLASS_HEADS       5   /* final LN -> K head projections          */
#define MTP_KCLASS_GEMM_OPROJ  6   /* attention out x W_o^T (residual part.)  */
#define MTP_KCLASS_SELECT      7   /* top_k, Viterbi lattice and accept       */
#define MTP_KCLASS_RESID_LN    8   /* residual + LayerNorm rows (batched path, two per layer) */
#define MTP_KCLASS_QKV_ATTN    9   /* LN1 -> x W_qkv^T, K/V into the cache, attention over the
                                      cached keys, in one launch (B * K <= 8 rows, d <= 1024) */
#define MTP_KCLASS_QKV_FRONT  10   /* LN1 -> x W_qkv^T, K/V into the cache, then the decode
                                      attention, in one launch whose attention workgroups wait
                                      for their head's QKV columns (B * K <= 16 rows) */
#define MTP_KCLASS_FFN_CHAIN  11   /* LN2 -> x W_1^T -> GELU, then x W_2^T (residual partials), in
                                      one launch whose W_2 workgroups wait for their K range of
                                      the GELU rows (B * K <= 16 rows) */
int mtp_profile_replay(mtp_ctx* ctx, int kclass, int iters, void* flush_buf, uint64_t flush_bytes,
                       double* avg_us);

/* ---- Transition-table estimation (Sec. 3.3: Q is derived from the
 * training corpus).  Context-free; all pointers are DEVICE pointers and the
 * work is enqueued on `hip_stream` (a hipStream_t, NULL = the null stream)
 * without host synchronisation.
 *
 * mtp_q_count adds bigram counts to counts (uint32 [vocab][vocab], row =
 * previous token, caller-zeroed; uint32 arithmetic wraps past 2^32 - 1 per
 * entry): for every utterance u = tokens[offsets[u] .. offsets[u+1]) (int32
 * tokens, int64 offsets [n_seqs + 1]), each adjacent pair inside u, and with
 * MTP_Q_COUNT_EOS also (last token of u, eos_id) for a non-empty u.  No pair
 * spans two utterances.  Input errors are counted, not fatal: status (uint64
 * [3], caller-zeroed, accumulated) gets in [0] the pairs skipped because an
 * id is outside [0, vocab), in [1] the utterances skipped because
 * 0 <= offsets[u] <= offsets[u+1] <= n_tokens does not hold, and in [2] one
 * if the utterances overlap so that they hold more pairs than n_tokens (then
 * nothing is counted).  workspace: device scratch of at least
 * mtp_q_workspace_size bytes for the same sizes (about 4 bytes per token
 * plus 60 MB for a 1025-token vocabulary), owned by the caller and not
 * shared by calls in flight.  Sizes: 0 <= n_tokens < 2^31, n_seqs >= 0,
 * 1 <= vocab <= 8192; tokens 16-byte and workspace 256-byte aligned.
 * MTP_EINVAL for other sizes or alignments, eos_id outside [0, vocab),
 * unknown flags or NULL pointers; MTP_ENOMEM if ws_bytes is too
 * small; MTP_EHIP if a launch fails.  The counts are exact integer sums: the
 * result does not depend on scheduling. */
#define MTP_Q_COUNT_EOS 1
int mtp_q_workspace_size(int64_t n_tokens, int64_t n_seqs, int vocab, uint64_t* bytes);
int mtp_q_count(const int32_t* tokens, int64_t n_tokens, const int64_t* offsets, int64_t n_seqs,
                int vocab, int eos_id, int flags, uint32_t* counts, uint64_t* status,
                void* workspace, uint64_t ws_bytes, void* hip_stream);

/* mtp_q_count without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, checks and results as
 * mtp_q_count; the scratch is a fixed array of MTP_Q_NOALLOC_SCRATCH_BYTES
 * inside the library's code object, one per GPU, held until the process
 * ends.  MTP_ENOMEM (nothing launched) when mtp_q_workspace_size reports more
 * than MTP_Q_NOALLOC_SCRATCH_BYTES for the sizes (about 10 M tokens for a
 * 1025-token vocabulary).  Calls no allocating routine.  Every call on one
 * GPU uses that GPU's one array: calls that overlap on a GPU (on different
 * streams or threads without ordering between them) race and give wrong
 * counts.  MTP_EHIP if the array's device address cannot be obtained. */
#define MTP_Q_NOALLOC_SCRATCH_BYTES (64u << 20)
int mtp_q_count_noalloc(const int32_t* tokens, int64_t n_tokens, const int64_t* offsets, int64_t n_seqs,
                        int vocab, int eos_id, int flags, uint32_t* counts, uint64_t* status, void* hip_stream);

/* log Q from the counts: logq[i][j] = float32(log(counts[i][j] + alpha) -
 * log(sum_j counts[i][j] + alpha * vocab)), evaluated in double (additive
 * smoothing alpha >= 0; alpha = 0 gives -inf for unseen pairs); a row whose
 * denominator is 0 is uniform, -log(vocab).  logq: float32 [vocab][vocab].
 * MTP_EINVAL for NULL pointers, vocab outside 1..8192 or a negative or
 * non-finite alpha. */
int mtp_q_normalize(const uint32_t* counts, int vocab, float alpha, float* logq, void* hip_stream);

/* ---- NAR module (context created with MTP_FLAG_NAR) ---------------------
 * For stage j = 2..n_q the trunk runs over each utterance's rows [phonemes;
 * prompt; target] with BIDIRECTIONAL attention (every row sees its whole
 * utterance).  Row inputs: phoneme rows the phoneme table; prompt rows the
 * sum of all n_q codebook tables at the prompt's codes; target rows the sum
 * of tables 1..j-1 at the known codes; every row adds its position (one
 * running index) and the stage vector of j.  After the final LayerNorm,
 * head j - 2 gives the target rows' logits over the vocab - 1 codes and
 * layer j is their argmax (lowest code on ties).
 *
 * mtp_nar_prepare (host arrays, copied; synchronises): B utterances with
 * phon (ids < n_phone) and phon_len[B]; prompt codes, per utterance an
 * [n_q][prompt_len[b]] block (layer-major), blocks concatenated; a1, the
 * first-layer codes of the targets, target_len[B], concatenated; codes <
 * vocab - 1; 1 <= phon + prompt + target <= max_prompt per utterance.
 * mtp_nar_run enqueues every stage on the context's stream (no host
 * synchronisation).  mtp_nar_get_codes (synchronises): per utterance
 * [k_heads][target_len[b]] (layers 2..n_q), concatenated.
 * mtp_nar_get_logits (synchronises): float32 [sum target_len][vocab - 1],
 * stage s = 0..k_heads-1 (layer s + 2), of the last run.
 * MTP_EINVAL for bad arguments or an AR context, MTP_ENOMEM if the KV pool is
 * too small, MTP_ESTATE for a run before a prepare or a get before a run. */
int mtp_nar_prepare(mtp_ctx* ctx, int B, const int32_t* phon, const int32_t* phon_len,
                    const int32_t* prompt, const int32_t* prompt_len,
                    const int32_t* a1, const int32_t* target_len);
int mtp_nar_run(mtp_ctx* ctx);
int mtp_nar_get_codes(mtp_ctx* ctx, int32_t* codes);
int mtp_nar_get_logits(mtp_ctx* ctx, int stage, float* logits);

/* Drops all sequence state (the next call must be mtp_prefill). */
int mtp_reset(mtp_ctx* ctx);
void mtp_destroy(mtp_ctx* ctx);
const char* mtp_last_error(const mtp_ctx* ctx);
const char* mtp_strerror(int code);

#ifdef __cplusplus
}
#endif
#endif /* MTP_H */
