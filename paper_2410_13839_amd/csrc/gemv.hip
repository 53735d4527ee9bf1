// Small-M (decode, M <= 16 rows) projections, bf16 MFMA, with the row-wise
// work fused in.
//
// At batch 1..4 a decode step is a chain of weight streams of 2-8 MB; each
// launch costs ~1.4 us before doing anything and every dependent global
// round trip about a microsecond, so the kernel keeps its critical path to
// one round trip plus the weight stream:
//
//  * activation rows are loaded compactly (no padding rows), each thread a
//    few float4 / 16-byte chunks, and before the weights: vmcnt retires in
//    order, so loads issued after the weight stream could only be consumed
//    after all weights landed; every load is unconditional from a clamped,
//    valid address (a predicated load compiles to a branch plus a full wait);
//  * the weight fragments of the workgroup's 16 output columns (its K range)
//    then go out at once, straight into MFMA registers; the packed weight
//    order makes every fragment one contiguous 1 KB wave load;
//  * while they stream, the prologue builds the bf16 activation tile in LDS:
//    LayerNorm of the residual rows (the residual itself is completed here:
//    h_in + the previous projection's four split-K partial sums + its bias,
//    written back once by workgroup 0), or token + position embedding + LN
//    (first layer), or the final LN of each sequence's last pending row
//    (heads), or plain bf16 rows;
//  * projections whose N is only d (out-projection, FFN2) split K four ways
//    and write partial sums, so 256 workgroups stream; their reduction is the
//    consumer's prologue above.  No workgroup waits on another: kernel
//    boundaries are the only synchronisation (device-scope fences between
//    XCDs cost tens of microseconds on this chip).
//
// MFMA: v_mfma_f32_16x16x32_bf16 with A = 16 weight rows (output columns n)
// and B = 16 activation rows (m); lane (r = l % 16, g = l / 16) supplies row
// r and k = 8g..8g+7 of each 32-wide k step, the same k for A and B.
// Activation rows >= M are never written to LDS: their garbage only reaches
// output columns >= M, which are never stored.
#include <algorithm>
#include <type_traits>

#include "attn_dec.h"
#include "common.h"
#include "launch.h"
#include "ln_rows.h"
#include "wave.h"

namespace mtp {

namespace {

__device__ __forceinline__ float wsum(float v) { return wave_sum64(v); }

__device__ __forceinline__ uint32_t pack2(float a, float b) {
    return bf16x2_bits(a, b);
}

// ---------------------------------------------------------------- epilogues
// Epilogue operands load in two steps: early(m) with the activation loads
// (phase A: it arrives before the weights), prefetch(early, m, n) after the
// weight loads, so operands that depend on early ones (the cache page of a
// key) arrive with the weights instead of one round trip after the product.
struct EpiNoEarly {};

// QKV of decode rows: row m = (seq m / Q, pending index m % Q).  K rows are
// 4 consecutive dims of one key; V goes to the transposed block (4 dims of one
// key, page_size elements apart).
struct EpiQKVDec {
    float* q;                // [M][d]
    const float* bias;       // [3d]
    const SeqState* st;
    KVView kv;
    int d, Q;
    bf16_t* qh;              // non-null: the queries go here instead, as bf16 q / 8 ([M][d])
    using Early = int2;      // the row's sequence's (ctx_len, pend_len)
    struct Pre { float b[4]; int page, slot; bool ok; };
    __device__ __forceinline__ Early early(int m) const {
        return *reinterpret_cast<const int2*>(&st[udiv_small(m, Q)]);
    }
    __device__ __forceinline__ Pre prefetch(const Early& e, int m, int n, int) const {
        Pre p;
#pragma unroll
        for (int i = 0; i < 4; ++i) p.b[i] = bias[n + i];
        // the page of the row's key (K and V^T share it); the index is
        // clamped to the block table for rows that store nothing
        const int seq = udiv_small(m, Q), i = m - seq * Q;
        const int pos = e.x + i;
        p.ok = i < e.y;
        p.slot = pos & (kv.page_size - 1);
        p.page = kv.block_table[(size_t)seq * kv.max_pages_per_seq + min(pos >> kv.page_shift, kv.max_pages_per_seq - 1)];
        return p;
    }
    __device__ __forceinline__ void store(const Pre& p, int m, int n, const float (&v)[4], int, int) const {
        const float r0 = v[0] + p.b[0], r1 = v[1] + p.b[1], r2 = v[2] + p.b[2], r3 = v[3] + p.b[3];
        if (n < d) {
            if (qh)
                *reinterpret_cast<uint2*>(qh + (size_t)m * d + n) =
                    make_uint2(pack2(r0 * 0.125f, r1 * 0.125f), pack2(r2 * 0.125f, r3 * 0.125f));
            else
                *reinterpret_cast<float4*>(q + (size_t)m * d + n) = make_float4(r0, r1, r2, r3);
            return;
        }
        if (!p.ok) return;
        const int c = (n < 2 * d) ? n - d : n - 2 * d;
        bf16_t* pool = reinterpret_cast<bf16_t*>(kv.pool);
        if (n < 2 * d) {
            bf16_t* dst = pool + kv_page_block(kv, p.page, 0, c >> 6) + (size_t)p.slot * MTP_HEAD_DIM + (c & 63);
            *reinterpret_cast<uint2*>(dst) = make_uint2(pack2(r0, r1), pack2(r2, r3));
        } else {
            bf16_t* dst = pool + kv_page_block(kv, p.page, 1, c >> 6) + (size_t)(c & 63) * kv.page_size + p.slot;
            const size_t P = kv.page_size;
            dst[0] = f32_to_bf16(r0);
            dst[P] = f32_to_bf16(r1);
            dst[2 * P] = f32_to_bf16(r2);
            dst[3 * P] = f32_to_bf16(r3);
        }
    }
};

struct EpiGeluB {
    bf16_t* out;
    const float* bias;
    int ldo;
    using Early = EpiNoEarly;
    struct Pre { float b[4]; };
    __device__ __forceinline__ Early early(int) const { return {}; }
    __device__ __forceinline__ Pre prefetch(const Early&, int, int n, int) const {
        Pre p;
#pragma unroll
        for (int i = 0; i < 4; ++i) p.b[i] = bias[n + i];
        return p;
    }
    __device__ __forceinline__ void store(const Pre& p, int m, int n, const float (&v)[4], int, int) const {
        float r[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) r[i] = gelu_erf(v[i] + p.b[i]);
        *reinterpret_cast<uint2*>(out + (size_t)m * ldo + n) = make_uint2(pack2(r[0], r[1]), pack2(r[2], r[3]));
    }
};

// FFN1 of the chained FFN: bias + GELU into the rows that FFN2 workgroups
// of the same launch poll, with device-scope stores (they reach memory, so
// that loads of the same scope on any XCD see them).  The value 0xFFFF (a
// NaN) marks a row element not yet stored, so it is never stored: a NaN
// that would round to it is stored as the canonical quiet NaN 0x7FC0.
__device__ __forceinline__ uint32_t ffn_unmark(uint32_t w) {
    if ((w & 0xFFFFu) == 0xFFFFu) w = (w & 0xFFFF0000u) | 0x7FC0u;
    if ((w >> 16) == 0xFFFFu) w = (w & 0xFFFFu) | 0x7FC00000u;
    return w;
}

struct EpiGeluShared {
    bf16_t* out;
    const float* bias;
    int ldo;
    using Early = EpiNoEarly;
    struct Pre { float b[4]; };
    __device__ __forceinline__ Early early(int) const { return {}; }
    __device__ __forceinline__ Pre prefetch(const Early&, int, int n, int) const {
        Pre p;
#pragma unroll
        for (int i = 0; i < 4; ++i) p.b[i] = bias[n + i];
        return p;
    }
    __device__ __forceinline__ void store(const Pre& p, int m, int n, const float (&v)[4], int, int) const {
        float r[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) r[i] = gelu_erf(v[i] + p.b[i]);
        const uint64_t w = (uint64_t)ffn_unmark(pack2(r[0], r[1])) | ((uint64_t)ffn_unmark(pack2(r[2], r[3])) << 32);
        __hip_atomic_store(reinterpret_cast<uint64_t*>(out + (size_t)m * ldo + n), w, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    }
};

// split-K partial sums of the out-projection / FFN2 in the form BF
// (store_partial4); the first K range also carries the residual input row
// and the bias, so the four partials sum to the complete new residual row
template <bool BF>
struct EpiPart {
    float* part;
    int ldp;        // N (= d)
    int M;
    const float* h;      // residual rows [M][N] entering the projection
    const float* bias;   // [N]
    using Early = EpiNoEarly;
    struct Pre { float4 b, x; };
    __device__ __forceinline__ Early early(int) const { return {}; }
    __device__ __forceinline__ Pre prefetch(const Early&, int m, int n, int) const {
        Pre p;
        const int nn = min(n, ldp - 4);
        p.b = *reinterpret_cast<const float4*>(bias + nn);
        p.x = *reinterpret_cast<const float4*>(h + (size_t)m * ldp + nn);
        return p;
    }
    __device__ __forceinline__ void store(const Pre& p, int m, int n, const float (&v)[4], int, int split) const {
        float4 o = make_float4(v[0], v[1], v[2], v[3]);
        if (split == 0) {
            o.x += p.b.x + p.x.x;
            o.y += p.b.y + p.x.y;
            o.z += p.b.z + p.x.z;
            o.w += p.b.w + p.x.w;
        }
        store_partial4<BF>(part, split, M, ldp, m, n, o);
    }
};

// FFN2 of the chained FFN: as EpiPart, but the residual input of the first
// K range is the sum of the previous projection's four partials (the rows
// FFN1's LayerNorm completes in the same launch), added in the order the
// LayerNorm prologue adds them.  BF: the partials' form (bfloat16 ranges 1..3
// with more than 4 rows), the same for pin and part, as both have M rows.
template <bool BF>
struct EpiPartRes {
    float* part;          // [4][M][ldp]
    int ldp;              // N (= d)
    int M;
    const float* pin;     // [4][pin_rows][ldp]: the out-projection's partials
    int pin_rows;
    const float* bias;    // [N]
    // the previous projection's partials: range 0 and ranges 1..3 as float32,
    // or as raw bfloat16 bits (converted in store(), so the loads need no
    // wait here)
    struct Pre { float4 b, p[BF ? 1 : 4]; uint2 ph[BF ? 3 : 1]; };
    __device__ __forceinline__ Pre prefetch(int m, int n, int split) const {
        Pre q;
        const int nn = min(n, ldp - 4);
        q.b = *reinterpret_cast<const float4*>(bias + nn);
        if (split == 0) {
            q.p[0] = load_partial_f32(pin, 0, pin_rows, ldp, m, nn);
#pragma unroll
            for (int s2 = 1; s2 < 4; ++s2) {
                if constexpr (BF) q.ph[s2 - 1] = load_partial_bits(pin, s2, pin_rows, ldp, m, nn);
                else q.p[s2 % (BF ? 1 : 4)] = load_partial_f32(pin, s2, pin_rows, ldp, m, nn);
            }
        }
        return q;
    }
    __device__ __forceinline__ void store(const Pre& q, int m, int n, const float (&v)[4], int split) const {
        float4 o = make_float4(v[0], v[1], v[2], v[3]);
        if (split == 0) {
            float4 p1, p2, p3;
            if constexpr (BF) {
                p1 = bf16x4_to_f32(q.ph[0]);
                p2 = bf16x4_to_f32(q.ph[1]);
                p3 = bf16x4_to_f32(q.ph[2 % (BF ? 3 : 1)]);
            } else {
                p1 = q.p[1 % (BF ? 1 : 4)];
                p2 = q.p[2 % (BF ? 1 : 4)];
                p3 = q.p[3 % (BF ? 1 : 4)];
            }
            const float4 p0 = q.p[0];
            const float x0 = (p0.x + p1.x) + (p2.x + p3.x);
            const float x1 = (p0.y + p1.y) + (p2.y + p3.y);
            const float x2 = (p0.z + p1.z) + (p2.z + p3.z);
            const float x3 = (p0.w + p1.w) + (p2.w + p3.w);
            o.x += q.b.x + x0;
            o.y += q.b.y + x1;
            o.z += q.b.z + x2;
            o.w += q.b.w + x3;
        }
        store_partial4<BF>(part, split, M, ldp, m, n, o);
    }
};

template <class E, class = void>
struct HeadForm { static constexpr int v = 0; };
template <class E>
struct HeadForm<E, std::void_t<decltype(E::PF)>> { static constexpr int v = E::PF; };

// logits of the heads.  PF: the form of the split-K partials their
// LayerNorm rows complete (store_partial4); the heads' rows are not the
// producer's, so the host picks it from the producer's row count.
template <int PFv>
struct EpiLogitsB {
    static constexpr int PF = PFv;
    float* out;
    const float* bias;
    int ldo;
    int N;
    using Early = EpiNoEarly;
    struct Pre { float b[4]; };
    __device__ __forceinline__ Early early(int) const { return {}; }
    __device__ __forceinline__ Pre prefetch(const Early&, int, int n, int) const {
        Pre p;
#pragma unroll
        for (int i = 0; i < 4; ++i) p.b[i] = bias[min(n + i, N - 1)];
        return p;
    }
    __device__ __forceinline__ void store(const Pre& p, int m, int n, const float (&v)[4], int nvalid, int) const {
        float* o = out + (size_t)m * ldo + n;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (i < nvalid) o[i] = v[i] + p.b[i];
    }
};

}  // namespace

// ------------------------------------------------------------------- kernel
// XM: 0 = bf16 rows, 1 = LN of the completed residual rows, 2 = embedding +
//     LN (decode rows of the first layer), 3 = final LN of each sequence's
//     last pending row (heads), 4 = merge of the attention key-split partials
//     of this workgroup's heads (out-projection), 5 = that merge plus the
//     pending chunk's own keys (after qkv_attn, which leaves them out).
// MR: rows (power of two >= M, <= 16); MAXF: weight fragments per wave;
// KCH: 1024-column chunks per row; MAXS: attention splits merged (XM 4, 5).
//
// 16 waves per workgroup: a CU with one workgroup of four waves keeps too few
// loads in flight to pull more than ~12-25 GB/s, with sixteen it pulls about
// twice that (measured), and every launch here is a single wave of
// workgroups, so the time is one workgroup's load latency and throughput.
// The LayerNorm modes' prologue is LnRows (ln_rows.h).
constexpr int GV_NW = 16;

// One workgroup's work: output columns [16 tile, 16 tile + 16) over K range
// `split` of S.
template <int MR, int XM, int MAXF, int KCH, int MAXS, int NW, class Epi>
__device__ __forceinline__ void gemv_body(const GemvArgs& a, const Epi& epi, const int tile, const int split,
                                          const int S) {
    constexpr int T = 64 * NW;
    extern __shared__ __attribute__((aligned(16))) bf16_t xs[];   // [16][K / S + 8], this K range
    // wave partial sums of the MFMA phase; before it, the LayerNorm gain and
    // shift ([2][K/4] float4, K <= 2048)
    __shared__ f32x4_t red[1024];
    constexpr bool LN = XM >= 1 && XM <= 3;
    // the partials' form: the heads' epilogue names it (their rows are not
    // the producer's); elsewhere it follows from MR (M > 4 iff MR > 4)
    using Rows = LnRows<MR, LN ? XM : 1, KCH, T, XM == 3 ? HeadForm<Epi>::v : (MR > 4 ? 1 : 0)>;
    __shared__ float2 s_stat[NW][LN ? Rows::RPT : 1];
    constexpr int XI = (MR * MAXF + 15) / 16;                          // 16-byte chunks per thread (XM 0)
    // XM 4: the (row, float4 column chunk) items of this K range (at most
    // MR * 64 * KCH) x the splits; GS groups of threads take every GS-th split
    constexpr int CPRM = 64 * KCH;
    constexpr int GS = (T / (MR * CPRM)) > 0 ? (T / (MR * CPRM)) : 1;
    constexpr int SPT = (MAXS + GS - 1) / GS;                          // splits per thread
    // each thread merges its own splits (group max, sum and weighted output)
    // and the GS groups combine through LDS once
    constexpr bool MERGE = XM == 4 || XM == 5;
    constexpr bool NK = XM == 5;                                       // the chunk's own keys merged here
    constexpr int NQ = NK ? MR : 1;                                    // pending rows per sequence <= MR
    __shared__ float2 s_ml[MERGE ? T : 1];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int n0 = tile * 16;
    const int K = a.K, M = a.M, N = a.N;
    const int ks = K / S;                         // this workgroup's K range
    const int kb = split * ks;
    const int nfrag = ks >> 5;
    const int nf = (nfrag - wave + NW - 1) / NW;  // fragments f = wave + NW i, i < nf
    const int ldl = ks + 8;
    // ---- A. activation-side loads (compact, from clamped addresses; branches
    //      only on wave-uniform conditions, which cost no extra waits) ----
    // LayerNorm rows (XM 1..3): the register arrays are the kernel's own
    float4 ln_hv[Rows::RPT], ln_pv[Rows::NPV][Rows::RES ? Rows::RPT : 1], ln_zv[XM == 3 ? Rows::RPT : 1];
    uint2 ln_ph[Rows::NPH][Rows::RES ? Rows::RPT : 1];
    uint2 ln_ee[XM == 2 ? Rows::RPT : 1], ln_ep[XM == 2 ? Rows::RPT : 1];
    bool ln_eok[XM == 2 ? Rows::RPT : 1];
    int ln_pl[XM == 3 ? Rows::RPT : 1];
    Rows lr{ln_hv, ln_pv, ln_ph, ln_zv, ln_ee, ln_ep, ln_eok, ln_pl};
    // bf16 chunks (XM 0) as one vector value: an array of uint4 held across
    // the barrier below is demoted to scratch by the compiler
    typedef unsigned int xq_t __attribute__((ext_vector_type(4 * XI)));
    xq_t xq;
    int2 sti = make_int2(0, 0);                  // XM 4, 5: (ctx_len, pend_len) of the item's sequence
    float2 mlv[MERGE ? SPT : 1];                 // XM 4, 5: (running max, sum) words of the thread's splits
    float4 ov[MERGE ? SPT : 1];                  // XM 4, 5: unnormalised outputs of the thread's splits
    float4 qn = make_float4(0.f, 0.f, 0.f, 0.f); // XM 5: the item's query dims, and the four dims of
    uint2 kn[NQ], vn[NQ];                        //   each pending key / value of its sequence (bf16)
    (void)qn; (void)kn; (void)vn;
#pragma unroll
    for (int j = 0; j < (MERGE ? SPT : 1); ++j) {
        ov[j] = make_float4(0.f, 0.f, 0.f, 0.f);
        mlv[j] = make_float2(-INFINITY, 0.f);
    }
    (void)xq; (void)sti; (void)mlv; (void)ov; (void)s_ml; (void)lr;
    if constexpr (XM == 0) {
        // rows [0, M) x columns [kb, kb + ks) as 16-byte chunks
        const int cpr = ks >> 3;                 // chunks per row
        const int total = M * cpr;
#pragma unroll
        for (int i = 0; i < XI; ++i) {
            const int idx = min(tid + T * i, total - 1);
            const int m = udiv_small(idx, cpr), c = (idx - m * cpr) * 8;
            const uint4 t = *reinterpret_cast<const uint4*>(a.x + (size_t)m * a.ldx + kb + c);
            xq[4 * i] = t.x;
            xq[4 * i + 1] = t.y;
            xq[4 * i + 2] = t.z;
            xq[4 * i + 3] = t.w;
        }
    } else if constexpr (MERGE) {
        // the thread's item (row, float4 chunk) in each of its splits
        // (sg, sg + GS, ...): the split's (max, sum) word of that row and
        // head and the item's unnormalised outputs; splits past the context
        // are discarded once the sequence's state is known
        const int cpr = ks >> 2, items = M * cpr;
        const int H = K >> 6, S = a.n_splits;
        const uint32_t sstride = (uint32_t)a.qt * 68;   // offsets fit 32 bits (< B*H*S*qt*68)
        const int TG = T / GS, sg = __builtin_amdgcn_readfirstlane(wave) / (TG >> 6);
        const int it = min(tid - sg * TG, items - 1);
        const int m = udiv_small(it, cpr), c = kb + (it - m * cpr) * 4;
        const int seq = udiv_small(m, a.Q), i = m - seq * a.Q;
        sti = *reinterpret_cast<const int2*>(&a.st[seq]);
        const float* e0 = a.apart + ((uint32_t)(seq * H + (c >> 6)) * S * sstride + (uint32_t)i * 68);
        // sg is uniform over a wave (groups are 256 threads or more) and S is
        // a kernel argument: skipping the splits that were not launched costs
        // no wait
#pragma unroll
        for (int j = 0; j < SPT; ++j)
            if (sg + GS * j < S) {
                const float* e = e0 + (uint32_t)(sg + GS * j) * sstride;
                mlv[j] = *reinterpret_cast<const float2*>(e);
                ov[j] = *reinterpret_cast<const float4*>(e + 4 + (c & 63));
            }
        if constexpr (NK) {
            // group 0 merges the pending chunk's own keys: the item's query
            // dims and those dims of each pending key and value of its
            // sequence (row seq Q + j of the side buffer)
            if (sg == 0) {
                qn = *reinterpret_cast<const float4*>(a.q + (size_t)m * K + c);
#pragma unroll
                for (int j = 0; j < NQ; ++j)
                    if (j < a.Q) {
                        const size_t kr = (size_t)(seq * a.Q + j) * K + c;
                        kn[j] = *reinterpret_cast<const uint2*>(a.kvnew + kr);
                        vn[j] = *reinterpret_cast<const uint2*>(a.kvnew + (size_t)M * K + kr);
                    }
            }
        }
    } else {
        lr.init(a, tid, wave);
        lr.load(a);
    }

    // the epilogue's early operands (the sequence state of the lane's row)
    const typename Epi::Early early = epi.early(min(r, M - 1));

    // Every wave's activation loads go out before any weight load: a CU
    // returns load data in request order, so an activation load queued behind
    // another wave's weight loads (HBM misses) would wait for them.
    __syncthreads();

    // ---- B. weights of this workgroup's 16 columns, all in flight: in the
    //      packed fragment order one 1 KB fragment per wave load ----
    const bf16_t* wp = a.W + ((size_t)tile * (K >> 5) + (kb >> 5)) * 512 + lane * 8;
    uint4 wv[MAXF];
#pragma unroll
    for (int i = 0; i < MAXF; ++i) {
        const int f = min(wave + NW * i, nfrag - 1);
        wv[i] = *reinterpret_cast<const uint4*>(wp + (size_t)f * 512);
    }
    // ---- C. epilogue operands ----
    const int em = r;
    const int en = n0 + 4 * g;
    const int envalid = min(4, N - en);
    const typename Epi::Pre pre = epi.prefetch(early, min(em, M - 1), min(en, N - 1), envalid);
    // every load above is issued before any of the prologue below may be
    // scheduled (the compiler otherwise sinks weight loads under the merge
    // arithmetic, serialising two memory round trips)
    __builtin_amdgcn_sched_barrier(0);

    // ---- D. activation tile in LDS ----
    if constexpr (XM == 0) {
        const int cpr = ks >> 3;
        const int total = M * cpr;
#pragma unroll
        for (int i = 0; i < XI; ++i) {
            const int idx = tid + T * i;
            if (idx < total) {
                const int m = udiv_small(idx, cpr), c = (idx - m * cpr) * 8;
                *reinterpret_cast<uint4*>(xs + (size_t)m * ldl + c) =
                    make_uint4(xq[4 * i], xq[4 * i + 1], xq[4 * i + 2], xq[4 * i + 3]);
            }
        }
    } else if constexpr (MERGE) {
        const int cpr = ks >> 2, items = M * cpr;
        const int S = a.n_splits;
        const int TG = T / GS, sg = __builtin_amdgcn_readfirstlane(wave) / (TG >> 6), it = tid - sg * TG;
        const int m = udiv_small(min(it, items - 1), cpr);
        const int c = kb + (min(it, items - 1) - m * cpr) * 4;
        const int i = m - udiv_small(m, a.Q) * a.Q;
        const int ctx = sti.x, pl = sti.y;
        // XM 4: splits past the context are not launched, their words may be
        // stale; XM 5: every split's word is written (max -inf when empty).
        // A key range fully masked for this row contributes nothing.
        const int n_active = NK ? S : min(S, udiv_small(ctx + pl + a.split_len - 1, a.split_len));
        bool live[SPT];
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < SPT; ++j) {
            live[j] = sg + GS * j < n_active && mlv[j].x != -INFINITY;
            if (live[j]) mx = fmaxf(mx, mlv[j].x);
        }
        float L = 0.f;
        f32x4_t o = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < SPT; ++j) {
            const float w = live[j] ? __expf(mlv[j].x - mx) : 0.f;
            const float4 os = live[j] ? ov[j] : make_float4(0.f, 0.f, 0.f, 0.f);
            L = fmaf(w, live[j] ? mlv[j].y : 0.f, L);
            o[0] = fmaf(w, os.x, o[0]);
            o[1] = fmaf(w, os.y, o[1]);
            o[2] = fmaf(w, os.z, o[2]);
            o[3] = fmaf(w, os.w, o[3]);
        }
        red[tid] = o;
        s_ml[tid] = make_float2(mx, L);
        __syncthreads();
        // XM 5: scores of the pending keys, q . k / 8 with q rounded to bf16
        // after the scale (as the cached keys' scores are taken): each lane
        // sums its four dims and the 16 lanes of the head (consecutive items,
        // K / 4 a multiple of 16) add theirs
        float scn[NQ];
        if constexpr (NK) {
            if (sg == 0) {
                const float q0 = bf16_to_f32(f32_to_bf16(qn.x * 0.125f)), q1 = bf16_to_f32(f32_to_bf16(qn.y * 0.125f));
                const float q2 = bf16_to_f32(f32_to_bf16(qn.z * 0.125f)), q3 = bf16_to_f32(f32_to_bf16(qn.w * 0.125f));
#pragma unroll
                for (int j = 0; j < NQ; ++j) {
                    float p = 0.f;
                    if (j < a.Q) {
                        p = q0 * __uint_as_float(kn[j].x << 16);
                        p = fmaf(q1, __uint_as_float(kn[j].x & 0xFFFF0000u), p);
                        p = fmaf(q2, __uint_as_float(kn[j].y << 16), p);
                        p = fmaf(q3, __uint_as_float(kn[j].y & 0xFFFF0000u), p);
                    }
                    scn[j] = sum16(p);
                }
            }
        }
        if (sg == 0 && it < items) {
            float gm[GS];
            float M2 = -INFINITY;
#pragma unroll
            for (int g2 = 0; g2 < GS; ++g2) {
                gm[g2] = s_ml[g2 * TG + it].x;
                M2 = fmaxf(M2, gm[g2]);
            }
            f32x4_t sum = f32x4_t{0.f, 0.f, 0.f, 0.f};
            float Lt = 0.f;
#pragma unroll
            for (int g2 = 0; g2 < GS; ++g2) {
                const float w = gm[g2] == -INFINITY ? 0.f : __expf(gm[g2] - M2);
                sum += w * red[g2 * TG + it];
                Lt = fmaf(w, s_ml[g2 * TG + it].y, Lt);
            }
            if constexpr (NK) {
                // row i attends the chunk's keys 0 .. i (its own position last)
                float M3 = M2;
#pragma unroll
                for (int j = 0; j < NQ; ++j)
                    if (j < a.Q && j <= i) M3 = fmaxf(M3, scn[j]);
                const float wo = M2 == -INFINITY ? 0.f : __expf(M2 - M3);
                sum *= wo;
                Lt *= wo;
#pragma unroll
                for (int j = 0; j < NQ; ++j)
                    if (j < a.Q && j <= i) {
                        const float p = __expf(scn[j] - M3);
                        Lt += p;
                        sum[0] = fmaf(p, __uint_as_float(vn[j].x << 16), sum[0]);
                        sum[1] = fmaf(p, __uint_as_float(vn[j].x & 0xFFFF0000u), sum[1]);
                        sum[2] = fmaf(p, __uint_as_float(vn[j].y << 16), sum[2]);
                        sum[3] = fmaf(p, __uint_as_float(vn[j].y & 0xFFFF0000u), sum[3]);
                    }
            }
            const bool valid = i < pl;
            const float inv = 1.f / Lt;
            const uint2 y = valid ? make_uint2(pack2(sum[0] * inv, sum[1] * inv), pack2(sum[2] * inv, sum[3] * inv))
                                  : make_uint2(0u, 0u);
            *reinterpret_cast<uint2*>(xs + (size_t)m * ldl + (c - kb)) = y;
        }
    } else {
        lr.build(a, tile == 0 && split == 0, xs, ldl, red, s_stat, wave, lane);
    }
    __syncthreads();

    // ---- E. MFMA over this wave's fragments ----
    f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < MAXF; ++i)
        if (i < nf) {
            const int f = wave + NW * i;
            const bf16x8_t xf = *reinterpret_cast<const bf16x8_t*>(xs + (size_t)r * ldl + f * 32 + g * 8);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wv[i]), xf, acc, 0, 0, 0);
        }

    // ---- F. sum the waves' K slices, epilogue ----
    red[wave * 64 + lane] = acc;
    __syncthreads();
    if (wave == 0 && em < M && en < N) {
        f32x4_t sum = red[lane];
#pragma unroll
        for (int w = 1; w < NW; ++w) sum += red[w * 64 + lane];
        const float v[4] = {sum[0], sum[1], sum[2], sum[3]};
        epi.store(pre, em, en, v, envalid, split);
    }
}

template <int MR, int XM, int MAXF, int KCH, int MAXS, int NW, class Epi>
__global__ __launch_bounds__(64 * NW) void gemv_kernel(GemvArgs a, Epi epi) {
    // Split-K launches (four K ranges): workgroup j takes K range j % 4 and
    // column tile j / 4, so that (the dispatcher dealing workgroups to the 8
    // XCDs in turn) each K range's workgroups share two XCDs, whose L2s then
    // hold only that range's activations (the out-projection's attention
    // split words of its four heads, FFN2's hidden columns) instead of all.
    const int S = gridDim.y;
    int tile = blockIdx.x, split = blockIdx.y;
    if (S == 4) {
        const int j = blockIdx.x + gridDim.x * blockIdx.y;
        tile = j >> 2;
        split = j & 3;
    }
    gemv_body<MR, XM, MAXF, KCH, MAXS, NW, Epi>(a, epi, tile, split, S);
}

// ---------------------------------------------------------- the fused front
// LN1 + QKV projection + decode attention of a small batch in one launch.
// The attention workgroups start with the QKV workgroups, prefetch their
// cached keys while the projection streams its weights, and then wait only
// for the 12 QKV column tiles of their own head (a flag per tile: four
// tiles each of the head's queries, keys and values), not for the whole
// projection and a launch boundary.
//
// Workgroup j runs on XCD (j + s) % 8: the dispatcher deals the workgroups
// of a launch to the 8 XCDs in turn, starting where the previous launch's
// dealing stopped (s), so workgroups j and j + 8 share an XCD (the library
// checks this once per context before it uses this kernel).  On XCD x the first 12 H / 8 workgroups are
// the QKV tiles of heads x, x + 8, ..., the rest the attention workgroups of
// those heads (batch x key splits each, split-major).  A head's producers
// and consumers thus share one L2, which carries the hand-off: the
// producers' stores and flags are plain stores, which reach it; the
// consumers read the flags, the queries and the pending keys with loads that
// skip their CU's L1.  An XCD dispatches its workgroups in order, producers
// first, so a consumer that waits never holds a CU one of its producers
// still needs.
template <int MR, int XM, int PD>
__global__ __launch_bounds__(64 * GV_NW) void qkv_front_kernel(GemvArgs a, EpiQKVDec epi, AttnMfmaArgs p,
                                                                FrontSync fs) {
    const int j = blockIdx.x, x = j & 7, loc = j >> 3;
    const int n_prod = 12 * (p.kv.n_heads >> 3);
    if (loc < n_prod) {
        const int hl = loc / 12, w = loc - 12 * hl;
        const int tile = attn_dec_detail::front_tile(fs, x + 8 * hl, w);
        gemv_body<MR, XM, 32 / GV_NW, 1, 1, GV_NW, EpiQKVDec>(a, epi, tile, 0, 1);
        // only wave 0 stores (the epilogue): once its stores are complete,
        // the tile is published
        if (threadIdx.x < 64) {
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            if (threadIdx.x == 0) fs.flags[tile] = 1u;
        }
    } else {
        // split-major: when the launch holds more workgroups than there are
        // CUs, those that wait for a CU are the last key splits, past the
        // context but at the longest
        const int cl = loc - n_prod, hpx = p.kv.n_heads >> 3, B = p.n_tiles;
        const int split = cl / (hpx * B), rem = cl - split * hpx * B;
        const int hl = rem / B, b = rem - hl * B;
        attn_dec_body<GV_NW, PD, MR, true>(p, b, x + 8 * hl, split, p.kv.n_heads, fs);
    }
}

// ------------------------------------------------------ the chained FFN
// FFN2 workgroup of the chained FFN: output columns [16 tile, 16 tile + 16)
// over K range `split` of four.  Its weights and epilogue operands go out
// first (they depend on nothing in this launch); then it polls its K range
// of the hidden rows, written by FFN1 workgroups of the same launch, with
// device-scope loads until none holds the sentinel, and finishes as the
// plain GEMV does.
__device__ __forceinline__ bool ffn_marked(uint64_t v) {
    const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
    return (lo & 0xFFFFu) == 0xFFFFu || (lo >> 16) == 0xFFFFu || (hi & 0xFFFFu) == 0xFFFFu || (hi >> 16) == 0xFFFFu;
}

template <int MR, int MAXF, int NW>
__device__ __forceinline__ void ffn2_chain_body(const GemvArgs& a, const EpiPartRes<(MR > 4)>& epi, const int tile,
                                                const int split, const FfnSync& fs) {
    constexpr int T = 64 * NW;
    constexpr int XI = (MR * MAXF + 15) / 16;     // 16-byte row chunks per thread
    extern __shared__ __attribute__((aligned(16))) bf16_t xs[];   // [16][K / 4 + 8]
    __shared__ f32x4_t red2[64 * NW];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int K = a.K, M = a.M, N = a.N;
    const int ks = K >> 2, kb = split * ks;
    const int nfrag = ks >> 5;
    const int nf = (nfrag - wave + NW - 1) / NW;
    const int ldl = ks + 8;
    // weights of the 16 columns over this K range, one 1 KB fragment per wave load
    const bf16_t* wp = a.W + ((size_t)tile * (K >> 5) + (kb >> 5)) * 512 + lane * 8;
    uint4 wv[MAXF];
    // Up to 8 rows the kernel fits two workgroups per CU (at most 60
    // registers), so an FFN2 workgroup shares its CU with an FFN1 tile: its
    // weight loads wait ~1 us (2,560 clocks) so that the tile's LayerNorm
    // rows and weights, the launch's critical path, go out first (a CU
    // returns loads in request order).  Measured at batch 1, K = 4: 252.5
    // us per step with no delay, 243-244.5 us for 1,500-3,600 clocks,
    // 254.5 us loading the weights only after the wait; K = 8: 296.4
    // against 288.8 us.  With one workgroup per CU (16 rows) the FFN2
    // workgroups start after FFN1 tiles end, and a delay only adds to the
    // step.
    if constexpr (MR <= 8) __builtin_amdgcn_s_sleep(40);
#pragma unroll
    for (int i = 0; i < MAXF; ++i) {
        const int f = min(wave + NW * i, nfrag - 1);
        wv[i] = *reinterpret_cast<const uint4*>(wp + (size_t)f * 512);
    }
    const int em = r, en = tile * 16 + 4 * g;
    typename EpiPartRes<(MR > 4)>::Pre pre{};
    if (wave == 0) pre = epi.prefetch(min(em, M - 1), min(en, N - 1), split);
    __builtin_amdgcn_sched_barrier(0);
    // the hidden rows [0, M) x [kb, kb + ks): while FFN1 runs, wave 0 polls
    // one word of each FFN1 tile of the range (a few hundred bytes a round,
    // instead of every row chunk of every wave competing with FFN1's weight
    // stream); then the waves that hold row chunks poll those until none
    // holds the sentinel.  Both waits are bounded; one that runs out is
    // counted.
    const int cpr = ks >> 3, total = M * cpr;
    uint64_t xv[XI][2];
#pragma unroll
    for (int i = 0; i < XI; ++i) xv[i][0] = xv[i][1] = 0;
    bool ready = true;
    if (wave == 0) {
        const uint64_t* probe = reinterpret_cast<const uint64_t*>(a.x + kb + 16 * min(lane, (ks >> 4) - 1));
        ready = false;
        for (int s = 0; s < fs.spin; ++s) {
            const uint64_t v = __hip_atomic_load(probe, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (__all(!ffn_marked(v))) { ready = true; break; }
            __builtin_amdgcn_s_sleep(2);
        }
    }
    __syncthreads();
    if (wave * 64 < total) {              // uniform: the wave holds row chunks
        bool done = false;
        for (int s = 0; s < fs.spin; ++s) {
            bool marked = false;
#pragma unroll
            for (int i = 0; i < XI; ++i) {
                const int idx = min(tid + T * i, total - 1);
                const int m = udiv_small(idx, cpr), c = (idx - m * cpr) * 8;
                const uint64_t* p = reinterpret_cast<const uint64_t*>(a.x + (size_t)m * a.ldx + kb + c);
                xv[i][0] = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                xv[i][1] = __hip_atomic_load(p + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                marked |= ffn_marked(xv[i][0]) || ffn_marked(xv[i][1]);
            }
            if (__all(!marked)) { done = true; break; }
            __builtin_amdgcn_s_sleep(2);
        }
        ready = ready && done;
    }
    if (!ready && lane == 0) atomicAdd(fs.err, 1u);
#pragma unroll
    for (int i = 0; i < XI; ++i) {
        const int idx = tid + T * i;
        if (idx < total) {
            const int m = udiv_small(idx, cpr), c = (idx - m * cpr) * 8;
            *reinterpret_cast<uint4*>(xs + (size_t)m * ldl + c) =
                make_uint4((uint32_t)xv[i][0], (uint32_t)(xv[i][0] >> 32), (uint32_t)xv[i][1],
                           (uint32_t)(xv[i][1] >> 32));
        }
    }
    __syncthreads();
    f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < MAXF; ++i)
        if (i < nf) {
            const int f = wave + NW * i;
            const bf16x8_t xf = *reinterpret_cast<const bf16x8_t*>(xs + (size_t)r * ldl + f * 32 + g * 8);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wv[i]), xf, acc, 0, 0, 0);
        }
    red2[wave * 64 + lane] = acc;
    __syncthreads();
    if (wave == 0 && em < M && en < N) {
        f32x4_t sum = red2[lane];
#pragma unroll
        for (int w = 1; w < NW; ++w) sum += red2[w * 64 + lane];
        const float v[4] = {sum[0], sum[1], sum[2], sum[3]};
        epi.store(pre, em, en, v, split);
    }
}

// LN2 + FFN1 + GELU and FFN2 of a small batch in one launch.  Workgroups
// j < d_ff / 16 are FFN1 column tiles (the plain GEMV with its LayerNorm
// prologue); the rest are FFN2 workgroups (column tile c / 4, K range
// c % 4), which start with FFN1, stream their weights meanwhile and wait
// only for the FFN1 tiles of their K range.  Those tiles lie on every XCD,
// so the hand-off goes through memory (device-scope stores and loads);
// it needs no flag: the rows themselves start as the sentinel.  FFN1
// workgroups precede every FFN2 workgroup in dispatch order and wait for
// nothing, so a waiting FFN2 workgroup never holds a CU an FFN1 tile still
// needs.  Each FFN1 tile also refills its columns of the next launch's
// rows (all 16 rows) with the sentinel, after its own work.
template <int MR, int MAXF2>
__global__ __launch_bounds__(64 * GV_NW) void ffn_chain_kernel(GemvArgs a1, EpiGeluShared e1, GemvArgs a2,
                                                                EpiPartRes<(MR > 4)> e2, FfnSync fs) {
    const int j = blockIdx.x;
    const int n_prod = a1.N >> 4;
    if (j < n_prod) {
        gemv_body<MR, 1, 32 / GV_NW, 1, 1, GV_NW, EpiGeluShared>(a1, e1, j, 0, 1);
        if (threadIdx.x >= 64 && threadIdx.x < 128) {
            const int l = threadIdx.x - 64;
            *reinterpret_cast<uint2*>(fs.next + (size_t)(l >> 2) * a1.ldo + j * 16 + (l & 3) * 4) =
                make_uint2(0xFFFFFFFFu, 0xFFFFFFFFu);
        }
    } else {
        const int c = j - n_prod;
        ffn2_chain_body<MR, MAXF2, GV_NW>(a2, e2, c >> 2, c & 3, fs);
    }
}

// Records, for each residue j % 8 of the workgroups of a launch of 1024
// threads, the set of XCDs (a bit each) they ran on.
__global__ __launch_bounds__(1024) void xcd_deal_check_kernel(unsigned* masks) {
    if (threadIdx.x == 0) {
        unsigned x;
        asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
        atomicOr(&masks[blockIdx.x & 7u], 1u << (x & 0xFu));
    }
}

// --------------------------------------------------------------- launching
template <int MR, int XM, int MAXF, int KCH, int MAXS, class Epi, int NW = GV_NW>
static hipError_t gemv_go(hipStream_t st, const GemvArgs& a, int splits, const Epi& e) {
    dim3 grid((a.N + 15) / 16, splits);
    const size_t lds = (size_t)16 * (a.K / splits + 8) * 2;
    static bool attr_set = false;
    if (lds > 32 * 1024 && !attr_set) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemv_kernel<MR, XM, MAXF, KCH, MAXS, NW, Epi>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, 128 * 1024);
        if (err != hipSuccess) return err;
        attr_set = true;
    }
    hipLaunchKernelGGL((gemv_kernel<MR, XM, MAXF, KCH, MAXS, NW, Epi>), grid, dim3(64 * NW), lds, st, a, e);
    return hipGetLastError();
}

// LayerNorm modes: K = d_model <= 2048, one K range
template <int XM, class Epi, int NW = GV_NW>
static hipError_t gemv_ln(hipStream_t st, const GemvArgs& a, const Epi& e) {
    // mode 1 reads the partials in the form its own row count implies
    if (XM == 1 && a.part_on && partials_bf16(a.part_rows) != partials_bf16(a.M)) return hipErrorInvalidValue;
    const bool wide = a.K > 1024;
    constexpr int MF = 32 / NW;                   // fragments per wave at K = 1024
#define MTP_GEMV_LN(MR) \
    return wide ? gemv_go<MR, XM, 2 * MF, 2, 1, Epi, NW>(st, a, 1, e) : gemv_go<MR, XM, MF, 1, 1, Epi, NW>(st, a, 1, e)
    if (a.M <= 1) MTP_GEMV_LN(1);
    if (a.M <= 2) MTP_GEMV_LN(2);
    if (a.M <= 4) MTP_GEMV_LN(4);
    if (a.M <= 8) MTP_GEMV_LN(8);
    MTP_GEMV_LN(16);
#undef MTP_GEMV_LN
}

// split-K partial producers (four K ranges) over bf16 rows
template <int MR>
static hipError_t gemv_part_rows(hipStream_t st, const GemvArgs& a) {
    const EpiPart<(MR > 4)> e{a.part_out, a.N, a.M, a.h, a.bias};   // M > 4 iff MR > 4
    const int per_wave = (a.K / 4 / 32 + GV_NW - 1) / GV_NW;
    if (per_wave <= 1) return gemv_go<MR, 0, 1, 1, 1>(st, a, 4, e);
    if (per_wave <= 2) return gemv_go<MR, 0, 2, 1, 1>(st, a, 4, e);
    if (per_wave <= 4) return gemv_go<MR, 0, 4, 1, 1>(st, a, 4, e);
    return gemv_go<MR, 0, 8, 1, 1>(st, a, 4, e);
}

// split-K partial producer over merged attention partials (K = d <= 2048)
template <int MR, int KCH, int XM = 4>
static hipError_t gemv_part_merge(hipStream_t st, const GemvArgs& a) {
    const EpiPart<(MR > 4)> e{a.part_out, a.N, a.M, a.h, a.bias};   // M > 4 iff MR > 4
    constexpr int GS = (16 / (MR * KCH)) > 0 ? 16 / (MR * KCH) : 1;
    if (a.n_splits <= 8) return gemv_go<MR, XM, 1, KCH, 8>(st, a, 4, e);
    if constexpr (8 * GS >= 16) {
        if (a.n_splits <= 16) return gemv_go<MR, XM, 1, KCH, 16>(st, a, 4, e);
    }
    if constexpr (XM == 4 && 8 * GS >= 32) {
        if (a.n_splits <= 24) return gemv_go<MR, XM, 1, KCH, 24>(st, a, 4, e);
        if (a.n_splits <= 32) return gemv_go<MR, XM, 1, KCH, 32>(st, a, 4, e);
    }
    return hipErrorInvalidValue;
}

// Largest attention split count the out-projection can merge for M rows of
// width d: each thread keeps at most 8 splits of one (row, float4) item, and
// the workgroup's 1024 threads cover the items GS times over; 0 if none.
int gemv_merge_max_splits(int M, int d) {
    if (M < 1 || M > 16 || d > 2048) return 0;
    int mr = 1;
    while (mr < M) mr <<= 1;
    const int kch = d > 1024 ? 2 : 1;
    const int gs = std::max(1, 16 / (mr * kch));
    return std::min(32, 8 * gs);
}

bool qkv_front_ok(int rows, int d, int n_heads, int batch, int split_len, int n_splits) {
    return rows >= 1 && rows <= 16 && d <= 1024 && d % 256 == 0 && n_heads % 8 == 0 && n_heads * 64 == d &&
           batch >= 1 && rows % batch == 0 && (split_len == 256 || split_len == 512) && n_splits >= 1 &&
           n_splits <= 64 && (int64_t)8 * (12 + batch * n_splits) * (n_heads / 8) <= 65535;
}

template <int MR, int XM, int PD>
static hipError_t qkv_front_go(hipStream_t st, const GemvArgs& a, const EpiQKVDec& e, const AttnMfmaArgs& p,
                               const FrontSync& fs) {
    const size_t lds = std::max<size_t>((size_t)16 * (a.K + 8) * 2, (size_t)GV_NW * MR * 64 * sizeof(float));
    static bool attr_set = false;
    if (lds > 32 * 1024 && !attr_set) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(&qkv_front_kernel<MR, XM, PD>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, 128 * 1024);
        if (err != hipSuccess) return err;
        attr_set = true;
    }
    const int hpx = p.kv.n_heads / 8;
    const int grid = 8 * hpx * (12 + fs.per_head);
    hipLaunchKernelGGL((qkv_front_kernel<MR, XM, PD>), dim3(grid), dim3(64 * GV_NW), lds, st, a, e, p, fs);
    return hipGetLastError();
}

template <int XM, int PD>
static hipError_t qkv_front_mr(hipStream_t st, const GemvArgs& a, const EpiQKVDec& e, const AttnMfmaArgs& p,
                               const FrontSync& fs) {
    if (a.M <= 1) return qkv_front_go<1, XM, PD>(st, a, e, p, fs);
    if (a.M <= 2) return qkv_front_go<2, XM, PD>(st, a, e, p, fs);
    if (a.M <= 4) return qkv_front_go<4, XM, PD>(st, a, e, p, fs);
    if (a.M <= 8) return qkv_front_go<8, XM, PD>(st, a, e, p, fs);
    return qkv_front_go<16, XM, PD>(st, a, e, p, fs);
}

hipError_t qkv_front(hipStream_t st, const GemvArgs& a, const AttnMfmaArgs& p, const FrontSync& fs) {
    const int H = p.kv.n_heads;
    if (a.epi != EPI_QKV || (a.xmode != 1 && a.xmode != 2) || a.N != 3 * a.K || a.d != a.K || p.mode != 0 ||
        p.kv.page_size != 16 || p.Q < 1 || p.Q > 16 || p.qt < p.Q || a.Q != p.Q || p.n_tiles * p.Q != a.M ||
        p.ldq != a.K || !p.qh || p.qh != a.qh || !qkv_front_ok(a.M, a.K, H, p.n_tiles, p.split_len, p.n_splits) ||
        fs.tiles_per_mat * 16 != a.K || fs.per_head != p.n_tiles * p.n_splits || !fs.flags || !fs.next_flags ||
        fs.flags == fs.next_flags || !fs.err || fs.spin < 0)
        return hipErrorInvalidValue;
    EpiQKVDec e{a.q, a.bias, a.st, a.kv, a.d, a.Q, a.qh};
    const bool pd2 = p.split_len == 512;
    if (a.xmode == 2) return pd2 ? qkv_front_mr<2, 2>(st, a, e, p, fs) : qkv_front_mr<2, 1>(st, a, e, p, fs);
    return pd2 ? qkv_front_mr<1, 2>(st, a, e, p, fs) : qkv_front_mr<1, 1>(st, a, e, p, fs);
}

bool ffn_chain_ok(int rows, int d, int d_ff) {
    return rows >= 1 && rows <= 16 && d >= 256 && d <= 1024 && d % 256 == 0 && d_ff >= 512 && d_ff % 512 == 0 &&
           d_ff / 4 <= 2 * GV_NW * 32;
}

template <int MR>
static hipError_t ffn_chain_go(hipStream_t st, const GemvArgs& a1, const EpiGeluShared& e1, const GemvArgs& a2,
                               const FfnSync& fs) {
    const EpiPartRes<(MR > 4)> e2{a2.part_out, a2.N, a2.M, a2.part, a2.part_rows, a2.bias};
    // the static LDS (two 16 KB reduction arrays) and this together stay
    // within the CU's 160 KB: raise the dynamic limit only as far as needed
    const size_t lds = (size_t)16 * (std::max(a1.K, a2.K / 4) + 8) * 2;
    static size_t attr_set = 32 * 1024;
    if (lds > attr_set) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(&ffn_chain_kernel<MR, 2>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (err != hipSuccess) return err;
        attr_set = lds;
    }
    const int grid = a1.N / 16 + (a2.N / 16) * 4;
    hipLaunchKernelGGL((ffn_chain_kernel<MR, 2>), dim3(grid), dim3(64 * GV_NW), lds, st, a1, e1, a2, e2, fs);
    return hipGetLastError();
}

hipError_t ffn_chain(hipStream_t st, const GemvArgs& a1, const GemvArgs& a2, const FfnSync& fs) {
    if (a1.epi != EPI_GELU || a1.xmode != 1 || a2.epi != EPI_PARTIAL || a2.xmode != 0 || a1.M != a2.M ||
        !ffn_chain_ok(a1.M, a1.K, a1.N) || a2.K != a1.N || a2.N != a1.K || a1.ldo != a1.N || a2.ldx != a1.N ||
        a2.x != a1.out || !a1.out || !a2.part || !a2.part_out || a2.part == a2.part_out || a2.part_rows < a2.M ||
        partials_bf16(a2.part_rows) != partials_bf16(a2.M) || !fs.next || fs.next == a1.out || !fs.err ||
        fs.spin < 0)
        return hipErrorInvalidValue;
    EpiGeluShared e1{(bf16_t*)a1.out, a1.bias, a1.ldo};
    if (a1.M <= 1) return ffn_chain_go<1>(st, a1, e1, a2, fs);
    if (a1.M <= 2) return ffn_chain_go<2>(st, a1, e1, a2, fs);
    if (a1.M <= 4) return ffn_chain_go<4>(st, a1, e1, a2, fs);
    if (a1.M <= 8) return ffn_chain_go<8>(st, a1, e1, a2, fs);
    return ffn_chain_go<16>(st, a1, e1, a2, fs);
}

hipError_t xcd_deal_check(hipStream_t st, unsigned* masks, int grid) {
    if (!masks || grid < 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(xcd_deal_check_kernel, dim3(grid), dim3(1024), 0, st, masks);
    return hipGetLastError();
}

hipError_t gemv(hipStream_t st, const GemvArgs& a) {
    if (a.M < 1 || a.M > 16 || a.N < 4 || a.K % 128) return hipErrorInvalidValue;
    if (a.epi == EPI_PARTIAL) {
        if (a.N % 4 || a.K > 4 * 8 * GV_NW * 32) return hipErrorInvalidValue;
        if (a.xmode == 5) {
            // after qkv_attn: <= 8 rows, d <= 1024, every split word written
            if (a.M > 8 || a.K > 1024 || a.K % 256 || a.n_splits < 1 || a.Q < 1 || a.M % a.Q ||
                a.n_splits > gemv_merge_max_splits(a.M, a.K) || a.n_splits > 16 || !a.q || !a.kvnew)
                return hipErrorInvalidValue;
            if (a.M <= 1) return gemv_part_merge<1, 1, 5>(st, a);
            if (a.M <= 2) return gemv_part_merge<2, 1, 5>(st, a);
            if (a.M <= 4) return gemv_part_merge<4, 1, 5>(st, a);
            return gemv_part_merge<8, 1, 5>(st, a);
        }
        if (a.xmode == 4) {
            if (a.K > 2048 || a.K % 256 || a.n_splits < 1 || a.Q < 1 ||
                a.n_splits > gemv_merge_max_splits(a.M, a.K) || a.split_len < 1)
                return hipErrorInvalidValue;
            const bool wide = a.K > 1024;
#define MTP_GEMV_MERGE(MR) return wide ? gemv_part_merge<MR, 2>(st, a) : gemv_part_merge<MR, 1>(st, a)
            if (a.M <= 1) MTP_GEMV_MERGE(1);
            if (a.M <= 2) MTP_GEMV_MERGE(2);
            if (a.M <= 4) MTP_GEMV_MERGE(4);
            if (a.M <= 8) MTP_GEMV_MERGE(8);
            MTP_GEMV_MERGE(16);
#undef MTP_GEMV_MERGE
        }
        if (a.xmode != 0) return hipErrorInvalidValue;
        if (a.M <= 1) return gemv_part_rows<1>(st, a);
        if (a.M <= 2) return gemv_part_rows<2>(st, a);
        if (a.M <= 4) return gemv_part_rows<4>(st, a);
        if (a.M <= 8) return gemv_part_rows<8>(st, a);
        return gemv_part_rows<16>(st, a);
    }
    if (a.K > 2048 || a.K % 256 || (a.epi != EPI_LOGITS && a.N % 4)) return hipErrorInvalidValue;
    switch (a.epi) {
    case EPI_QKV: {
        EpiQKVDec e{a.q, a.bias, a.st, a.kv, a.d, a.Q, nullptr};
        if (a.xmode == 2) return gemv_ln<2>(st, a, e);
        if (a.xmode == 1) return gemv_ln<1>(st, a, e);
        return hipErrorInvalidValue;
    }
    case EPI_GELU: {
        EpiGeluB e{(bf16_t*)a.out, a.bias, a.ldo};
        if (a.xmode == 1) return gemv_ln<1>(st, a, e);
        return hipErrorInvalidValue;
    }
    case EPI_LOGITS: {
        // K x 1025 columns is a few tiles more than there are CUs: 8-wave
        // workgroups, two per CU, so the extra tiles do not form a second round
        if (a.xmode != 3) return hipErrorInvalidValue;
        if (a.part_on && partials_bf16(a.part_rows)) {
            EpiLogitsB<1> e{(float*)a.out, a.bias, a.ldo, a.N};
            return gemv_ln<3, EpiLogitsB<1>, 8>(st, a, e);
        }
        EpiLogitsB<0> e{(float*)a.out, a.bias, a.ldo, a.N};
        return gemv_ln<3, EpiLogitsB<0>, 8>(st, a, e);
    }
    }
    return hipErrorInvalidValue;
}

}  // namespace mtp
