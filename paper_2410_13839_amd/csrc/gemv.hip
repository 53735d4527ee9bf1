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

#include "common.h"
#include "launch.h"
#include "wave.h"

namespace mtp {

namespace {

__device__ __forceinline__ float wsum(float v) { return wave_sum64(v); }

__device__ __forceinline__ uint32_t pack2(float a, float b) {
    return (uint32_t)f32_to_bf16(a) | ((uint32_t)f32_to_bf16(b) << 16);
}

// ---------------------------------------------------------------- epilogues
// QKV of decode rows: row m = (seq m / Q, pending index m % Q).  K rows are
// 4 consecutive dims of one key; V goes to the transposed block (4 dims of one
// key, page_size elements apart).
struct EpiQKVDec {
    float* q;                // [M][d]
    const float* bias;       // [3d]
    const SeqState* st;
    KVView kv;
    int d, Q;
    struct Pre { float b[4]; int ctx, pl; };
    __device__ __forceinline__ Pre prefetch(int m, int n, int) const {
        Pre p;
#pragma unroll
        for (int i = 0; i < 4; ++i) p.b[i] = bias[n + i];
        const SeqState& s = st[udiv_small(m, Q)];
        p.ctx = s.ctx_len;
        p.pl = s.pend_len;
        return p;
    }
    __device__ __forceinline__ void store(const Pre& p, int m, int n, const float (&v)[4], int) const {
        const float r0 = v[0] + p.b[0], r1 = v[1] + p.b[1], r2 = v[2] + p.b[2], r3 = v[3] + p.b[3];
        if (n < d) {
            *reinterpret_cast<float4*>(q + (size_t)m * d + n) = make_float4(r0, r1, r2, r3);
            return;
        }
        const int seq = udiv_small(m, Q), i = m - seq * Q;
        if (i >= p.pl) return;
        const int pos = p.ctx + i;
        const int c = (n < 2 * d) ? n - d : n - 2 * d;
        bf16_t* pool = reinterpret_cast<bf16_t*>(kv.pool);
        if (n < 2 * d) {
            bf16_t* dst = pool + kv.offset(seq, pos, 0, c >> 6) + (c & 63);
            *reinterpret_cast<uint2*>(dst) = make_uint2(pack2(r0, r1), pack2(r2, r3));
        } else {
            bf16_t* dst = pool + kv.vt_offset(seq, pos, c >> 6) + (size_t)(c & 63) * kv.page_size;
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
    struct Pre { float b[4]; };
    __device__ __forceinline__ Pre prefetch(int, int n, int) const {
        Pre p;
#pragma unroll
        for (int i = 0; i < 4; ++i) p.b[i] = bias[n + i];
        return p;
    }
    __device__ __forceinline__ void store(const Pre& p, int m, int n, const float (&v)[4], int) const {
        float r[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) r[i] = gelu_erf(v[i] + p.b[i]);
        *reinterpret_cast<uint2*>(out + (size_t)m * ldo + n) = make_uint2(pack2(r[0], r[1]), pack2(r[2], r[3]));
    }
};

// split-K partial sums of the out-projection / FFN2: part[split][m][n]; the
// first K range also carries the residual input row and the bias, so the
// four partials sum to the complete new residual row
struct EpiPart {
    float* part;
    int ldp;        // N (= d)
    int M;
    const float* h;      // residual rows [M][N] entering the projection
    const float* bias;   // [N]
    struct Pre { float4 b, x; };
    __device__ __forceinline__ Pre prefetch(int m, int n, int) const {
        Pre p;
        const int nn = min(n, ldp - 4);
        p.b = *reinterpret_cast<const float4*>(bias + nn);
        p.x = *reinterpret_cast<const float4*>(h + (size_t)m * ldp + nn);
        return p;
    }
    __device__ __forceinline__ void store(const Pre& p, int m, int n, const float (&v)[4], int) const {
        float4 o = make_float4(v[0], v[1], v[2], v[3]);
        if (blockIdx.y == 0) {
            o.x += p.b.x + p.x.x;
            o.y += p.b.y + p.x.y;
            o.z += p.b.z + p.x.z;
            o.w += p.b.w + p.x.w;
        }
        *reinterpret_cast<float4*>(part + ((size_t)blockIdx.y * M + m) * ldp + n) = o;
    }
};

struct EpiLogitsB {
    float* out;
    const float* bias;
    int ldo;
    int N;
    struct Pre { float b[4]; };
    __device__ __forceinline__ Pre prefetch(int, int n, int) const {
        Pre p;
#pragma unroll
        for (int i = 0; i < 4; ++i) p.b[i] = bias[min(n + i, N - 1)];
        return p;
    }
    __device__ __forceinline__ void store(const Pre& p, int m, int n, const float (&v)[4], int nvalid) const {
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
//     of this workgroup's heads (out-projection).
// MR: rows (power of two >= M, <= 16); MAXF: weight fragments per wave;
// KCH: 1024-column chunks per row; MAXS: attention splits merged (XM 4).
//
// 16 waves per workgroup: a CU with one workgroup of four waves keeps too few
// loads in flight to pull more than ~12-25 GB/s, with sixteen it pulls about
// twice that (measured), and every launch here is a single wave of
// workgroups, so the time is one workgroup's load latency and throughput.
// LayerNorm-mode prologue: thread t owns the float4 column chunk t % (K/4) of
// rows t / (K/4), t / (K/4) + RG, ... (RG = 1024 / (K/4) row groups), so the
// LayerNorm parameters are loaded once per thread and a row's statistics
// are a reduction over the K/4/64 waves of its row group.
constexpr int GV_NW = 16;

template <int MR, int XM, int MAXF, int KCH, int MAXS, int NW, class Epi>
__global__ __launch_bounds__(64 * NW) void gemv_kernel(GemvArgs a, Epi epi) {
    constexpr int T = 64 * NW;
    extern __shared__ __attribute__((aligned(16))) bf16_t xs[];   // [16][K / S + 8], this K range
    // wave partial sums of the MFMA phase; before it, the LayerNorm gain and
    // shift ([2][K/4] float4, K <= 2048)
    __shared__ f32x4_t red[1024];
    constexpr bool LN = XM >= 1 && XM <= 3;
    constexpr bool RES = XM == 1 || XM == 3;                           // residual completed here
    constexpr int RPT = (MR * KCH * 256 + T - 1) / T;                  // rows per thread (LN modes)
    __shared__ float2 s_stat[NW][LN ? RPT : 1];
    constexpr int XI = (MR * MAXF + 15) / 16;                          // 16-byte chunks per thread (XM 0)
    // XM 4: the (row, float4 column chunk) items of this K range (at most
    // MR * 64 * KCH) x the splits; GS groups of threads take every GS-th split
    constexpr int CPRM = 64 * KCH;
    constexpr int GS = (T / (MR * CPRM)) > 0 ? (T / (MR * CPRM)) : 1;
    constexpr int SPT = (MAXS + GS - 1) / GS;                          // splits per thread
    // each thread merges its own splits (group max, sum and weighted output)
    // and the GS groups combine through LDS once
    __shared__ float2 s_ml[XM == 4 ? T : 1];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int n0 = blockIdx.x * 16;
    const int S = gridDim.y, split = blockIdx.y;
    const int K = a.K, M = a.M, N = a.N;
    const int ks = K / S;                         // this workgroup's K range
    const int kb = split * ks;
    const int nfrag = ks >> 5;
    const int nf = (nfrag - wave + NW - 1) / NW;  // fragments f = wave + NW i, i < nf
    const int ldl = ks + 8;
    // LayerNorm-mode mapping; rg is uniform over a wave (K/4 is a multiple of 64)
    const int K4 = K >> 2;
    const int RG = T / K4;                        // row groups (>= 1 for K <= 2048)
    const int rg = __builtin_amdgcn_readfirstlane(wave) / (K4 >> 6);   // scalar division
    const int cc = min((tid - rg * K4) * 4, K - 4);
    (void)RG; (void)rg; (void)cc; (void)K4;

    // ---- A. activation-side loads (compact, from clamped addresses; branches
    //      only on wave-uniform conditions, which cost no extra waits) ----
    float4 hv[LN ? RPT : 1];                     // residual / embedding rows
    float4 pv[RES ? 4 : 1][RES ? RPT : 1];       // split-K partials of the producer
    float4 zv[XM == 3 ? RPT : 1];                // prefill hidden state (heads, first step)
    uint2 emb_e[XM == 2 ? RPT : 1], emb_p[XM == 2 ? RPT : 1];   // first layer: embedding, position rows
    bool emb_ok[XM == 2 ? RPT : 1];
    float4 gv = make_float4(0.f, 0.f, 0.f, 0.f), bv = gv;
    // bf16 chunks (XM 0) as one vector value: an array of uint4 held across
    // the barrier below is demoted to scratch by the compiler
    typedef unsigned int xq_t __attribute__((ext_vector_type(4 * XI)));
    xq_t xq;
    int st_pl[XM == 3 ? RPT : 1];
    int2 sti = make_int2(0, 0);                  // XM 4: (ctx_len, pend_len) of the item's sequence
    float2 mlv[XM == 4 ? SPT : 1];               // XM 4: (running max, sum) words of the thread's splits
    float4 ov[XM == 4 ? SPT : 1];                // XM 4: unnormalised outputs of the thread's splits
#pragma unroll
    for (int j = 0; j < (XM == 4 ? SPT : 1); ++j) {
        ov[j] = make_float4(0.f, 0.f, 0.f, 0.f);
        mlv[j] = make_float2(-INFINITY, 0.f);
    }
    (void)pv; (void)zv; (void)xq; (void)st_pl; (void)sti; (void)mlv; (void)ov; (void)gv; (void)bv; (void)hv;
    (void)s_ml; (void)emb_e; (void)emb_p; (void)emb_ok;
    const bool has_part = a.part_on != 0;      // kernel argument: uniform
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
    } else if constexpr (XM == 4) {
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
    } else {
        // LayerNorm gain and shift: loaded by row group 0 only, shared through LDS
        if (rg == 0) {
            gv = *reinterpret_cast<const float4*>(a.g + cc);
            bv = *reinterpret_cast<const float4*>(a.beta + cc);
        }
        if constexpr (XM == 2) {
            // first layer: each pending token's embedding and position rows;
            // the sequence state first, then the rows it names, so that they
            // arrive ahead of the weights (loads return in request order)
#pragma unroll
            for (int j = 0; j < RPT; ++j) {
                const int m = rg + RG * j;
                if (m < M && rg < RG) {
                    const int seq = m / a.Q, i = m - seq * a.Q;
                    const SeqState& st = a.st[seq];
                    const bool valid = i < st.pend_len;
                    emb_ok[j] = valid;
                    emb_e[j] = *reinterpret_cast<const uint2*>(a.emb + (size_t)(valid ? st.pend_ids[i] : 0) * K + cc);
                    emb_p[j] = *reinterpret_cast<const uint2*>(a.pos + (size_t)(valid ? st.ctx_len + i : 0) * K + cc);
                }
            }
        }
        if constexpr (RES) {
            // XM 1: row m; XM 3: the last row of sequence m's pending chunk,
            // plus the prefill state (chosen once the state is in).  With
            // partials the four of them sum to the row (the first carries the
            // residual input and bias); without, the row is h itself.
#pragma unroll
            for (int j = 0; j < RPT; ++j) {
                const int m = rg + RG * j;
                if (m < M && rg < RG) {
                    const int row = (XM == 1) ? m : ((a.Q > 0) ? m * a.Q + a.Q - 1 : 0);
                    if constexpr (XM == 3) st_pl[j] = a.st[m].pend_len;
                    if (has_part) {
#pragma unroll
                        for (int s2 = 0; s2 < 4; ++s2)
                            pv[s2][j] = *reinterpret_cast<const float4*>(a.part + ((size_t)s2 * a.part_rows + row) * a.ldh + cc);
                    } else {
                        hv[j] = *reinterpret_cast<const float4*>(a.h + (size_t)row * a.ldh + cc);
                    }
                    if constexpr (XM == 3) zv[j] = *reinterpret_cast<const float4*>(a.hz + (size_t)m * a.ldh + cc);
                }
            }
        }
    }

    // Every wave's activation loads go out before any weight load: a CU
    // returns load data in request order, so an activation load queued behind
    // another wave's weight loads (HBM misses) would wait for them.
    __syncthreads();

    // ---- B. weights of this workgroup's 16 columns, all in flight: in the
    //      packed fragment order one 1 KB fragment per wave load ----
    const bf16_t* wp = a.W + ((size_t)blockIdx.x * (K >> 5) + (kb >> 5)) * 512 + lane * 8;
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
    const typename Epi::Pre pre = epi.prefetch(min(em, M - 1), min(en, N - 1), envalid);
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
    } else if constexpr (XM == 4) {
        const int cpr = ks >> 2, items = M * cpr;
        const int S = a.n_splits;
        const int TG = T / GS, sg = __builtin_amdgcn_readfirstlane(wave) / (TG >> 6), it = tid - sg * TG;
        const int m = udiv_small(min(it, items - 1), cpr);
        const int c = kb + (min(it, items - 1) - m * cpr) * 4;
        const int i = m - udiv_small(m, a.Q) * a.Q;
        const int ctx = sti.x, pl = sti.y;
        const int n_active = min(S, udiv_small(ctx + pl + a.split_len - 1, a.split_len));
        // this thread's splits: splits past the context (or a key range fully
        // masked for this row) contribute nothing; their words may be stale
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
            const bool valid = i < pl;
            const float inv = 1.f / Lt;
            const uint2 y = valid ? make_uint2(pack2(sum[0] * inv, sum[1] * inv), pack2(sum[2] * inv, sum[3] * inv))
                                  : make_uint2(0u, 0u);
            *reinterpret_cast<uint2*>(xs + (size_t)m * ldl + (c - kb)) = y;
        }
    } else {
        // row group 0 shares the LayerNorm gain and shift
        f32x4_t* s_gb = red;                      // [2][K/4]
        if (rg == 0) {
            s_gb[cc >> 2] = f32x4_t{gv.x, gv.y, gv.z, gv.w};
            s_gb[K4 + (cc >> 2)] = f32x4_t{bv.x, bv.y, bv.z, bv.w};
        }
        if constexpr (XM == 2) {
            // embedding of each pending token at its position (first layer)
#pragma unroll
            for (int j = 0; j < RPT; ++j) {
                const int m = rg + RG * j;
                if (m < M && rg < RG) {
                    const bool valid = emb_ok[j];
                    const uint2 e = emb_e[j];
                    const uint2 q = emb_p[j];
                    float4 x;
                    x.x = __uint_as_float(e.x << 16) + __uint_as_float(q.x << 16);
                    x.y = __uint_as_float(e.x & 0xFFFF0000u) + __uint_as_float(q.x & 0xFFFF0000u);
                    x.z = __uint_as_float(e.y << 16) + __uint_as_float(q.y << 16);
                    x.w = __uint_as_float(e.y & 0xFFFF0000u) + __uint_as_float(q.y & 0xFFFF0000u);
                    hv[j] = valid ? x : make_float4(0.f, 0.f, 0.f, 0.f);
                }
            }
        } else {
            // the residual row: the sum of the four partials, or h itself
#pragma unroll
            for (int j = 0; j < RPT; ++j) {
                const int m = rg + RG * j;
                if (m < M && rg < RG) {
                    float4 x = hv[j];
                    if (has_part) {
                        x.x = (pv[0][j].x + pv[1][j].x) + (pv[2][j].x + pv[3][j].x);
                        x.y = (pv[0][j].y + pv[1][j].y) + (pv[2][j].y + pv[3][j].y);
                        x.z = (pv[0][j].z + pv[1][j].z) + (pv[2][j].z + pv[3][j].z);
                        x.w = (pv[0][j].w + pv[1][j].w) + (pv[2][j].w + pv[3][j].w);
                    }
                    if constexpr (XM == 3) {
                        const int pl = st_pl[j];
                        if (!(a.Q > 0 && pl == a.Q)) x = zv[j];
                        // a partially filled pending chunk (not produced by the
                        // decode loop, which leaves 0 or Q rows): that row instead
                        if (a.Q > 0 && pl > 0 && pl < a.Q) {
                            const int row = m * a.Q + pl - 1;
                            if (has_part) {
                                float4 p4[4];
#pragma unroll
                                for (int s2 = 0; s2 < 4; ++s2)
                                    p4[s2] = *reinterpret_cast<const float4*>(a.part + ((size_t)s2 * a.part_rows + row) * a.ldh + cc);
                                x.x = (p4[0].x + p4[1].x) + (p4[2].x + p4[3].x);
                                x.y = (p4[0].y + p4[1].y) + (p4[2].y + p4[3].y);
                                x.z = (p4[0].z + p4[1].z) + (p4[2].z + p4[3].z);
                                x.w = (p4[0].w + p4[1].w) + (p4[2].w + p4[3].w);
                            } else {
                                x = *reinterpret_cast<const float4*>(a.h + (size_t)row * a.ldh + cc);
                            }
                        }
                    }
                    hv[j] = x;
                }
            }
        }
        // workgroup 0 writes the completed rows (the next projection's residual input)
        if (a.h_out && blockIdx.x == 0 && blockIdx.y == 0 && rg < RG) {
#pragma unroll
            for (int j = 0; j < RPT; ++j) {
                const int m = rg + RG * j;
                if (m < M) *reinterpret_cast<float4*>(a.h_out + (size_t)m * a.ldh + cc) = hv[j];
            }
        }
        // LayerNorm statistics: one pass (sum, sum of squares) per row; the
        // waves of a row group cover its row exactly once
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
            const int m = rg + RG * j;
            if (m < M && rg < RG) {
                const float4 x = hv[j];
                float s1 = (x.x + x.y) + (x.z + x.w);
                float s2 = (x.x * x.x + x.y * x.y) + (x.z * x.z + x.w * x.w);
                s1 = wave_sum64(s1);
                s2 = wave_sum64(s2);
                if (lane == 0) s_stat[wave][j] = make_float2(s1, s2);
            }
        }
        __syncthreads();
        const float inv_k = 1.f / (float)K;
        const int wpg = K4 >> 6;                  // waves per row group
        const f32x4_t g4 = s_gb[cc >> 2], b4 = s_gb[K4 + (cc >> 2)];
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
            const int m = rg + RG * j;
            if (m >= M || rg >= RG) continue;
            float t1 = 0.f, t2 = 0.f;
            for (int w = rg * wpg; w < (rg + 1) * wpg; ++w) {
                const float2 v = s_stat[w][j];
                t1 += v.x;
                t2 += v.y;
            }
            const float mean = t1 * inv_k;
            const float var = fmaxf(t2 * inv_k - mean * mean, 0.f);
            const float rstd = rsqrtf(var + 1e-5f);
            const float4 x = hv[j];
            const float y0 = (x.x - mean) * rstd * g4[0] + b4[0];
            const float y1 = (x.y - mean) * rstd * g4[1] + b4[1];
            const float y2 = (x.z - mean) * rstd * g4[2] + b4[2];
            const float y3 = (x.w - mean) * rstd * g4[3] + b4[3];
            *reinterpret_cast<uint2*>(xs + (size_t)m * ldl + cc) = make_uint2(pack2(y0, y1), pack2(y2, y3));
        }
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
        epi.store(pre, em, en, v, envalid);
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
static hipError_t gemv_part_rows(hipStream_t st, const GemvArgs& a, const EpiPart& e) {
    const int per_wave = (a.K / 4 / 32 + GV_NW - 1) / GV_NW;
    if (per_wave <= 1) return gemv_go<MR, 0, 1, 1, 1>(st, a, 4, e);
    if (per_wave <= 2) return gemv_go<MR, 0, 2, 1, 1>(st, a, 4, e);
    if (per_wave <= 4) return gemv_go<MR, 0, 4, 1, 1>(st, a, 4, e);
    return gemv_go<MR, 0, 8, 1, 1>(st, a, 4, e);
}

// split-K partial producer over merged attention partials (K = d <= 2048)
template <int MR, int KCH>
static hipError_t gemv_part_merge(hipStream_t st, const GemvArgs& a, const EpiPart& e) {
    constexpr int GS = (16 / (MR * KCH)) > 0 ? 16 / (MR * KCH) : 1;
    if (a.n_splits <= 8) return gemv_go<MR, 4, 1, KCH, 8>(st, a, 4, e);
    if constexpr (8 * GS >= 16) {
        if (a.n_splits <= 16) return gemv_go<MR, 4, 1, KCH, 16>(st, a, 4, e);
    }
    if constexpr (8 * GS >= 32) {
        if (a.n_splits <= 24) return gemv_go<MR, 4, 1, KCH, 24>(st, a, 4, e);
        if (a.n_splits <= 32) return gemv_go<MR, 4, 1, KCH, 32>(st, a, 4, e);
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

hipError_t gemv(hipStream_t st, const GemvArgs& a) {
    if (a.M < 1 || a.M > 16 || a.N < 4 || a.K % 128) return hipErrorInvalidValue;
    if (a.epi == EPI_PARTIAL) {
        if (a.N % 4 || a.K > 4 * 8 * GV_NW * 32) return hipErrorInvalidValue;
        EpiPart e{a.part_out, a.N, a.M, a.h, a.bias};
        if (a.xmode == 4) {
            if (a.K > 2048 || a.K % 256 || a.n_splits < 1 || a.Q < 1 ||
                a.n_splits > gemv_merge_max_splits(a.M, a.K) || a.split_len < 1)
                return hipErrorInvalidValue;
            const bool wide = a.K > 1024;
#define MTP_GEMV_MERGE(MR) return wide ? gemv_part_merge<MR, 2>(st, a, e) : gemv_part_merge<MR, 1>(st, a, e)
            if (a.M <= 1) MTP_GEMV_MERGE(1);
            if (a.M <= 2) MTP_GEMV_MERGE(2);
            if (a.M <= 4) MTP_GEMV_MERGE(4);
            if (a.M <= 8) MTP_GEMV_MERGE(8);
            MTP_GEMV_MERGE(16);
#undef MTP_GEMV_MERGE
        }
        if (a.xmode != 0) return hipErrorInvalidValue;
        if (a.M <= 1) return gemv_part_rows<1>(st, a, e);
        if (a.M <= 2) return gemv_part_rows<2>(st, a, e);
        if (a.M <= 4) return gemv_part_rows<4>(st, a, e);
        if (a.M <= 8) return gemv_part_rows<8>(st, a, e);
        return gemv_part_rows<16>(st, a, e);
    }
    if (a.K > 2048 || a.K % 256 || (a.epi != EPI_LOGITS && a.N % 4)) return hipErrorInvalidValue;
    switch (a.epi) {
    case EPI_QKV: {
        EpiQKVDec e{a.q, a.bias, a.st, a.kv, a.d, a.Q};
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
        EpiLogitsB e{(float*)a.out, a.bias, a.ldo, a.N};
        if (a.xmode == 3) return gemv_ln<3, EpiLogitsB, 8>(st, a, e);
        return hipErrorInvalidValue;
    }
    }
    return hipErrorInvalidValue;
}

}  // namespace mtp
