// The front of a small-batch decode layer in one launch: LayerNorm of the
// residual rows, the QKV projection, and the attention of the pending chunk
// over the keys already in the cache (B * Q <= 8 rows, bf16, d <= 1024).
//
// At batch 1..2 a decode layer is a chain of dependent launches, each a few
// microseconds of launch latency and one global round trip around a weight
// stream of 2-8 MB.  The projection and the attention share a launch here
// because head h's attention needs only head h's query columns: each of the
// G workgroups of head h (one per key split) computes all 64 query columns
// of its head itself (d * 64 bf16 weights, 128 KB at d = 1024; the G
// workgroups of a head are placed on one XCD, so all but the first read them
// from its L2), and no workgroup waits for another.  Keys and values of the
// pending rows come from eight of those workgroups (one 16-column tile
// each), which store them in the paged cache and in a small side buffer; the
// pending rows' attention to their own chunk (keys ctx .. ctx + i for row i)
// is left to the out-projection's merge prologue (gemv xmode 5), after the
// kernel boundary has made those keys visible.
//
// Workgroup (head, split s), 16 waves:
//  A. the LayerNorm input rows (LnRows), each sequence's (ctx_len,
//     pend_len) and the page of this wave's 16-key group of split s in each
//     sequence (lane b: sequence b);
//  B. the head's query weights (wave w: tile w / 4, k fragments w % 4 + 4 i),
//     the key / value tile s (s < 8; wave w: fragments w + 16 i), all in
//     flight at once, then the first sequence's K / V group;
//  D. LayerNorm into the LDS tile;
//  E. MFMA (v_mfma_f32_16x16x32_bf16, A = 16 weight rows, B = 16 rows);
//  F. wave sums: the head's queries (+ bias) into LDS (split 0 also stores
//     them for the out-projection); keys / values (+ bias) into the cache
//     and the side buffer;
//  G. per sequence, the attention arithmetic of attn_dec_kernel on this
//     wave's 16 keys of split s (keys [s SL, (s + 1) SL) of the cached
//     context): S^T = K Q^T / 8, online softmax, O^T = V^T P^T with P kept
//     in registers; the waves merged through LDS; the split's word (max,
//     sum, 64 unnormalised outputs) of each pending row stored for the
//     out-projection (max = -inf for a split past the context).
#include <algorithm>

#include "common.h"
#include "launch.h"
#include "ln_rows.h"
#include "wave.h"

namespace mtp {

namespace {
constexpr int QA_NW = 16;        // waves per workgroup
constexpr int QA_T = 64 * QA_NW;
constexpr int QA_PSTR = 68;      // floats per split word: max, sum, 2 pad, 64 outputs
constexpr int QA_QLD = 68;       // LDS row stride of the query tile (floats)
constexpr int QA_MAXROWS = 8;
constexpr int QA_MAXK = 1024;
constexpr int QA_MING = 8;       // workgroups (key splits) per head: at least the 8 K / V tiles
constexpr int QA_MAXG = 16;
constexpr int QA_MAXSL = 16 * QA_NW;   // keys per split: one 16-key group per wave

typedef short s16x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t qa_pk2(float a, float b) {
    return bf16x2_bits(a, b);
}

int split_len_for(int64_t max_ctx, int g) {
    const int64_t sl = (std::max<int64_t>(max_ctx, 1) + g - 1) / g;
    return (int)((sl + 15) / 16 * 16);
}
}  // namespace

template <int MR, int XM>
__global__ __launch_bounds__(QA_T) void qkv_attn_kernel(GemvArgs a) {
    using Rows = LnRows<MR, XM, 1, QA_T, (MR > 4 ? 1 : 0)>;          // M > 4 iff MR > 4
    // the first sequence's K / V group is loaded with the weights; at 8 rows
    // the LayerNorm registers leave no room for it (it is loaded in G)
    constexpr bool PRE = MR <= 4;
    extern __shared__ __attribute__((aligned(16))) unsigned char qa_lds[];
    bf16_t* xs = reinterpret_cast<bf16_t*>(qa_lds);   // [16][K + 8] LayerNorm rows (D, E)
    float* s_o = reinterpret_cast<float*>(qa_lds);     // [waves][64][17] attention outputs (G), after E
    __shared__ f32x4_t red[2 * QA_NW * 64];             // LayerNorm gain / shift (D); wave sums (E, F)
    __shared__ float2 s_stat[QA_NW][Rows::RPT];
    __shared__ __attribute__((aligned(16))) float s_q[16 * QA_QLD];   // the head's query rows (fp32)
    __shared__ float s_m[QA_NW][16], s_l[QA_NW][16];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, g = lane >> 4;
    const int K = a.K, M = a.M, Q = a.Q, d = a.d;
    const int H = K >> 6, G = a.n_splits, SL = a.split_len;
    const int B = M / Q;
    // Workgroups are dealt to the 8 XCDs round robin: the G workgroups of a
    // head go to one XCD, whose L2 then serves its query weights G times.
    const int id = blockIdx.x;
    int head, s;
    if ((H & 7) == 0) {
        const int slot = id >> 3, hi = slot / G;
        head = (id & 7) + 8 * hi;
        s = slot - hi * G;
    } else {
        head = id / G;
        s = id - head * G;
    }

    // ---- A. activation-side loads, before any weight load (a CU returns
    //      load data in request order) ----
    float4 ln_hv[Rows::RPT], ln_pv[Rows::NPV][Rows::RES ? Rows::RPT : 1], ln_zv[1];
    uint2 ln_ph[Rows::NPH][Rows::RES ? Rows::RPT : 1];
    uint2 ln_ee[XM == 2 ? Rows::RPT : 1], ln_ep[XM == 2 ? Rows::RPT : 1];
    bool ln_eok[XM == 2 ? Rows::RPT : 1];
    int ln_pl[1];
    Rows lr{ln_hv, ln_pv, ln_ph, ln_zv, ln_ee, ln_ep, ln_eok, ln_pl};
    lr.init(a, tid, wave);
    lr.load(a);
    // lane b: sequence b's (ctx_len, pend_len) and the page of this wave's
    // key group of split s (clamped to the block table, whose unused
    // entries name page 0, so every load stays in the pool)
    const int bl = min(lane, B - 1);
    const int2 stv = *reinterpret_cast<const int2*>(&a.st[bl]);
    const int maxp = a.kv.max_pages_per_seq;
    const int kb = s * SL;
    const int pg = a.kv.block_table[(size_t)bl * maxp + min((kb >> 4) + wave, maxp - 1)];
    __syncthreads();

    // ---- B. weights: the head's 4 query tiles and the K / V tile s ----
    const int KF = K >> 5;                 // 32-wide k fragments per column tile
    const int nfq = K >> 7;                // query fragments per wave (4 waves per tile)
    uint4 wq[QA_MAXK / 128];
    {
        const bf16_t* wp = a.W + (size_t)(4 * head + (wave >> 2)) * KF * 512 + lane * 8;
#pragma unroll
        for (int i = 0; i < QA_MAXK / 128; ++i) {
            const int f = min((wave & 3) + 4 * i, KF - 1);
            wq[i] = *reinterpret_cast<const uint4*>(wp + (size_t)f * 512);
        }
    }
    const bool has_kv = s < 8;             // uniform
    const int kvc = s < 4 ? d + 64 * head + 16 * s : 2 * d + 64 * head + 16 * (s - 4);   // first column
    uint4 wk[QA_MAXK / 512];
    if (has_kv) {
        const bf16_t* wp = a.W + (size_t)(kvc >> 4) * KF * 512 + lane * 8;
#pragma unroll
        for (int i = 0; i < QA_MAXK / 512; ++i) {
            const int f = min(wave + QA_NW * i, KF - 1);
            wk[i] = *reinterpret_cast<const uint4*>(wp + (size_t)f * 512);
        }
    }
    // epilogue operands: the bias of the wave's reduced tile
    float4 bq = make_float4(0.f, 0.f, 0.f, 0.f), bk = bq;
    if (wave < 4) bq = *reinterpret_cast<const float4*>(a.bias + 64 * head + 16 * wave + 4 * g);
    if (wave == 4 && has_kv) bk = *reinterpret_cast<const float4*>(a.bias + kvc + 4 * g);
    // the first sequence's K / V group of this wave (its page arrived with A)
    const bf16_t* pool = reinterpret_cast<const bf16_t*>(a.kv.pool);
    const bool wgrp = 16 * wave < SL;      // the wave owns a 16-key group of the split (uniform)
    uint4 kf0[2];
    uint2 vf0[4];
    if (PRE && wgrp) {
        const int page = __builtin_amdgcn_readlane(pg, 0);
        const bf16_t* kp = pool + kv_page_block(a.kv, page, 0, head) + r * MTP_HEAD_DIM + g * 8;
        kf0[0] = *reinterpret_cast<const uint4*>(kp);
        kf0[1] = *reinterpret_cast<const uint4*>(kp + 32);
        const bf16_t* vp = pool + kv_page_block(a.kv, page, 1, head) + 4 * g;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) vf0[dt] = *reinterpret_cast<const uint2*>(vp + (16 * dt + r) * 16);
    }
    // every load above is issued before the prologue arithmetic below
    __builtin_amdgcn_sched_barrier(0);

    // ---- D. LayerNorm rows into LDS (workgroup 0 writes the completed
    //      residual rows for the out-projection) ----
    const int ldl = K + 8;
    lr.build(a, id == 0, xs, ldl, red, s_stat, wave, lane);
    __syncthreads();

    // ---- E. MFMA ----
    f32x4_t aq = f32x4_t{0.f, 0.f, 0.f, 0.f}, ak = aq;
#pragma unroll
    for (int i = 0; i < QA_MAXK / 128; ++i)
        if (i < nfq) {
            const int f = (wave & 3) + 4 * i;
            const bf16x8_t xf = *reinterpret_cast<const bf16x8_t*>(xs + (size_t)r * ldl + f * 32 + g * 8);
            aq = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wq[i]), xf, aq, 0, 0, 0);
        }
    if (has_kv) {
#pragma unroll
        for (int i = 0; i < QA_MAXK / 512; ++i) {
            const int f = wave + QA_NW * i;
            if (f < KF) {
                const bf16x8_t xf = *reinterpret_cast<const bf16x8_t*>(xs + (size_t)r * ldl + f * 32 + g * 8);
                ak = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wk[i]), xf, ak, 0, 0, 0);
            }
        }
    }
    red[wave * 64 + lane] = aq;
    red[(QA_NW + wave) * 64 + lane] = ak;
    __syncthreads();

    // ---- F. wave sums and their epilogues; lane (r, g) holds row r,
    //      columns 4 g .. 4 g + 3 of the tile ----
    if (wave < 4) {
        f32x4_t sum = red[(4 * wave) * 64 + lane];
#pragma unroll
        for (int j = 1; j < 4; ++j) sum += red[(4 * wave + j) * 64 + lane];
        const float4 v = make_float4(sum[0] + bq.x, sum[1] + bq.y, sum[2] + bq.z, sum[3] + bq.w);
        const int col = 16 * wave + 4 * g;
        *reinterpret_cast<float4*>(s_q + r * QA_QLD + col) = v;
        if (s == 0 && r < M) *reinterpret_cast<float4*>(a.q + (size_t)r * d + 64 * head + col) = v;
    } else if (wave == 4 && has_kv) {
        f32x4_t sum = red[QA_NW * 64 + lane];
#pragma unroll
        for (int w = 1; w < QA_NW; ++w) sum += red[(QA_NW + w) * 64 + lane];
        const float r0 = sum[0] + bk.x, r1 = sum[1] + bk.y, r2 = sum[2] + bk.z, r3 = sum[3] + bk.w;
        const int seq = udiv_small(min(r, M - 1), Q), i = min(r, M - 1) - seq * Q;
        const int ctx = __shfl(stv.x, seq), pl = __shfl(stv.y, seq);
        if (r < M && i < pl) {
            const int pos = ctx + i;
            const bool is_k = kvc < 2 * d;
            const int c = (is_k ? kvc - d : kvc - 2 * d) + 4 * g;   // column within the d keys (values)
            bf16_t* cache = reinterpret_cast<bf16_t*>(a.kv.pool);
            const uint2 packed = make_uint2(qa_pk2(r0, r1), qa_pk2(r2, r3));
            if (is_k) {
                *reinterpret_cast<uint2*>(cache + a.kv.offset(seq, pos, 0, c >> 6) + (c & 63)) = packed;
            } else {
                bf16_t* vt = cache + a.kv.vt_offset(seq, pos, c >> 6) + (size_t)(c & 63) * a.kv.page_size;
                const size_t P = a.kv.page_size;
                vt[0] = f32_to_bf16(r0);
                vt[P] = f32_to_bf16(r1);
                vt[2 * P] = f32_to_bf16(r2);
                vt[3 * P] = f32_to_bf16(r3);
            }
            *reinterpret_cast<uint2*>(a.kvnew + ((size_t)(is_k ? 0 : M) + r) * d + c) = packed;
        }
    }
    __syncthreads();

    // ---- G. attention of each sequence's pending rows over split s of its
    //      cached keys ----
    const int nwa = min(QA_NW, SL >> 4);   // waves that own a key group
    const int sstride = a.qt * QA_PSTR;
    for (int b = 0; b < B; ++b) {
        const int ctx = __builtin_amdgcn_readlane(stv.x, b), pl = __builtin_amdgcn_readlane(stv.y, b);
        const int ke = min(kb + SL, ctx);
        const int wk0 = kb + 16 * wave;
        float m_run = -INFINITY, l_run = 0.f;
        f32x4_t acc[4];
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) acc[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        if (wgrp && wk0 < ke && pl > 0) {       // uniform
            uint4 k0, k1;
            uint2 v[4];
            if (PRE && b == 0) {
                k0 = kf0[0];
                k1 = kf0[1];
#pragma unroll
                for (int dt = 0; dt < 4; ++dt) v[dt] = vf0[dt];
            } else {
                const int page = __builtin_amdgcn_readlane(pg, b);
                const bf16_t* kp = pool + kv_page_block(a.kv, page, 0, head) + r * MTP_HEAD_DIM + g * 8;
                k0 = *reinterpret_cast<const uint4*>(kp);
                k1 = *reinterpret_cast<const uint4*>(kp + 32);
                const bf16_t* vp = pool + kv_page_block(a.kv, page, 1, head) + 4 * g;
#pragma unroll
                for (int dt = 0; dt < 4; ++dt) v[dt] = *reinterpret_cast<const uint2*>(vp + (16 * dt + r) * 16);
            }
            // queries of sequence b (rows b Q + r), scaled by 1/8, as the MFMA B operand
            const float* qp = s_q + (b * Q + min(r, Q - 1)) * QA_QLD + g * 8;
            bf16x8_t qf[2];
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                const float4 x0 = *reinterpret_cast<const float4*>(qp + 32 * h2);
                const float4 x1 = *reinterpret_cast<const float4*>(qp + 32 * h2 + 4);
                qf[h2] = __builtin_bit_cast(bf16x8_t, make_uint4(qa_pk2(x0.x * 0.125f, x0.y * 0.125f),
                                                                 qa_pk2(x0.z * 0.125f, x0.w * 0.125f),
                                                                 qa_pk2(x1.x * 0.125f, x1.y * 0.125f),
                                                                 qa_pk2(x1.z * 0.125f, x1.w * 0.125f)));
            }
            f32x4_t sc4 = f32x4_t{0.f, 0.f, 0.f, 0.f};
            sc4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, k0), qf[0], sc4, 0, 0, 0);
            sc4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, k1), qf[1], sc4, 0, 0, 0);
            // S^T[key 4 g + e][query r]: every cached key precedes the chunk
            float sc[4];
            float mx = -INFINITY;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const bool ok = (wk0 + 4 * g + e < ke) && (r < pl);
                sc[e] = ok ? sc4[e] : -INFINITY;
                mx = fmaxf(mx, sc[e]);
            }
            mx = xor16_max(mx);
            mx = xor32_max(mx);
            m_run = mx;
            float pe[4], sum = 0.f;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                pe[e] = (sc[e] == -INFINITY) ? 0.f : __expf(sc[e] - mx);
                sum += pe[e];
            }
            sum = xor16_sum(sum);
            sum = xor32_sum(sum);
            l_run = sum;
            const s16x4_t pf = __builtin_bit_cast(s16x4_t, make_uint2(qa_pk2(pe[0], pe[1]), qa_pk2(pe[2], pe[3])));
            // V^T entries of keys past the context may hold anything: zero them
            const int nvalid = ke - (wk0 + 4 * g);
#pragma unroll
            for (int dt = 0; dt < 4; ++dt) {
                uint2 vv = v[dt];
                if (nvalid < 4) {
                    uint32_t w0 = vv.x, w1 = vv.y;
                    if (nvalid <= 0) w0 = 0u;
                    else if (nvalid == 1) w0 &= 0x0000FFFFu;
                    if (nvalid <= 2) w1 = 0u;
                    else w1 &= 0x0000FFFFu;
                    vv = make_uint2(w0, w1);
                }
                acc[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4_t, vv), pf, acc[dt], 0, 0, 0);
            }
        }
        // merge the waves' states through LDS
        if (wave < nwa && g == 0) s_m[wave][r] = m_run;
        __syncthreads();
        if (wave < nwa) {
            float mw = -INFINITY;
            for (int w = 0; w < nwa; ++w) mw = fmaxf(mw, s_m[w][r]);
            const float wsc = (m_run == -INFINITY) ? 0.f : __expf(m_run - mw);
#pragma unroll
            for (int dt = 0; dt < 4; ++dt)
#pragma unroll
                for (int e = 0; e < 4; ++e) s_o[(wave * 64 + 16 * dt + 4 * g + e) * 17 + r] = acc[dt][e] * wsc;
            if (g == 0) s_l[wave][r] = l_run * wsc;
        }
        __syncthreads();
        {
            const int dim = tid >> 4, q = tid & 15;   // 1024 threads: one (dim, query) pair each
            if (q < pl) {
                float o = 0.f, L = 0.f, mq = -INFINITY;
                for (int w = 0; w < nwa; ++w) {
                    o += s_o[(w * 64 + dim) * 17 + q];
                    L += s_l[w][q];
                    mq = fmaxf(mq, s_m[w][q]);
                }
                float* e = a.apart + ((size_t)(b * H + head) * G + s) * sstride + q * QA_PSTR;
                e[4 + dim] = o;
                if (dim == 0) {
                    e[0] = mq;
                    e[1] = L;
                }
            }
        }
        __syncthreads();                        // s_o, s_m, s_l are reused by the next sequence
    }
}

template <int MR, int XM>
static hipError_t qa_go(hipStream_t st, const GemvArgs& a) {
    const int nwa = std::min(QA_NW, a.split_len >> 4);
    const size_t lds = std::max((size_t)16 * (a.K + 8) * 2, (size_t)nwa * 64 * 17 * sizeof(float));
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(&qkv_attn_kernel<MR, XM>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)std::max((size_t)16 * (QA_MAXK + 8) * 2,
                                                           (size_t)QA_NW * 64 * 17 * sizeof(float)));
        if (err != hipSuccess) return err;
        attr_set = true;
    }
    hipLaunchKernelGGL((qkv_attn_kernel<MR, XM>), dim3((a.K >> 6) * a.n_splits), dim3(QA_T), lds, st, a);
    return hipGetLastError();
}

bool qkv_attn_ok(int rows, int d, int n_heads, int64_t max_ctx, int n_splits) {
    return rows >= 1 && rows <= QA_MAXROWS && d >= 256 && d <= QA_MAXK && d % 256 == 0 && n_heads * 64 == d &&
           n_splits >= QA_MING && n_splits <= QA_MAXG && split_len_for(max_ctx, n_splits) <= QA_MAXSL;
}

hipError_t qkv_attn(hipStream_t st, const GemvArgs& a) {
    if (a.M < 1 || a.M > QA_MAXROWS || a.Q < 1 || a.M % a.Q || a.qt < a.Q || a.qt > MTP_ATTN_QT) return hipErrorInvalidValue;
    if (a.K != a.d || a.K < 256 || a.K > QA_MAXK || a.K % 256 || a.N != 3 * a.d) return hipErrorInvalidValue;
    if (a.n_splits < QA_MING || a.n_splits > QA_MAXG || a.split_len < 16 || a.split_len > QA_MAXSL || a.split_len % 16)
        return hipErrorInvalidValue;
    if (!a.apart || !a.kvnew || !a.q || !a.st || a.kv.page_size != 16) return hipErrorInvalidValue;
    if (a.xmode == 1 && a.part_on && partials_bf16(a.part_rows) != partials_bf16(a.M)) return hipErrorInvalidValue;
#define MTP_QA(MR)                                                       \
    do {                                                                 \
        if (a.xmode == 1) return qa_go<MR, 1>(st, a);                    \
        if (a.xmode == 2) return qa_go<MR, 2>(st, a);                    \
        return hipErrorInvalidValue;                                     \
    } while (0)
    if (a.M <= 1) MTP_QA(1);
    if (a.M <= 2) MTP_QA(2);
    if (a.M <= 4) MTP_QA(4);
    MTP_QA(8);
#undef MTP_QA
}

// Split plan of qkv_attn: keys per split for a context of max_ctx keys over
// g workgroups per head.
int qkv_attn_split_len(int64_t max_ctx, int g) { return split_len_for(max_ctx, g); }

}  // namespace mtp
