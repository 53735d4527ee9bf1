// Small-M (decode) projections, bf16 MFMA, with the row-wise work fused in.
//
// At batch 1..8 a decode step is a chain of weight streams of 2-12 MB each;
// every dependent global round trip costs about a microsecond, so this
// kernel is built to have as few of them as possible on its critical path:
//
//  * every W fragment of the workgroup's 16 output columns (its K slice) is
//    loaded into registers at kernel start, before anything else; W rows are
//    read 64 contiguous bytes per row per load, one full 128-byte line per
//    two consecutive fragments;
//  * epilogue operands (bias, per-row KV-cache addresses) are fetched at
//    kernel start too;
//  * the activation rows are produced in a prologue while the weights are in
//    flight: LayerNorm of the fp32 residual rows (LN1, LN2, final LN), or the
//    token + position embedding followed by LN1 for the first layer; the
//    bf16 result goes to LDS and feeds the MFMA B operand;
//  * or, for the out-projection, the prologue merges the decode-attention
//    split partials (max, sum, unnormalised output) into the bf16 rows;
//  * each workgroup owns whole output columns (no split-K), so the residual
//    epilogue adds into h directly and no cross-workgroup reduction, atomic
//    or device-scope fence is needed: kernel boundaries are the only sync.
//
// MFMA: v_mfma_f32_16x16x32_bf16 with A = 16 weight rows (output columns n)
// and B = 16 activation rows (m); lane (r = l % 16, g = l / 16) supplies
// row r and k = 8g..8g+7 of each 32-wide k step, the same k for A and B.
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
        const SeqState& s = st[m / Q];
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
        const int seq = m / Q, i = m - seq * Q;
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

// h[m][n] += v + bias  (the residual add of O-proj and FFN2).
struct EpiResid {
    float* h;
    const float* bias;
    int ldh;
    struct Pre { float b[4]; float4 h0; };
    __device__ __forceinline__ Pre prefetch(int m, int n, int) const {
        Pre p;
#pragma unroll
        for (int i = 0; i < 4; ++i) p.b[i] = bias[n + i];
        p.h0 = *reinterpret_cast<const float4*>(h + (size_t)m * ldh + n);
        return p;
    }
    __device__ __forceinline__ void store(const Pre& p, int m, int n, const float (&v)[4], int) const {
        float4 o = p.h0;
        o.x += v[0] + p.b[0];
        o.y += v[1] + p.b[1];
        o.z += v[2] + p.b[2];
        o.w += v[3] + p.b[3];
        *reinterpret_cast<float4*>(h + (size_t)m * ldh + n) = o;
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
        for (int i = 0; i < nvalid; ++i) o[i] = v[i] + p.b[i];
    }
};

}  // namespace

// ------------------------------------------------------------------- kernel
// XM: 0 = bf16 rows from global, 1 = LN(h rows), 2 = embed + LN (decode rows),
//     3 = final LN of each sequence's last pending row (heads),
//     4 = merge of decode-attention split partials (no LN).
template <int MT, int XM, int MAXF, class Epi>
__global__ __launch_bounds__(256) void gemv_kernel(GemvArgs a, Epi epi) {
    extern __shared__ __attribute__((aligned(16))) bf16_t xs[];   // [MT*16][K + 8] (XM != 0)
    __shared__ f32x4_t red[4][MT][64];
    constexpr int ROWS = MT * 16;
    constexpr int MAXS = 8;                       // attention splits merged in the prologue
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int n0 = blockIdx.x * 16;
    const int K = a.K, M = a.M, N = a.N;
    const int nfrag = K >> 5;
    const int nf = (nfrag - wave + 3) >> 2;       // fragments f = wave + 4 i, i < nf
    const int ldl = K + 8;                        // LDS row stride (bf16)
    const int m0 = wave;                          // first activation row of this wave

    // 1. Activation-side loads go out first.  vmcnt retires in order, so
    //    anything issued after the weight stream could only be consumed once
    //    all weights have landed; issued before, the prologue overlaps the
    //    stream.  Every load below is unconditional from a clamped, valid
    //    address: a predicated load becomes a branch plus a full vmcnt wait at
    //    the join, which would serialise the round trips.  Rows, columns and
    //    fragments outside the problem produce values that are never stored
    //    or never enter a reduction.
    const int mc = min(m0, M - 1);
    uint4 xv[XM == 0 ? MAXF : 1][MT];
    float4 gg[8], bb[8], x0[8], x1[8];
    int st_pl = 0, st_ctx = 0;
    if constexpr (XM == 0) {
#pragma unroll
        for (int i = 0; i < MAXF; ++i)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const int m = min(r + 16 * mt, M - 1);
                const int f = min(wave + 4 * i, nfrag - 1);
                xv[i][mt] = *reinterpret_cast<const uint4*>(a.x + (size_t)m * a.ldx + f * 32 + g * 8);
            }
    } else if constexpr (XM == 4) {
        const SeqState& s = a.st[mc / a.Q];
        st_pl = s.pend_len;
        st_ctx = s.ctx_len;
    } else {
        const float* row0 = a.h + (size_t)mc * a.ldh;
        if constexpr (XM == 3) row0 = a.h + (size_t)(a.Q > 0 ? mc * a.Q + a.Q - 1 : 0) * a.ldh;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int c = min(lane * 4 + 256 * j, K - 4);
            gg[j] = *reinterpret_cast<const float4*>(a.g + c);
            bb[j] = *reinterpret_cast<const float4*>(a.beta + c);
            if constexpr (XM == 1 || XM == 3) x0[j] = *reinterpret_cast<const float4*>(row0 + c);
            if constexpr (XM == 3) x1[j] = *reinterpret_cast<const float4*>(a.hz + (size_t)mc * a.ldh + c);
        }
        if constexpr (XM == 3) st_pl = a.st[mc].pend_len;
    }

    // 2. weights of this workgroup's 16 columns, all in flight at once
    const int nrow = min(n0 + r, N - 1);
    const bf16_t* wp = a.W + (size_t)nrow * K + g * 8;
    uint4 wv[MAXF];
#pragma unroll
    for (int i = 0; i < MAXF; ++i) {
        const int f = min(wave + 4 * i, nfrag - 1);
        wv[i] = *reinterpret_cast<const uint4*>(wp + f * 32);
    }
    // 3. epilogue operands
    const int em = r + 16 * (wave < MT ? wave : 0);
    const int en = n0 + 4 * g;
    const int envalid = min(4, N - en);
    const typename Epi::Pre pre = epi.prefetch(min(em, M - 1), min(en, N - 1), envalid);

    // 4. activation rows -> bf16 in LDS
    if constexpr (XM == 4) {
        for (int m = wave; m < ROWS; m += 4) {
            bf16_t* dst = xs + (size_t)m * ldl;
            int pl = st_pl, ctx = st_ctx;
            if (m != m0 && m < M) {
                const SeqState& s = a.st[m / a.Q];
                pl = s.pend_len;
                ctx = s.ctx_len;
            }
            const int seq = m / a.Q, i = m - seq * a.Q;
            if (m >= M || i >= pl) {
                for (int c = lane * 4; c < K; c += 256) *reinterpret_cast<uint2*>(dst + c) = make_uint2(0, 0);
                continue;
            }
            const int H = K >> 6;
            const int n_active = min(a.n_splits, (ctx + pl + a.split_len - 1) / a.split_len);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int c = lane * 4 + 256 * j;
                if (c >= K) continue;
                const int head = c >> 6, dim = c & 63;
                const float* e0 = a.apart + ((size_t)(seq * H + head) * a.n_splits) * (a.qt * 68) + i * 68;
                float ms[MAXS], ls[MAXS];
                float4 os[MAXS];
#pragma unroll
                for (int sp = 0; sp < MAXS; ++sp) {
                    const float* e = e0 + (size_t)min(sp, n_active - 1) * a.qt * 68;
                    ms[sp] = e[0];
                    ls[sp] = e[1];
                    os[sp] = *reinterpret_cast<const float4*>(e + 4 + dim);
                }
#pragma unroll
                for (int sp = 0; sp < MAXS; ++sp)
                    if (sp >= n_active) ms[sp] = -INFINITY;
                float Mx = -INFINITY;
#pragma unroll
                for (int sp = 0; sp < MAXS; ++sp) Mx = fmaxf(Mx, ms[sp]);
                float L = 0.f;
                float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
                for (int sp = 0; sp < MAXS; ++sp) {
                    const float w = (ms[sp] == -INFINITY) ? 0.f : __expf(ms[sp] - Mx);
                    L = fmaf(w, ls[sp], L);
                    o.x = fmaf(w, os[sp].x, o.x);
                    o.y = fmaf(w, os[sp].y, o.y);
                    o.z = fmaf(w, os[sp].z, o.z);
                    o.w = fmaf(w, os[sp].w, o.w);
                }
                const float inv = 1.f / L;
                *reinterpret_cast<uint2*>(dst + c) = make_uint2(pack2(o.x * inv, o.y * inv), pack2(o.z * inv, o.w * inv));
            }
        }
        __syncthreads();
    } else if constexpr (XM != 0) {
        for (int m = wave; m < ROWS; m += 4) {
            bf16_t* dst = xs + (size_t)m * ldl;
            if (m >= M) {
                for (int c = lane * 4; c < K; c += 256) *reinterpret_cast<uint2*>(dst + c) = make_uint2(0, 0);
                continue;
            }
            float4 x[8];
            if (m == m0 && XM != 2) {
                if constexpr (XM == 3) {
                    const bool last_row = a.Q > 0 && st_pl == a.Q;
                    const bool other = a.Q > 0 && st_pl > 0 && st_pl != a.Q;
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        x[j] = last_row ? x0[j] : x1[j];
                        if (other && lane * 4 + 256 * j < K)
                            x[j] = *reinterpret_cast<const float4*>(a.h + (size_t)(m * a.Q + st_pl - 1) * a.ldh + lane * 4 + 256 * j);
                    }
                } else {
#pragma unroll
                    for (int j = 0; j < 8; ++j) x[j] = x0[j];
                }
            } else if constexpr (XM == 2) {
                const int seq = m / a.Q, i = m - seq * a.Q;
                const SeqState& s = a.st[seq];
                const bool valid = i < s.pend_len;
                const bf16_t* erow = a.emb + (size_t)(valid ? s.pend_ids[i] : 0) * K;
                const bf16_t* prow = a.pos + (size_t)(valid ? s.ctx_len + i : 0) * K;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int c = lane * 4 + 256 * j;
                    x[j] = make_float4(0.f, 0.f, 0.f, 0.f);
                    if (c < K && valid) {
                        const uint2 e = *reinterpret_cast<const uint2*>(erow + c);
                        const uint2 q = *reinterpret_cast<const uint2*>(prow + c);
                        x[j].x = __uint_as_float(e.x << 16) + __uint_as_float(q.x << 16);
                        x[j].y = __uint_as_float(e.x & 0xFFFF0000u) + __uint_as_float(q.x & 0xFFFF0000u);
                        x[j].z = __uint_as_float(e.y << 16) + __uint_as_float(q.y << 16);
                        x[j].w = __uint_as_float(e.y & 0xFFFF0000u) + __uint_as_float(q.y & 0xFFFF0000u);
                    }
                }
                if (blockIdx.x == 0) {
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const int c = lane * 4 + 256 * j;
                        if (c < K) *reinterpret_cast<float4*>(a.h_out + (size_t)m * a.ldh + c) = x[j];
                    }
                }
            } else {
                const float* src;
                if constexpr (XM == 3) {
                    const int pl = a.st[m].pend_len;
                    src = (a.Q > 0 && pl > 0) ? a.h + (size_t)(m * a.Q + pl - 1) * a.ldh : a.hz + (size_t)m * a.ldh;
                } else {
                    src = a.h + (size_t)m * a.ldh;
                }
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int c = lane * 4 + 256 * j;
                    x[j] = (c < K) ? *reinterpret_cast<const float4*>(src + c) : make_float4(0.f, 0.f, 0.f, 0.f);
                }
            }
            float s = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (lane * 4 + 256 * j < K) s += (x[j].x + x[j].y) + (x[j].z + x[j].w);
            const float mean = wsum(s) / (float)K;
            float v = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (lane * 4 + 256 * j < K) {
                    const float dx = x[j].x - mean, dy = x[j].y - mean, dz = x[j].z - mean, dw = x[j].w - mean;
                    v += (dx * dx + dy * dy) + (dz * dz + dw * dw);
                }
            const float rstd = rsqrtf(wsum(v) / (float)K + 1e-5f);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int c = lane * 4 + 256 * j;
                if (c < K) {
                    const float y0 = (x[j].x - mean) * rstd * gg[j].x + bb[j].x;
                    const float y1 = (x[j].y - mean) * rstd * gg[j].y + bb[j].y;
                    const float y2 = (x[j].z - mean) * rstd * gg[j].z + bb[j].z;
                    const float y3 = (x[j].w - mean) * rstd * gg[j].w + bb[j].w;
                    *reinterpret_cast<uint2*>(dst + c) = make_uint2(pack2(y0, y1), pack2(y2, y3));
                }
            }
        }
        __syncthreads();
    }

    // 5. MFMA over this wave's fragments
    f32x4_t acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < MAXF; ++i)
        if (i < nf) {
            const int f = wave + 4 * i;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                bf16x8_t xf;
                if constexpr (XM == 0) xf = __builtin_bit_cast(bf16x8_t, xv[i][mt]);
                else xf = *reinterpret_cast<const bf16x8_t*>(xs + (size_t)(r + 16 * mt) * ldl + f * 32 + g * 8);
                acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wv[i]), xf, acc[mt], 0, 0, 0);
            }
        }

    // 6. sum the four waves' K quarters, epilogue
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) red[wave][mt][lane] = acc[mt];
    __syncthreads();
    if (wave < MT && em < M && en < N) {
        const f32x4_t sum = (red[0][wave][lane] + red[1][wave][lane]) + (red[2][wave][lane] + red[3][wave][lane]);
        const float v[4] = {sum[0], sum[1], sum[2], sum[3]};
        epi.store(pre, em, en, v, envalid);
    }
}

// --------------------------------------------------------------- launching
template <int MT, int XM, int MAXF, class Epi>
static hipError_t gemv_go(hipStream_t st, const GemvArgs& a, const Epi& e) {
    dim3 grid((a.N + 15) / 16);
    size_t lds = XM ? (size_t)MT * 16 * (a.K + 8) * 2 : 0;
    static bool attr_set = false;
    if (lds > 48 * 1024 && !attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemv_kernel<MT, XM, MAXF, Epi>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 140 * 1024);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    hipLaunchKernelGGL((gemv_kernel<MT, XM, MAXF, Epi>), grid, dim3(256), lds, st, a, e);
    return hipGetLastError();
}

template <int XM, class Epi>
static hipError_t gemv_pick(hipStream_t st, const GemvArgs& a, const Epi& e) {
    const int per_wave = (a.K / 32 + 3) / 4;
    if (a.M <= 16) {
        if (per_wave <= 8) return gemv_go<1, XM, 8>(st, a, e);
        if (per_wave <= 16) return gemv_go<1, XM, 16>(st, a, e);
        if (per_wave <= 32) return gemv_go<1, XM, 32>(st, a, e);
        if (per_wave <= 48) return gemv_go<1, XM, 48>(st, a, e);
    } else if (a.M <= 32) {
        if (per_wave <= 8) return gemv_go<2, XM, 8>(st, a, e);
        if (per_wave <= 16) return gemv_go<2, XM, 16>(st, a, e);
        if (per_wave <= 32) return gemv_go<2, XM, 32>(st, a, e);
        if (per_wave <= 48) return gemv_go<2, XM, 48>(st, a, e);
    }
    return hipErrorInvalidValue;
}

hipError_t gemv(hipStream_t st, const GemvArgs& a) {
    if (a.M < 1 || a.M > 32 || a.K % 32 || a.K > 48 * 4 * 32 || (a.xmode != 0 && a.K > 2048)) return hipErrorInvalidValue;
    if (a.xmode == 4 && (a.n_splits > 8 || a.qt > MTP_ATTN_QT)) return hipErrorInvalidValue;
    switch (a.epi) {
    case EPI_QKV: {
        EpiQKVDec e{a.q, a.bias, a.st, a.kv, a.d, a.Q};
        if (a.xmode == 2) return gemv_pick<2>(st, a, e);
        return gemv_pick<1>(st, a, e);
    }
    case EPI_GELU: {
        EpiGeluB e{(bf16_t*)a.out, a.bias, a.ldo};
        return gemv_pick<1>(st, a, e);
    }
    case EPI_RESID: {
        EpiResid e{a.h_res, a.bias, a.ldo};
        if (a.xmode == 4) return gemv_pick<4>(st, a, e);
        return gemv_pick<0>(st, a, e);
    }
    case EPI_LOGITS: {
        EpiLogitsB e{(float*)a.out, a.bias, a.ldo, a.N};
        return gemv_pick<3>(st, a, e);
    }
    }
    return hipErrorInvalidValue;
}

}  // namespace mtp
