// LayerNorm prologue of the small-M (<= 16 rows) decode kernels: the rows of
// a LayerNorm input, normalised and rounded to bf16 into an LDS tile.
//
// Row sources (XM): 1 = the residual rows, completed here as the sum of the
// producer's four split-K partials (the first of which, in float32, carries
// the residual input and the bias; the others are bfloat16) or taken from h; 2 = token embedding + learned position
// of each pending token (first layer); 3 = the final LayerNorm input of each
// sequence's last pending row (heads).
//
// Thread t owns the float4 column chunk t % (K/4) of rows t / (K/4),
// t / (K/4) + RG, ... (RG = T / (K/4) row groups), so the gain and shift are
// loaded once per thread (by row group 0, shared through LDS) and a row's
// statistics are a reduction over the K/4/64 waves of its row group.
//
// load() issues every load (phase A of the kernels: before any weight load,
// since a CU returns load data in request order); build() runs after the
// weight loads are in flight and leaves the tile in LDS, before the caller's
// barrier.  The register arrays are locals of the calling kernel that the
// struct refers to: each is then a separate homogeneous array, which the
// compiler keeps in registers (as members of one mixed struct they would be
// placed in scratch memory).
#pragma once

#include "common.h"
#include "launch.h"
#include "wave.h"

namespace mtp {

// PF: the form of the producer's split-K partials (store_partial4): 0 the
// float32 form, 1 the bfloat16 one.
template <int MR, int XM, int KCH, int T, int PF>
struct LnRows {
    static constexpr bool RES = XM == 1 || XM == 3;                    // residual completed here
    static constexpr int RPT = (MR * KCH * 256 + T - 1) / T;           // rows per thread
    static constexpr bool BFP = PF == 1;
    static constexpr int NPV = RES ? (BFP ? 1 : 4) : 1;                // float32 ranges held
    static constexpr int NPH = RES && BFP ? 3 : 1;                     // bfloat16 ranges held
    float4 (&hv)[RPT];                                                  // residual / embedding rows
    float4 (&pv)[NPV][RES ? RPT : 1];                                   // the producer's partials: float32 ranges
    uint2 (&ph)[NPH][RES ? RPT : 1];                                    //   and bfloat16 ranges 1..3 (raw bits)
    float4 (&zv)[XM == 3 ? RPT : 1];                                    // prefill hidden state (heads, first step)
    uint2 (&emb_e)[XM == 2 ? RPT : 1];                                  // first layer: embedding,
    uint2 (&emb_p)[XM == 2 ? RPT : 1];                                  //   position rows
    bool (&emb_ok)[XM == 2 ? RPT : 1];
    int (&st_pl)[XM == 3 ? RPT : 1];
    float4 gv, bv;
    int K, K4, RG, rg, cc;
    bool has_part;

    __device__ __forceinline__ void init(const GemvArgs& a, int tid, int wave) {
        K = a.K;
        K4 = K >> 2;
        RG = T / K4;                                   // row groups (>= 1 for K <= 2048)
        // rg is uniform over a wave (K/4 is a multiple of 64): scalar division
        rg = __builtin_amdgcn_readfirstlane(wave) / (K4 >> 6);
        cc = min((tid - rg * K4) * 4, K - 4);
        has_part = a.part_on != 0;                     // kernel argument: uniform
        gv = make_float4(0.f, 0.f, 0.f, 0.f);
        bv = gv;
    }

    // Phase A: every load of the prologue, from clamped addresses; branches
    // only on wave-uniform conditions (they cost no extra waits).
    __device__ __forceinline__ void load(const GemvArgs& a) {
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
                if (m < a.M && rg < RG) {
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
                if (m < a.M && rg < RG) {
                    const int row = (XM == 1) ? m : ((a.Q > 0) ? m * a.Q + a.Q - 1 : 0);
                    if constexpr (XM == 3) st_pl[j] = a.st[m].pend_len;
                    if (has_part) {
                        pv[0][j] = load_partial_f32(a.part, 0, a.part_rows, a.ldh, row, cc);
#pragma unroll
                        for (int s2 = 1; s2 < 4; ++s2) {
                            if constexpr (BFP) ph[s2 - 1][j] = load_partial_bits(a.part, s2, a.part_rows, a.ldh, row, cc);
                            else pv[s2 % NPV][j] = load_partial_f32(a.part, s2, a.part_rows, a.ldh, row, cc);
                        }
                    } else {
                        hv[j] = *reinterpret_cast<const float4*>(a.h + (size_t)row * a.ldh + cc);
                    }
                    if constexpr (XM == 3) zv[j] = *reinterpret_cast<const float4*>(a.hz + (size_t)m * a.ldh + cc);
                }
            }
        }
    }

    // Phase D: the rows, their statistics and the bf16 LayerNorm output in
    // xs[m][c] (row stride ldl).  `writer` (one workgroup of the grid)
    // stores the completed rows to a.h_out for the next projection.
    // s_gb: [2][K/4] LDS words; s_stat: [waves][RPT].
    __device__ __forceinline__ void build(const GemvArgs& a, bool writer, bf16_t* xs, int ldl, f32x4_t* s_gb,
                                          float2 (*s_stat)[RPT], int wave, int lane) {
        const int M = a.M;
        // row group 0 shares the LayerNorm gain and shift
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
                        const float4 p0 = pv[0][j];
                        float4 p1, p2, p3;
                        if constexpr (BFP) {
                            p1 = bf16x4_to_f32(ph[0][j]);
                            p2 = bf16x4_to_f32(ph[1][j]);
                            p3 = bf16x4_to_f32(ph[NPH - 1][j]);
                        } else {
                            p1 = pv[1 % NPV][j];
                            p2 = pv[2 % NPV][j];
                            p3 = pv[3 % NPV][j];
                        }
                        x.x = (p0.x + p1.x) + (p2.x + p3.x);
                        x.y = (p0.y + p1.y) + (p2.y + p3.y);
                        x.z = (p0.z + p1.z) + (p2.z + p3.z);
                        x.w = (p0.w + p1.w) + (p2.w + p3.w);
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
                                p4[0] = load_partial_f32(a.part, 0, a.part_rows, a.ldh, row, cc);
#pragma unroll
                                for (int s2 = 1; s2 < 4; ++s2)
                                    p4[s2] = BFP ? bf16x4_to_f32(load_partial_bits(a.part, s2, a.part_rows, a.ldh, row, cc))
                                                 : load_partial_f32(a.part, s2, a.part_rows, a.ldh, row, cc);
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
        // one workgroup writes the completed rows (the next projection's residual input)
        if (a.h_out && writer && rg < RG) {
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
            *reinterpret_cast<uint2*>(xs + (size_t)m * ldl + cc) =
                make_uint2(ln_pack2(y0, y1), ln_pack2(y2, y3));
        }
    }

    __device__ static __forceinline__ uint32_t ln_pack2(float a, float b) {
        return bf16x2_bits(a, b);
    }
};

}  // namespace mtp
