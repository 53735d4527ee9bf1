// Row-wise kernels of the trunk: embedding gather, residual reduction and
// LayerNorm.  One workgroup per row; d_model <= 2048.
#include "common.h"
#include "launch.h"
#include "wave.h"

namespace mtp {

namespace {
constexpr int MAXC = 8;   // columns per thread (d <= 2048)

template <typename T> __device__ __forceinline__ float ld(const T* p);
template <> __device__ __forceinline__ float ld<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float ld<bf16_t>(const bf16_t* p) { return bf16_to_f32(*p); }

__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    __syncthreads();
    if (lane == 0) red[wave] = v;
    __syncthreads();
    return (red[0] + red[1]) + (red[2] + red[3]);
}

// LayerNorm of the row held in x[0..nc) (columns c = tid + 256 j), eps 1e-5.
template <typename OutT>
__device__ __forceinline__ void layer_norm_store(const float (&x)[MAXC], int d, const float* g, const float* b,
                                                 OutT* out, float* red) {
    const int tid = threadIdx.x;
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
        int c = tid + 256 * j;
        if (c < d) s += x[j];
    }
    const float mean = block_sum(s, red) / (float)d;
    float v = 0.f;
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
        int c = tid + 256 * j;
        if (c < d) { float t = x[j] - mean; v = fmaf(t, t, v); }
    }
    const float var = block_sum(v, red) / (float)d;
    const float rstd = rsqrtf(var + 1e-5f);
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
        int c = tid + 256 * j;
        if (c < d) ActIO<OutT>::store(out + c, (x[j] - mean) * rstd * g[c] + b[c]);
    }
}
// The same LayerNorm, the output row `row` in fragment order (K = d).
template <typename OutT>
__device__ __forceinline__ void layer_norm_store_pk(const float (&x)[MAXC], int d, const float* g, const float* b,
                                                    OutT* out, int row, float* red) {
    const int tid = threadIdx.x;
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
        int c = tid + 256 * j;
        if (c < d) s += x[j];
    }
    const float mean = block_sum(s, red) / (float)d;
    float v = 0.f;
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
        int c = tid + 256 * j;
        if (c < d) { float t = x[j] - mean; v = fmaf(t, t, v); }
    }
    const float var = block_sum(v, red) / (float)d;
    const float rstd = rsqrtf(var + 1e-5f);
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
        int c = tid + 256 * j;
        if (c < d) ActIO<OutT>::store(out + frag_off(row, c, d), (x[j] - mean) * rstd * g[c] + b[c]);
    }
}
}  // namespace

template <typename WT>
__global__ __launch_bounds__(256) void embed_ln_kernel(EmbedArgs a) {
    __shared__ float red[4];
    const int r = blockIdx.x, tid = threadIdx.x;
    int seq, pos, tok;
    if (a.mode == 0) {
        seq = r / a.Q;
        const int i = r - seq * a.Q;
        const SeqState& s = a.st[seq];
        const bool valid = i < s.pend_len;
        pos = valid ? s.ctx_len + i : -1;
        tok = valid ? s.pend_ids[i] : 0;
        if (tid == 0) {
            a.rows[r] = RowInfo{seq, pos};
            if (i == 0) a.tiles[seq] = make_int2(r, s.pend_len);
        }
    } else {
        RowInfo ri = a.rows[r];
        seq = ri.seq;
        pos = ri.pos;
        tok = a.ids[r];
    }
    using ActT = WT;
    float* h = a.h + (size_t)r * a.d;
    ActT* u = reinterpret_cast<ActT*>(a.u) + (size_t)r * a.d;
    if (pos < 0) {
        for (int c = tid; c < a.d; c += 256) {
            h[c] = 0.f;
            ActIO<ActT>::store(a.packed ? reinterpret_cast<ActT*>(a.u) + frag_off(r, c, a.d) : u + c, 0.f);
        }
        return;
    }
    const WT* table = (pos < a.st[seq].phon_len) ? reinterpret_cast<const WT*>(a.emb_phone)
                                                  : reinterpret_cast<const WT*>(a.emb_ac);
    const WT* erow = table + (size_t)tok * a.d;
    const WT* prow = reinterpret_cast<const WT*>(a.pos) + (size_t)pos * a.d;
    float x[MAXC];
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
        int c = tid + 256 * j;
        x[j] = 0.f;
        if (c < a.d) {
            x[j] = ld<WT>(erow + c) + ld<WT>(prow + c);
            h[c] = x[j];
        }
    }
    if (a.packed) layer_norm_store_pk<ActT>(x, a.d, a.ln_g, a.ln_b, reinterpret_cast<ActT*>(a.u), r, red);
    else layer_norm_store<ActT>(x, a.d, a.ln_g, a.ln_b, u, red);
}

// One row per workgroup, thread t owning the float4 column chunks t and
// t + 256.  Every load of the row (the residual, the bias, all NS split-K
// partial sums, the LayerNorm gamma and beta) is issued before the first
// store, so the kernel costs one global round trip; the partial sums are
// added in split order.
template <typename ActT, int NS>
__global__ __launch_bounds__(256) void resid_ln_kernel(ResidArgs a) {
    __shared__ float red[4];
    const int r = blockIdx.x, tid = threadIdx.x;
    const int d = a.d;
    float* h = a.h + (size_t)r * d;
    const float* __restrict__ part = a.part + (size_t)r * d;
    float4 hv[2], bv[2], pv[NS][2], gv[2], be[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int c = 4 * (tid + 256 * j);
        const int cc = c < d ? c : 0;
        hv[j] = *reinterpret_cast<const float4*>(h + cc);
        bv[j] = *reinterpret_cast<const float4*>(a.bias + cc);
        if (a.ln_g) {
            gv[j] = *reinterpret_cast<const float4*>(a.ln_g + cc);
            be[j] = *reinterpret_cast<const float4*>(a.ln_b + cc);
        }
#pragma unroll
        for (int sp = 0; sp < NS; ++sp)
            pv[sp][j] = *reinterpret_cast<const float4*>(part + sp * a.split_stride + cc);
    }
    float x[8];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        float4 s = pv[0][j];
#pragma unroll
        for (int sp = 1; sp < NS; ++sp) {
            s.x += pv[sp][j].x; s.y += pv[sp][j].y; s.z += pv[sp][j].z; s.w += pv[sp][j].w;
        }
        x[4 * j + 0] = hv[j].x + (s.x + bv[j].x);
        x[4 * j + 1] = hv[j].y + (s.y + bv[j].y);
        x[4 * j + 2] = hv[j].z + (s.z + bv[j].z);
        x[4 * j + 3] = hv[j].w + (s.w + bv[j].w);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int c = 4 * (tid + 256 * j);
        if (c < d) *reinterpret_cast<float4*>(h + c) = make_float4(x[4 * j], x[4 * j + 1], x[4 * j + 2], x[4 * j + 3]);
    }
    if (!a.ln_g) return;
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < 2; ++j)
        if (4 * (tid + 256 * j) < d) sum += (x[4 * j] + x[4 * j + 1]) + (x[4 * j + 2] + x[4 * j + 3]);
    const float mean = block_sum(sum, red) / (float)d;
    float var = 0.f;
#pragma unroll
    for (int j = 0; j < 2; ++j)
        if (4 * (tid + 256 * j) < d) {
#pragma unroll
            for (int i = 0; i < 4; ++i) { const float t = x[4 * j + i] - mean; var = fmaf(t, t, var); }
        }
    const float rstd = rsqrtf(block_sum(var, red) / (float)d + 1e-5f);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int c = 4 * (tid + 256 * j);
        if (c < d) {
            // four consecutive columns stay consecutive in fragment order
            ActT* u = reinterpret_cast<ActT*>(a.u) + (a.packed ? frag_off(r, c, d) : (size_t)r * d + c);
            const float y0 = (x[4 * j + 0] - mean) * rstd * gv[j].x + be[j].x;
            const float y1 = (x[4 * j + 1] - mean) * rstd * gv[j].y + be[j].y;
            const float y2 = (x[4 * j + 2] - mean) * rstd * gv[j].z + be[j].z;
            const float y3 = (x[4 * j + 3] - mean) * rstd * gv[j].w + be[j].w;
            if constexpr (sizeof(ActT) == 2) {
                *reinterpret_cast<uint2*>(u) =
                    make_uint2((uint32_t)f32_to_bf16(y0) | ((uint32_t)f32_to_bf16(y1) << 16),
                               (uint32_t)f32_to_bf16(y2) | ((uint32_t)f32_to_bf16(y3) << 16));
            } else {
                *reinterpret_cast<float4*>(u) = make_float4(y0, y1, y2, y3);
            }
        }
    }
}

template <typename ActT>
__global__ __launch_bounds__(256) void final_ln_kernel(FinalArgs a) {
    __shared__ float red[4];
    const int b = blockIdx.x, tid = threadIdx.x;
    int src = -1;
    if (a.mode == 0) {
        const int pl = a.st[b].pend_len;
        if (a.Q > 0 && pl > 0) src = b * a.Q + pl - 1;
    } else {
        src = a.last_row[b];
    }
    float* hz = a.hz + (size_t)b * a.d;
    float x[MAXC];
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
        int c = tid + 256 * j;
        x[j] = 0.f;
        if (c < a.d) {
            if (src >= 0) {
                x[j] = a.h[(size_t)src * a.d + c];
                hz[c] = x[j];
            } else {
                x[j] = hz[c];
            }
        }
    }
    if (a.z && a.packed) layer_norm_store_pk<ActT>(x, a.d, a.ln_g, a.ln_b, reinterpret_cast<ActT*>(a.z), b, red);
    else if (a.z) layer_norm_store<ActT>(x, a.d, a.ln_g, a.ln_b, reinterpret_cast<ActT*>(a.z) + (size_t)b * a.d, red);
}

hipError_t embed_ln(hipStream_t st, const EmbedArgs& a) {
    if (a.n_rows <= 0) return hipSuccess;
    if (a.dtype == 1) hipLaunchKernelGGL(embed_ln_kernel<bf16_t>, dim3(a.n_rows), dim3(256), 0, st, a);
    else hipLaunchKernelGGL(embed_ln_kernel<float>, dim3(a.n_rows), dim3(256), 0, st, a);
    return hipGetLastError();
}

template <typename ActT>
static hipError_t resid_ln_t(hipStream_t st, const ResidArgs& a) {
    const dim3 g(a.n_rows), b(256);
    switch (a.n_split) {
    case 1: hipLaunchKernelGGL((resid_ln_kernel<ActT, 1>), g, b, 0, st, a); break;
    case 2: hipLaunchKernelGGL((resid_ln_kernel<ActT, 2>), g, b, 0, st, a); break;
    case 4: hipLaunchKernelGGL((resid_ln_kernel<ActT, 4>), g, b, 0, st, a); break;
    case 8: hipLaunchKernelGGL((resid_ln_kernel<ActT, 8>), g, b, 0, st, a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t resid_ln(hipStream_t st, const ResidArgs& a) {
    if (a.n_rows <= 0) return hipSuccess;
    if (a.d % 4 != 0 || a.d > 2048) return hipErrorInvalidValue;
    return a.dtype == 1 ? resid_ln_t<bf16_t>(st, a) : resid_ln_t<float>(st, a);
}

hipError_t final_ln(hipStream_t st, const FinalArgs& a) {
    if (a.dtype == 1) hipLaunchKernelGGL(final_ln_kernel<bf16_t>, dim3(a.B), dim3(256), 0, st, a);
    else hipLaunchKernelGGL(final_ln_kernel<float>, dim3(a.B), dim3(256), 0, st, a);
    return hipGetLastError();
}

// ------------------------------------------------------------ NAR rows
template <typename WT>
__global__ __launch_bounds__(256) void nar_embed_ln_kernel(NarEmbedArgs a) {
    using ActT = WT;
    __shared__ float red[4];
    const int r = blockIdx.x, tid = threadIdx.x;
    const RowInfo ri = a.rows[r];
    const SeqState& s = a.st[ri.seq];
    int code[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) code[i] = a.codes[(size_t)r * 8 + i];
    const bool phon = ri.pos < s.phon_len;
    const int nt = phon ? 0 : (ri.pos < s.prompt_len ? a.n_q : a.stage + 1);   // codebook tables summed
    const WT* ep = reinterpret_cast<const WT*>(a.emb_phone) + (size_t)code[0] * a.d;
    const WT* ec = reinterpret_cast<const WT*>(a.emb_codes);
    const WT* prow = reinterpret_cast<const WT*>(a.pos) + (size_t)ri.pos * a.d;
    const float* sv = a.stage_vec + (size_t)a.stage * a.d;
    float* h = a.h + (size_t)r * a.d;
    float x[MAXC];
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
        const int c = tid + 256 * j;
        x[j] = 0.f;
        if (c < a.d) {
            float e = phon ? ld<WT>(ep + c) : 0.f;
#pragma unroll
            for (int i = 0; i < 8; ++i)
                if (i < nt) e += ld<WT>(ec + ((size_t)i * a.cb + code[i]) * a.d + c);
            x[j] = (e + ld<WT>(prow + c)) + sv[c];
            h[c] = x[j];
        }
    }
    if (a.packed) layer_norm_store_pk<ActT>(x, a.d, a.ln_g, a.ln_b, reinterpret_cast<ActT*>(a.u), r, red);
    else layer_norm_store<ActT>(x, a.d, a.ln_g, a.ln_b, reinterpret_cast<ActT*>(a.u) + (size_t)r * a.d, red);
}

template <typename ActT>
__global__ __launch_bounds__(256) void rows_ln_kernel(RowsLnArgs a) {
    __shared__ float red[4];
    const int r = blockIdx.x, tid = threadIdx.x;
    const float* h = a.h + (size_t)r * a.d;
    float x[MAXC];
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
        const int c = tid + 256 * j;
        x[j] = c < a.d ? h[c] : 0.f;
    }
    if (a.packed) layer_norm_store_pk<ActT>(x, a.d, a.ln_g, a.ln_b, reinterpret_cast<ActT*>(a.u), r, red);
    else layer_norm_store<ActT>(x, a.d, a.ln_g, a.ln_b, reinterpret_cast<ActT*>(a.u) + (size_t)r * a.d, red);
}

// bf16 rows: one wave per row, four rows per workgroup.  Lane l owns the
// eight-column chunks starting at 8 (l + 64 j); eight consecutive columns are
// also consecutive in fragment order, so every chunk leaves as one 16-byte
// store.  Both statistics are wave reductions: no LDS and no barrier.
template <int NCH>
__global__ __launch_bounds__(256) void rows_ln_wave_kernel(RowsLnArgs a) {
    const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (r >= a.n_rows) return;   // wave-uniform
    const int d = a.d;
    const float* h = a.h + (size_t)r * d;
    // the row, gamma and beta all in flight together
    float x[NCH][8];
    float4 gb[NCH][4];
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const int c = 8 * (lane + 64 * j);
        const int cc = c < d ? c : 0;
        const float4 lo = *reinterpret_cast<const float4*>(h + cc);
        const float4 hi = *reinterpret_cast<const float4*>(h + cc + 4);
        gb[j][0] = *reinterpret_cast<const float4*>(a.ln_g + cc);
        gb[j][1] = *reinterpret_cast<const float4*>(a.ln_g + cc + 4);
        gb[j][2] = *reinterpret_cast<const float4*>(a.ln_b + cc);
        gb[j][3] = *reinterpret_cast<const float4*>(a.ln_b + cc + 4);
        const bool ok = c < d;
        x[j][0] = ok ? lo.x : 0.f; x[j][1] = ok ? lo.y : 0.f; x[j][2] = ok ? lo.z : 0.f; x[j][3] = ok ? lo.w : 0.f;
        x[j][4] = ok ? hi.x : 0.f; x[j][5] = ok ? hi.y : 0.f; x[j][6] = ok ? hi.z : 0.f; x[j][7] = ok ? hi.w : 0.f;
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NCH; ++j)
#pragma unroll
        for (int i = 0; i < 8; ++i) s += x[j][i];
    const float mean = wave_sum64(s) / (float)d;
    float v = 0.f;
#pragma unroll
    for (int j = 0; j < NCH; ++j)
        if (8 * (lane + 64 * j) < d) {
#pragma unroll
            for (int i = 0; i < 8; ++i) { const float t = x[j][i] - mean; v = fmaf(t, t, v); }
        }
    const float rstd = rsqrtf(wave_sum64(v) / (float)d + 1e-5f);
    bf16_t* u = reinterpret_cast<bf16_t*>(a.u);
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const int c = 8 * (lane + 64 * j);
        if (c >= d) continue;
        const float4 g0 = gb[j][0], g1 = gb[j][1], b0 = gb[j][2], b1 = gb[j][3];
        const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
        const float b[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const bf16_t e0 = f32_to_bf16((x[j][2 * i] - mean) * rstd * g[2 * i] + b[2 * i]);
            const bf16_t e1 = f32_to_bf16((x[j][2 * i + 1] - mean) * rstd * g[2 * i + 1] + b[2 * i + 1]);
            w[i] = (uint32_t)e0 | ((uint32_t)e1 << 16);
        }
        bf16_t* dst = u + (a.packed ? frag_off(r, c, d) : (size_t)r * d + c);
        *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
    }
}

// One wave per listed row.
__global__ __launch_bounds__(256) void rows_argmax_kernel(ArgmaxArgs a) {
    const int i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (i >= a.n) return;
    const int row = a.tgt_rows[i];
    const float* lg = a.logits + (size_t)row * a.ld;
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    for (int c = lane; c < a.cb; c += 64) {
        const float v = lg[c];
        const bool b = (v > bv) | ((v == bv) & (c < bi));
        bv = b ? v : bv;
        bi = b ? c : bi;
    }
    for (int o = 32; o >= 1; o >>= 1) {
        const float ov = __shfl_xor(bv, o);
        const int oi = __shfl_xor(bi, o);
        const bool b = (ov > bv) | ((ov == bv) & (oi < bi));
        bv = b ? ov : bv;
        bi = b ? oi : bi;
    }
    if (lane == 0) a.codes[(size_t)row * 8 + a.slot] = bi < a.cb ? bi : 0;   // (all-NaN row: code 0)
}

hipError_t nar_embed_ln(hipStream_t st, const NarEmbedArgs& a) {
    if (a.n_rows <= 0) return hipSuccess;
    if (a.dtype == 1) hipLaunchKernelGGL(nar_embed_ln_kernel<bf16_t>, dim3(a.n_rows), dim3(256), 0, st, a);
    else hipLaunchKernelGGL(nar_embed_ln_kernel<float>, dim3(a.n_rows), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t rows_ln(hipStream_t st, const RowsLnArgs& a) {
    if (a.n_rows <= 0) return hipSuccess;
    if (a.dtype == 1 && a.d % 8 == 0 && a.d <= 2048) {
        const dim3 g((a.n_rows + 3) / 4), b(256);
        switch ((a.d + 511) / 512) {
        case 1: hipLaunchKernelGGL(rows_ln_wave_kernel<1>, g, b, 0, st, a); break;
        case 2: hipLaunchKernelGGL(rows_ln_wave_kernel<2>, g, b, 0, st, a); break;
        case 3: hipLaunchKernelGGL(rows_ln_wave_kernel<3>, g, b, 0, st, a); break;
        default: hipLaunchKernelGGL(rows_ln_wave_kernel<4>, g, b, 0, st, a); break;
        }
        return hipGetLastError();
    }
    if (a.dtype == 1) hipLaunchKernelGGL(rows_ln_kernel<bf16_t>, dim3(a.n_rows), dim3(256), 0, st, a);
    else hipLaunchKernelGGL(rows_ln_kernel<float>, dim3(a.n_rows), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t rows_argmax(hipStream_t st, const ArgmaxArgs& a) {
    if (a.n <= 0) return hipSuccess;
    hipLaunchKernelGGL(rows_argmax_kernel, dim3((a.n + 3) / 4), dim3(256), 0, st, a);
    return hipGetLastError();
}

// ------------------------------------------------------------ cache flush
__global__ __launch_bounds__(256) void cache_flush_kernel(const uint4* p, size_t n16, uint32_t* sink) {
    uint32_t acc = 0;
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += (size_t)gridDim.x * 256) {
        const uint4 v = p[i];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x9E3779B9u) sink[blockIdx.x & 63] = acc;   // keeps the loads alive
}

hipError_t cache_flush(hipStream_t st, void* buf, size_t bytes) {
    if (!buf || bytes < 1024 || bytes % 16) return hipErrorInvalidValue;
    hipLaunchKernelGGL(cache_flush_kernel, dim3(2048), dim3(256), 0, st, reinterpret_cast<const uint4*>(buf),
                       bytes / 16, reinterpret_cast<uint32_t*>(buf));
    return hipGetLastError();
}

}  // namespace mtp
