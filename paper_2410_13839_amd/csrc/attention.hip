// Causal attention of up to 8 query rows of one sequence over its paged KV
// cache (decode: the pending chunk of K tokens; prefill: 8-row tiles of the
// prompt).  Memory-bound at decode, so it is VALU, not MFMA:
//
//  * one workgroup per (tile, head, key split); 256 threads = 32 key groups
//    x 8 dimension chunks, so 8 consecutive lanes read one key's 128-byte
//    head row and a wave reads 1 KB of contiguous page memory per load;
//  * scores are reduced over the 8 dimension lanes with xor shuffles and
//    staged in LDS for a chunk of 256 keys, softmax statistics are kept
//    online across chunks (running max, running sum, rescaled accumulator);
//  * with several key splits (flash-decoding style), each split writes
//    (max, sum, unnormalised output) and attn_combine merges them.
#include <math.h>

#include "common.h"
#include "launch.h"

namespace mtp {

namespace {
constexpr int CH = 256;        // keys per LDS chunk (== threads per block)
constexpr int PSTRIDE = 66;    // floats per partial row: max, sum, 64 outputs

template <typename KVT> struct KVRow;
template <> struct KVRow<bf16_t> {
    __device__ static __forceinline__ void load8(const bf16_t* p, float (&f)[8]) {
        uint4 v = *reinterpret_cast<const uint4*>(p);
        f[0] = __uint_as_float(v.x << 16); f[1] = __uint_as_float(v.x & 0xFFFF0000u);
        f[2] = __uint_as_float(v.y << 16); f[3] = __uint_as_float(v.y & 0xFFFF0000u);
        f[4] = __uint_as_float(v.z << 16); f[5] = __uint_as_float(v.z & 0xFFFF0000u);
        f[6] = __uint_as_float(v.w << 16); f[7] = __uint_as_float(v.w & 0xFFFF0000u);
    }
};
template <> struct KVRow<float> {
    __device__ static __forceinline__ void load8(const float* p, float (&f)[8]) {
        float4 a = *reinterpret_cast<const float4*>(p);
        float4 b = *reinterpret_cast<const float4*>(p + 4);
        f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
        f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
    }
};

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    return v;
}
}  // namespace

template <typename KVT, typename OutT, int QT>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs p) {
    const int tile = blockIdx.x, head = blockIdx.y, split = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int kg = tid >> 3, dc = tid & 7;
    __shared__ float s_p[QT][CH];
    __shared__ float s_red[4][QT];
    __shared__ float s_acc[4][QT][64];

    const int2 tl = p.tiles[tile];
    const int row0 = tl.x, nrows = tl.y;
    if (nrows <= 0) return;
    float* part = nullptr;
    if (p.n_splits > 1)
        part = p.part + ((size_t)(tile * gridDim.y + head) * p.n_splits + split) * (QT * PSTRIDE);
    const int seq = p.rows[row0].seq;
    const int pos0 = p.rows[row0].pos;
    const int kend = pos0 + nrows;
    const int kb = split * p.split_len;
    const int ke = min(kb + p.split_len, kend);
    if (kb >= ke) {
        if (part)
            for (int e = tid; e < QT * PSTRIDE; e += 256) part[e] = (e % PSTRIDE == 0) ? -INFINITY : 0.f;
        return;
    }

    float qv[QT][8];
#pragma unroll
    for (int i = 0; i < QT; ++i) {
        if (i < nrows) {
            const float* qp = p.q + (size_t)(row0 + i) * p.ldq + head * 64 + dc * 8;
            float4 a = *reinterpret_cast<const float4*>(qp);
            float4 b = *reinterpret_cast<const float4*>(qp + 4);
            qv[i][0] = a.x * 0.125f; qv[i][1] = a.y * 0.125f; qv[i][2] = a.z * 0.125f; qv[i][3] = a.w * 0.125f;
            qv[i][4] = b.x * 0.125f; qv[i][5] = b.y * 0.125f; qv[i][6] = b.z * 0.125f; qv[i][7] = b.w * 0.125f;
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) qv[i][e] = 0.f;
        }
    }
    float m_run[QT], l_run[QT], acc[QT][8];
#pragma unroll
    for (int i = 0; i < QT; ++i) {
        m_run[i] = -INFINITY;
        l_run[i] = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[i][e] = 0.f;
    }
    const KVT* pool = reinterpret_cast<const KVT*>(p.kv.pool);

    for (int c0 = kb; c0 < ke; c0 += CH) {
        const int cn = min(CH, ke - c0);
        // scores q . k for this chunk
        for (int j = 0; j < CH / 32; ++j) {
            const int kk = kg + 32 * j;
            if (j * 32 >= cn) break;                       // uniform across the block
            float sc[QT];
            if (kk < cn) {
                float kf[8];
                KVRow<KVT>::load8(pool + p.kv.offset(seq, c0 + kk, 0, head) + dc * 8, kf);
#pragma unroll
                for (int i = 0; i < QT; ++i) {
                    float s = 0.f;
#pragma unroll
                    for (int e = 0; e < 8; ++e) s = fmaf(qv[i][e], kf[e], s);
                    sc[i] = s;
                }
            } else {
#pragma unroll
                for (int i = 0; i < QT; ++i) sc[i] = 0.f;
            }
#pragma unroll
            for (int i = 0; i < QT; ++i) {
                sc[i] += __shfl_xor(sc[i], 1);
                sc[i] += __shfl_xor(sc[i], 2);
                sc[i] += __shfl_xor(sc[i], 4);
            }
            if (dc == 0 && kk < cn) {
#pragma unroll
                for (int i = 0; i < QT; ++i) s_p[i][kk] = (c0 + kk <= pos0 + i) ? sc[i] : -INFINITY;
            }
        }
        __syncthreads();
        // chunk softmax statistics; thread tid owns key tid of the chunk
        float v[QT];
#pragma unroll
        for (int i = 0; i < QT; ++i) v[i] = (tid < cn) ? s_p[i][tid] : -INFINITY;
#pragma unroll
        for (int i = 0; i < QT; ++i) {
            float mx = wave_max(v[i]);
            if (lane == 0) s_red[wave][i] = mx;
        }
        __syncthreads();
        float mnew[QT], scale[QT], pr[QT];
#pragma unroll
        for (int i = 0; i < QT; ++i) {
            float cm = fmaxf(fmaxf(s_red[0][i], s_red[1][i]), fmaxf(s_red[2][i], s_red[3][i]));
            mnew[i] = fmaxf(m_run[i], cm);
            scale[i] = (m_run[i] == -INFINITY) ? 0.f : __expf(m_run[i] - mnew[i]);
            pr[i] = (v[i] == -INFINITY) ? 0.f : __expf(v[i] - mnew[i]);
        }
        __syncthreads();
        if (tid < cn) {
#pragma unroll
            for (int i = 0; i < QT; ++i) s_p[i][tid] = pr[i];
        }
#pragma unroll
        for (int i = 0; i < QT; ++i) {
            float sm = wave_sum(pr[i]);
            if (lane == 0) s_red[wave][i] = sm;
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < QT; ++i) {
            float cs = (s_red[0][i] + s_red[1][i]) + (s_red[2][i] + s_red[3][i]);
            l_run[i] = l_run[i] * scale[i] + cs;
            m_run[i] = mnew[i];
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[i][e] *= scale[i];
        }
        // probabilities x V
        for (int j = 0; j < CH / 32; ++j) {
            const int kk = kg + 32 * j;
            if (j * 32 >= cn) break;
            if (kk < cn) {
                float vf[8];
                KVRow<KVT>::load8(pool + p.kv.offset(seq, c0 + kk, 1, head) + dc * 8, vf);
#pragma unroll
                for (int i = 0; i < QT; ++i) {
                    const float pp = s_p[i][kk];
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[i][e] = fmaf(pp, vf[e], acc[i][e]);
                }
            }
        }
        __syncthreads();
    }

    // reduce the accumulators over the 32 key groups
#pragma unroll
    for (int i = 0; i < QT; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            float a = acc[i][e];
            a += __shfl_xor(a, 8);
            a += __shfl_xor(a, 16);
            a += __shfl_xor(a, 32);
            acc[i][e] = a;
        }
    if (lane < 8) {
#pragma unroll
        for (int i = 0; i < QT; ++i)
#pragma unroll
            for (int e = 0; e < 8; ++e) s_acc[wave][i][dc * 8 + e] = acc[i][e];
    }
    __syncthreads();
    for (int idx = tid; idx < QT * 64; idx += 256) {
        const int i = idx >> 6, dim = idx & 63;
        if (i >= nrows) continue;
        const float o = (s_acc[0][i][dim] + s_acc[1][i][dim]) + (s_acc[2][i][dim] + s_acc[3][i][dim]);
        if (part) {
            part[i * PSTRIDE + 2 + dim] = o;
            if (dim == 0) {
                part[i * PSTRIDE] = m_run[i];
                part[i * PSTRIDE + 1] = l_run[i];
            }
        } else {
            ActIO<OutT>::store(reinterpret_cast<OutT*>(p.out) + (size_t)(row0 + i) * p.ldo + head * 64 + dim,
                               o / l_run[i]);
        }
    }
}

template <typename OutT>
__global__ __launch_bounds__(256) void attn_combine(AttnArgs p) {
    const int tile = blockIdx.x, head = blockIdx.y;
    const int2 tl = p.tiles[tile];
    const int row0 = tl.x, nrows = tl.y;
    const int qt = p.qt;
    const float* base = p.part + (size_t)(tile * gridDim.y + head) * p.n_splits * (qt * PSTRIDE);
    for (int idx = threadIdx.x; idx < qt * 64; idx += blockDim.x) {
        const int i = idx >> 6, dim = idx & 63;
        if (i >= nrows) continue;
        float M = -INFINITY;
        for (int s = 0; s < p.n_splits; ++s) M = fmaxf(M, base[(size_t)s * qt * PSTRIDE + i * PSTRIDE]);
        float num = 0.f, den = 0.f;
        for (int s = 0; s < p.n_splits; ++s) {
            const float* e = base + (size_t)s * qt * PSTRIDE + i * PSTRIDE;
            const float m = e[0];
            if (m == -INFINITY) continue;
            const float w = __expf(m - M);
            den = fmaf(w, e[1], den);
            num = fmaf(w, e[2 + dim], num);
        }
        ActIO<OutT>::store(reinterpret_cast<OutT*>(p.out) + (size_t)(row0 + i) * p.ldo + head * 64 + dim, num / den);
    }
}

template <typename KVT, typename OutT>
static hipError_t attn_launch(hipStream_t st, const AttnArgs& a) {
    dim3 grid(a.n_tiles, a.kv.n_heads, a.n_splits);
    switch (a.qt) {
    case 1: hipLaunchKernelGGL((attn_kernel<KVT, OutT, 1>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((attn_kernel<KVT, OutT, 2>), grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((attn_kernel<KVT, OutT, 4>), grid, dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL((attn_kernel<KVT, OutT, 8>), grid, dim3(256), 0, st, a); break;
    default: return hipErrorInvalidValue;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.n_splits <= 1) return e;
    hipLaunchKernelGGL((attn_combine<OutT>), dim3(a.n_tiles, a.kv.n_heads), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t attention(hipStream_t st, const AttnArgs& a) {
    if (a.dtype == 1) return attn_launch<bf16_t, bf16_t>(st, a);
    return attn_launch<float, float>(st, a);
}

}  // namespace mtp
