// Causal attention of up to 8 query rows of one sequence over its paged fp32
// KV cache (decode: the pending chunk of K tokens; prefill: 8-row tiles of
// the prompt), for the fp32 model.  Memory-bound at decode, so it is VALU:
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
#include "wave.h"

namespace mtp {

namespace {
constexpr int CH = 256;        // keys per LDS chunk (== threads per block)
constexpr int PSTRIDE = 68;    // floats per partial row: max, sum, 2 pad, 64 outputs (16-byte aligned)

template <typename KVT> struct KVRow;
template <> struct KVRow<float> {
    __device__ static __forceinline__ void load8(const float* p, float (&f)[8]) {
        float4 a = *reinterpret_cast<const float4*>(p);
        float4 b = *reinterpret_cast<const float4*>(p + 4);
        f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
        f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
    }
};

__device__ __forceinline__ float wave_max(float v) { return wave_max64(v); }
__device__ __forceinline__ float wave_sum(float v) { return wave_sum64(v); }
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
    const int kend = p.bidir ? p.st[seq].ctx_len : pos0 + nrows;
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
            for (int i = 0; i < QT; ++i) sc[i] = sum8(sc[i]);
            if (dc == 0 && kk < cn) {
#pragma unroll
                for (int i = 0; i < QT; ++i) s_p[i][kk] = (p.bidir || c0 + kk <= pos0 + i) ? sc[i] : -INFINITY;
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
            acc[i][e] = sum_stride8(acc[i][e]);
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
            part[i * PSTRIDE + 4 + dim] = o;
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
            num = fmaf(w, e[4 + dim], num);
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

// fp32 caches only: bf16 caches take the MFMA kernels of attn_mfma.hip
hipError_t attention(hipStream_t st, const AttnArgs& a) {
    if (a.dtype != 0) return hipErrorInvalidValue;
    return attn_launch<float, float>(st, a);
}

}  // namespace mtp

// ---------------------------------------------------------------- decode
// One workgroup per (sequence, head, key split).  The sequence state gives
// the rows (the pending chunk) and the context length directly; each chunk
// of up to 256 keys requests every K and V row at once, and softmax
// statistics run online across chunks.  With one split the normalised bf16
// output is written; with several, each split writes (max, sum,
// unnormalised output) and the merge happens in the consumer (the
// out-projection prologue, or attn_decode_merge).
namespace mtp {

template <typename KVT, typename OutT, int QT>
__global__ __launch_bounds__(256) void attn_decode_kernel(AttnDecArgs p) {
    constexpr int NJ = 8;                     // keys per thread per chunk
    const int b = blockIdx.x, head = blockIdx.y, split = blockIdx.z;
    const int H = gridDim.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int kg = tid >> 3, dc = tid & 7;
    __shared__ float s_p[QT][256];
    __shared__ float s_red[4][QT];
    __shared__ float s_acc[4][QT][64];
    const KVT* pool = reinterpret_cast<const KVT*>(p.kv.pool);
    const size_t vstride = (size_t)p.kv.n_heads * p.kv.page_size * MTP_HEAD_DIM;
    const int kb = split * p.split_len;

    // Issued together, before the sequence state is known: the state, the
    // queries of every possible pending row, and the K/V rows of the first
    // chunk (page table entries first).  Keys past the context are masked
    // below; every address stays inside the sequence's block table row.
    const int nrows = p.st[b].pend_len;
    const int pos0 = p.st[b].ctx_len;
    float qv[QT][8];
#pragma unroll
    for (int i = 0; i < QT; ++i) {
        const float* qp = p.q + (size_t)(b * p.Q + min(i, p.Q - 1)) * p.ldq + head * 64 + dc * 8;
        const float4 x0 = *reinterpret_cast<const float4*>(qp);
        const float4 x1 = *reinterpret_cast<const float4*>(qp + 4);
        qv[i][0] = x0.x * 0.125f; qv[i][1] = x0.y * 0.125f; qv[i][2] = x0.z * 0.125f; qv[i][3] = x0.w * 0.125f;
        qv[i][4] = x1.x * 0.125f; qv[i][5] = x1.y * 0.125f; qv[i][6] = x1.z * 0.125f; qv[i][7] = x1.w * 0.125f;
    }
    const int max_key = p.kv.max_pages_per_seq * p.kv.page_size - 1;
    float kf[NJ][8], vf[NJ][8];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const size_t off = p.kv.offset(b, min(kb + kg + 32 * j, max_key), 0, head) + dc * 8;
        KVRow<KVT>::load8(pool + off, kf[j]);
        KVRow<KVT>::load8(pool + off + vstride, vf[j]);
    }
    if (nrows <= 0) return;
    const int kend = pos0 + nrows;
    if (kb >= kend) return;
    const int ke = min(kb + p.split_len, kend);
#pragma unroll
    for (int i = 0; i < QT; ++i)
        if (i >= nrows)
#pragma unroll
            for (int e = 0; e < 8; ++e) qv[i][e] = 0.f;
    float m_run[QT], l_run[QT], acc[QT][8];
#pragma unroll
    for (int i = 0; i < QT; ++i) {
        m_run[i] = -INFINITY;
        l_run[i] = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[i][e] = 0.f;
    }
    for (int c0 = kb; c0 < ke; c0 += 256) {
        const int cn = min(256, ke - c0);
        if (c0 != kb) {
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                const size_t off = p.kv.offset(b, min(c0 + kg + 32 * j, max_key), 0, head) + dc * 8;
                KVRow<KVT>::load8(pool + off, kf[j]);
                KVRow<KVT>::load8(pool + off + vstride, vf[j]);
            }
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int kk = kg + 32 * j;
            float sc[QT];
#pragma unroll
            for (int i = 0; i < QT; ++i) {
                float s = 0.f;
#pragma unroll
                for (int e = 0; e < 8; ++e) s = fmaf(qv[i][e], kf[j][e], s);
                sc[i] = sum8(s);
            }
            if (dc == 0 && kk < cn) {
#pragma unroll
                for (int i = 0; i < QT; ++i) s_p[i][kk] = (c0 + kk <= pos0 + i) ? sc[i] : -INFINITY;
            }
        }
        __syncthreads();
        float v[QT];
#pragma unroll
        for (int i = 0; i < QT; ++i) {
            v[i] = (tid < cn) ? s_p[i][tid] : -INFINITY;
            const float mx = wave_max(v[i]);
            if (lane == 0) s_red[wave][i] = mx;
        }
        __syncthreads();
        float mnew[QT], scale[QT], pr[QT];
#pragma unroll
        for (int i = 0; i < QT; ++i) {
            const float cm = fmaxf(fmaxf(s_red[0][i], s_red[1][i]), fmaxf(s_red[2][i], s_red[3][i]));
            mnew[i] = fmaxf(m_run[i], cm);
            scale[i] = (m_run[i] == -INFINITY) ? 0.f : __expf(m_run[i] - mnew[i]);
            pr[i] = (v[i] == -INFINITY) ? 0.f : __expf(v[i] - mnew[i]);
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < QT; ++i) {
            if (tid < cn) s_p[i][tid] = pr[i];
            const float sm = wave_sum(pr[i]);
            if (lane == 0) s_red[wave][i] = sm;
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < QT; ++i) {
            const float cs = (s_red[0][i] + s_red[1][i]) + (s_red[2][i] + s_red[3][i]);
            l_run[i] = l_run[i] * scale[i] + cs;
            m_run[i] = mnew[i];
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[i][e] *= scale[i];
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int kk = kg + 32 * j;
            if (kk < cn) {
#pragma unroll
                for (int i = 0; i < QT; ++i) {
                    const float pp = s_p[i][kk];
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[i][e] = fmaf(pp, vf[j][e], acc[i][e]);
                }
            }
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < QT; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            acc[i][e] = sum_stride8(acc[i][e]);
        }
    if (lane < 8) {
#pragma unroll
        for (int i = 0; i < QT; ++i)
#pragma unroll
            for (int e = 0; e < 8; ++e) s_acc[wave][i][dc * 8 + e] = acc[i][e];
    }
    __syncthreads();
    if (p.n_splits == 1) {
        OutT* out = reinterpret_cast<OutT*>(p.out);
        for (int idx = tid; idx < QT * 64; idx += 256) {
            const int i = idx >> 6, dim = idx & 63;
            if (i >= nrows) continue;
            const float o = (s_acc[0][i][dim] + s_acc[1][i][dim]) + (s_acc[2][i][dim] + s_acc[3][i][dim]);
            ActIO<OutT>::store(out + (size_t)(b * p.Q + i) * p.ldo + head * 64 + dim, o / l_run[i]);
        }
        return;
    }
    float* mine = p.part + ((size_t)(b * H + head) * p.n_splits + split) * (QT * PSTRIDE);
    for (int idx = tid; idx < QT * 64; idx += 256) {
        const int i = idx >> 6, dim = idx & 63;
        if (i >= nrows) continue;
        mine[i * PSTRIDE + 4 + dim] = (s_acc[0][i][dim] + s_acc[1][i][dim]) + (s_acc[2][i][dim] + s_acc[3][i][dim]);
        if (dim == 0) {
            mine[i * PSTRIDE] = m_run[i];
            mine[i * PSTRIDE + 1] = l_run[i];
        }
    }
}

// Merge of the split partials: one workgroup per (sequence, head).
template <typename OutT>
__global__ __launch_bounds__(256) void attn_decode_merge(AttnDecArgs p) {
    const int b = blockIdx.x, head = blockIdx.y, H = gridDim.y;
    const int qt = p.qt;
    __shared__ float s_w[64][MTP_ATTN_QT];
    __shared__ float s_l[MTP_ATTN_QT];
    const int nrows = p.st[b].pend_len;
    if (nrows <= 0) return;
    const int kend = p.st[b].ctx_len + nrows;
    const int n_active = min(p.n_splits, (kend + p.split_len - 1) / p.split_len);
    const float* base = p.part + (size_t)(b * H + head) * p.n_splits * (qt * PSTRIDE);
    // (max, sum) of every (split, row) into LDS
    for (int idx = threadIdx.x; idx < n_active * qt; idx += blockDim.x) {
        const int s = idx / qt, i = idx - s * qt;
        s_w[s][i] = (i < nrows) ? base[(size_t)s * qt * PSTRIDE + i * PSTRIDE] : 0.f;
    }
    __syncthreads();
    if (threadIdx.x < qt && (int)threadIdx.x < nrows) {
        const int i = threadIdx.x;
        float M = -INFINITY;
        for (int s = 0; s < n_active; ++s) M = fmaxf(M, s_w[s][i]);
        float L = 0.f;
        for (int s = 0; s < n_active; ++s) {
            const float w = (s_w[s][i] == -INFINITY) ? 0.f : __expf(s_w[s][i] - M);
            L = fmaf(w, base[(size_t)s * qt * PSTRIDE + i * PSTRIDE + 1], L);
            s_w[s][i] = w;
        }
        s_l[i] = L;
    }
    __syncthreads();
    OutT* out = reinterpret_cast<OutT*>(p.out);
    for (int idx = threadIdx.x; idx < qt * 64; idx += blockDim.x) {
        const int i = idx >> 6, dim = idx & 63;
        if (i >= nrows) continue;
        float o = 0.f;
#pragma unroll 8
        for (int s = 0; s < n_active; ++s) o = fmaf(s_w[s][i], base[(size_t)s * qt * PSTRIDE + i * PSTRIDE + 4 + dim], o);
        const int row = b * p.Q + i, col = head * 64 + dim;
        ActIO<OutT>::store(out + (p.packed ? frag_off(row, col, p.ldo) : (size_t)row * p.ldo + col), o / s_l[i]);
    }
}

template <typename KVT, typename OutT>
static hipError_t attn_dec_launch(hipStream_t st, const AttnDecArgs& a) {
    dim3 grid(a.B, a.kv.n_heads, a.n_splits);
    switch (a.qt) {
    case 1: hipLaunchKernelGGL((attn_decode_kernel<KVT, OutT, 1>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((attn_decode_kernel<KVT, OutT, 2>), grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((attn_decode_kernel<KVT, OutT, 4>), grid, dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL((attn_decode_kernel<KVT, OutT, 8>), grid, dim3(256), 0, st, a); break;
    default: return hipErrorInvalidValue;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.n_splits == 1 || !a.merge) return e;
    hipLaunchKernelGGL((attn_decode_merge<OutT>), dim3(a.B, a.kv.n_heads), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t attention_decode_merge(hipStream_t st, const AttnDecArgs& a) {
    if (a.n_splits <= 1) return hipSuccess;
    if (a.dtype == 1) hipLaunchKernelGGL((attn_decode_merge<bf16_t>), dim3(a.B, a.kv.n_heads), dim3(256), 0, st, a);
    else hipLaunchKernelGGL((attn_decode_merge<float>), dim3(a.B, a.kv.n_heads), dim3(256), 0, st, a);
    return hipGetLastError();
}

// fp32 caches only (bf16 decode runs attn_dec_kernel of attn_mfma.hip, whose
// split partials attention_decode_merge also merges)
hipError_t attention_decode(hipStream_t st, const AttnDecArgs& a) {
    if (a.split_len < 32 || a.split_len % 32 || a.n_splits < 1 || a.n_splits > 64) return hipErrorInvalidValue;
    if (a.dtype != 0) return hipErrorInvalidValue;
    return attn_dec_launch<float, float>(st, a);
}

}  // namespace mtp
