// Attention for the bf16 cache on MFMA: decode (attn_dec_kernel) and prefill
// (attn_prefill_fa_kernel), flash-style online softmax with every key product on
// the matrix cores and the probabilities kept in registers.
#include <math.h>

#include "attn_dec.h"
#include "common.h"
#include "launch.h"
#include "wave.h"

namespace mtp {

namespace {
__device__ __forceinline__ uint32_t pk2(float a, float b) {
    return bf16x2_bits(a, b);
}
}  // namespace

// Decode attention (attn_dec.h): one workgroup per (sequence, head, key
// split) of NW waves.
template <int NW, int PD>
__global__ __launch_bounds__(64 * NW) void attn_dec_kernel(AttnMfmaArgs p) {
    attn_dec_body<NW, PD, 16, false>(p, blockIdx.x, blockIdx.y, blockIdx.z, gridDim.y, FrontSync{});
}

template <int NW, int PD>
static hipError_t attn_dec_go_pd(hipStream_t st, const AttnMfmaArgs& a) {
    const size_t lds = (size_t)NW * 16 * 64 * sizeof(float);    // attn_dec_body's s_acc at QN = 16
    static bool attr_set = false;
    if (!attr_set && lds > 48 * 1024) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_dec_kernel<NW, PD>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (err != hipSuccess) return err;
        attr_set = true;
    }
    hipLaunchKernelGGL((attn_dec_kernel<NW, PD>), dim3(a.n_tiles, a.kv.n_heads, a.n_splits), dim3(64 * NW), lds, st, a);
    return hipGetLastError();
}

// Ring depth: two 16-key groups per wave once a split holds that many, for
// 16-wave workgroups (one per CU); smaller workgroups keep one group in
// flight per wave and gain more waves per CU instead (at batch 32: 684 vs
// 695 us per decode step).
template <int NW>
static hipError_t attn_dec_go(hipStream_t st, const AttnMfmaArgs& a) {
    const int groups = (a.split_len + 16 * NW - 1) / (16 * NW);
    if (groups >= 2 && NW == 16) return attn_dec_go_pd<NW, 2>(st, a);
    return attn_dec_go_pd<NW, 1>(st, a);
}

// Prefill attention, flash style (bf16 cache, 16-key pages): one workgroup
// of 4 waves per (64-row query tile, head); wave w owns the tile's query rows
// 16 w .. 16 w + 15 and runs over the keys in blocks of 64 (four pages).
// Each block's K rows and V^T rows are staged once in LDS for the four waves
// (double-buffered: the next block's loads sit in registers while the
// current one is consumed; keys past the context are zeroed in V^T, whose
// products with a zero probability must not meet a NaN), and each wave makes
// one online-softmax update per block:
//   S^T[key][q] = K[key][:] . Q[q][:]       16 x 16 x 32 MFMA, 2 k steps per
//                                          16-key tile; Q is pre-scaled by
//                                          log2(e) / 8, so exp2 applies
//   O^T[dim][q] += V^T[dim][key] P^T[key][q] 16 x 16 x 32 MFMA whose 32-deep
//                                          k index takes keys 4 g .. 4 g + 3
//                                          of two 16-key tiles: lane (r, g)'s
//                                          P^T operand is then exactly its own
//                                          S^T values after exp2.
// Causal, or bidirectional (every row sees its sequence's ctx_len keys) with
// p.bidir.  Rows of the tile past its row count compute and are not stored.
// Workgroup barrier for LDS hand-offs: waits for this wave's LDS operations
// only, so global loads issued for later blocks stay in flight across it
// (__syncthreads() would wait for them too).
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__global__ __launch_bounds__(256) void attn_prefill_fa_kernel(AttnMfmaArgs p) {
    constexpr int KP = 72;                       // padded staged row (bf16): 144 B
    __shared__ __attribute__((aligned(16))) bf16_t sk[2][64 * KP];   // [key][dim]
    __shared__ __attribute__((aligned(16))) bf16_t sv[2][64 * KP];   // [dim][key]
    const int head = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int2 tile = p.tiles[blockIdx.x];
    const int row0 = tile.x, nrows = tile.y;
    if (nrows <= 0) return;                      // uniform over the workgroup
    const int b = p.rows[row0].seq;
    const int pos0 = p.rows[row0].pos;
    const bool bidir = p.bidir != 0;
    const int kend = bidir ? p.st[b].ctx_len : pos0 + nrows;
    const int nblk = (kend + 63) >> 6;
    const bf16_t* pool = reinterpret_cast<const bf16_t*>(p.kv.pool);
    // the sequence's pages up to the last block, looked up once into LDS (a
    // load whose address waits on a page-table load would also wait for the
    // loads of the block in flight before it)
    extern __shared__ int s_pg[];
    const int npg = min(p.kv.max_pages_per_seq, nblk * 4);
    for (int i = tid; i < npg; i += 256) s_pg[i] = p.kv.block_table[(size_t)b * p.kv.max_pages_per_seq + i];
    __syncthreads();

    // staging: thread t moves the 16-byte chunks t and t + 256 of the block's
    // four 2 KB K blocks and of its four 2 KB V^T blocks
    // Two register sets (A, B): a block's loads go out two blocks before its
    // compute (one block of compute hid too little of the load latency).
    // Thread t moves the 16-byte chunks t and t + 256 of the block's four
    // 2 KB K blocks and of its four 2 KB V^T blocks; the chunks are plain
    // variables (arrays of them ended up in scratch memory).
#define MTP_FA_GLOAD1(KR, VR, I, BLK)                                                             \
    {                                                                                             \
        const int c = tid + 256 * (I), pg = c >> 7, w = c & 127;                                  \
        const int page = s_pg[min((BLK) * 4 + pg, npg - 1)];                                      \
        KR = *reinterpret_cast<const uint4*>(pool + kv_page_block(p.kv, page, 0, head) + w * 8);  \
        VR = *reinterpret_cast<const uint4*>(pool + kv_page_block(p.kv, page, 1, head) + w * 8);  \
    }
#define MTP_FA_SSTORE1(KR, VR, I, BUF, BLK)                                                       \
    {                                                                                             \
        const int c = tid + 256 * (I), pg = c >> 7, w = c & 127;                                  \
        /* K chunk w: slot w / 8, dims 8 (w % 8) ..; V^T chunk w: dim w / 2, keys 8 (w % 2) .. */ \
        *reinterpret_cast<uint4*>(&sk[BUF][(pg * 16 + (w >> 3)) * KP + (w & 7) * 8]) = KR;        \
        uint4 v = VR;                                                                             \
        const int k0 = (BLK) * 64 + pg * 16 + (w & 1) * 8;                                        \
        if (k0 + 8 > kend) { /* keys past the context: zero */                                    \
            uint32_t m[4];                                                                        \
            _Pragma("unroll") for (int j = 0; j < 4; ++j) {                                       \
                const uint32_t lo = k0 + 2 * j < kend ? 0x0000FFFFu : 0u;                         \
                const uint32_t hi = k0 + 2 * j + 1 < kend ? 0xFFFF0000u : 0u;                     \
                m[j] = lo | hi;                                                                   \
            }                                                                                     \
            v = make_uint4(v.x & m[0], v.y & m[1], v.z & m[2], v.w & m[3]);                       \
        }                                                                                         \
        *reinterpret_cast<uint4*>(&sv[BUF][(w >> 1) * KP + pg * 16 + (w & 1) * 8]) = v;           \
    }
    uint4 kA0, kA1, vA0, vA1, kB0, kB1, vB0, vB1;
    auto gloadA = [&](int blk) { MTP_FA_GLOAD1(kA0, vA0, 0, blk) MTP_FA_GLOAD1(kA1, vA1, 1, blk) };
    auto gloadB = [&](int blk) { MTP_FA_GLOAD1(kB0, vB0, 0, blk) MTP_FA_GLOAD1(kB1, vB1, 1, blk) };
    auto sstoreA = [&](int buf, int blk) { MTP_FA_SSTORE1(kA0, vA0, 0, buf, blk) MTP_FA_SSTORE1(kA1, vA1, 1, buf, blk) };
    auto sstoreB = [&](int buf, int blk) { MTP_FA_SSTORE1(kB0, vB0, 0, buf, blk) MTP_FA_SSTORE1(kB1, vB1, 1, buf, blk) };
#undef MTP_FA_GLOAD1
#undef MTP_FA_SSTORE1

    // every stage issues its loads and its LDS stores, the last ones of a
    // clamped (repeated) block into a buffer nobody reads: with conditional
    // ones the compiler's wait counts become the conservative merge of both
    // paths and wait for the newest loads too
    gloadA(0);
    gloadB(min(1, nblk - 1));
    bf16x8_t qf[2];
    {
        const float sc = 0.18033688011112042f;   // log2(e) / sqrt(64)
        const float* qp = p.q + (size_t)(row0 + min(16 * wave + r, nrows - 1)) * p.ldq + head * 64 + g * 8;
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
            const float4 x = *reinterpret_cast<const float4*>(qp + 32 * h2);
            const float4 y = *reinterpret_cast<const float4*>(qp + 32 * h2 + 4);
            qf[h2] = __builtin_bit_cast(bf16x8_t, make_uint4(pk2(x.x * sc, x.y * sc), pk2(x.z * sc, x.w * sc),
                                                             pk2(y.x * sc, y.y * sc), pk2(y.z * sc, y.w * sc)));
        }
    }
    const int qpos = pos0 + 16 * wave + r;       // this lane's query position
    const int qlast = pos0 + 16 * wave + 15;     // the wave's last query position
    float m_run = -INFINITY, l_run = 0.f;
    f32x4_t acc[4];
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) acc[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    auto compute = [&](int buf, int blk) {
        const int kb0 = blk * 64;
        if (bidir || kb0 <= qlast) {             // uniform per wave: some key of the block is visible
            const bf16_t* K = sk[buf];
            const bf16_t* VT = sv[buf];
            f32x4_t sc4[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const bf16_t* kr = K + (16 * t + r) * KP + 8 * g;
                sc4[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*reinterpret_cast<const bf16x8_t*>(kr), qf[0],
                                                                 f32x4_t{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                sc4[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*reinterpret_cast<const bf16x8_t*>(kr + 32), qf[1],
                                                                 sc4[t], 0, 0, 0);
            }
            if (kb0 + 64 > kend || (!bidir && kb0 + 63 > pos0 + 16 * wave)) {   // uniform per wave
#pragma unroll
                for (int t = 0; t < 4; ++t)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int key = kb0 + 16 * t + 4 * g + e;
                        const bool ok = key < kend && (bidir || key <= qpos);
                        sc4[t][e] = ok ? sc4[t][e] : -INFINITY;
                    }
            }
            float mx = -INFINITY;
#pragma unroll
            for (int t = 0; t < 4; ++t)
                mx = fmaxf(mx, fmaxf(fmaxf(sc4[t][0], sc4[t][1]), fmaxf(sc4[t][2], sc4[t][3])));
            mx = xor16_max(mx);
            mx = xor32_max(mx);
            const float m_new = fmaxf(m_run, mx);
            const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
            const float scale = __builtin_amdgcn_exp2f(m_run - m_use);
            float sum = 0.f;
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    sc4[t][e] = __builtin_amdgcn_exp2f(sc4[t][e] - m_use);
                    sum += sc4[t][e];
                }
            sum = xor16_sum(sum);
            sum = xor32_sum(sum);
            l_run = l_run * scale + sum;
            m_run = m_new;
#pragma unroll
            for (int dt = 0; dt < 4; ++dt) acc[dt] *= scale;
#pragma unroll
            for (int pr = 0; pr < 2; ++pr) {
                const int t0 = 2 * pr, t1 = 2 * pr + 1;
                const bf16x8_t pf = __builtin_bit_cast(
                    bf16x8_t, make_uint4(pk2(sc4[t0][0], sc4[t0][1]), pk2(sc4[t0][2], sc4[t0][3]),
                                         pk2(sc4[t1][0], sc4[t1][1]), pk2(sc4[t1][2], sc4[t1][3])));
#pragma unroll
                for (int dt = 0; dt < 4; ++dt) {
                    const bf16_t* vr = VT + (16 * dt + r) * KP + 4 * g;
                    const uint2 va = *reinterpret_cast<const uint2*>(vr + 16 * t0);
                    const uint2 vb = *reinterpret_cast<const uint2*>(vr + 16 * t1);
                    const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, make_uint4(va.x, va.y, vb.x, vb.y));
                    acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, acc[dt], 0, 0, 0);
                }
            }
        }
    };
    sstoreA(0, 0);
    lds_barrier();
    for (int blk = 0; blk < nblk; blk += 2) {
        // block blk in LDS buffer 0, block blk + 1 in registers B
        gloadA(min(blk + 2, nblk - 1));
        compute(0, blk);
        sstoreB(1, min(blk + 1, nblk - 1));
        lds_barrier();
        if (blk + 1 >= nblk) break;
        // block blk + 1 in LDS buffer 1, block blk + 2 in registers A
        gloadB(min(blk + 3, nblk - 1));
        compute(1, blk + 1);
        sstoreA(0, min(blk + 2, nblk - 1));
        lds_barrier();
    }

    // O = O^T / l: lane (r, g) holds dims 16 dt + 4 g .. + 3 of query row r
    const int q = 16 * wave + r;
    if (q < nrows) {
        const float inv = 1.0f / l_run;
        const int row = row0 + q;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) {
            const int col = head * 64 + 16 * dt + 4 * g;
            const uint2 o = make_uint2(pk2(acc[dt][0] * inv, acc[dt][1] * inv), pk2(acc[dt][2] * inv, acc[dt][3] * inv));
            *reinterpret_cast<uint2*>(p.out + (p.packed ? frag_off(row, col, p.ldo) : (size_t)row * p.ldo + col)) = o;
        }
    }
}

hipError_t attention_mfma(hipStream_t st, const AttnMfmaArgs& a) {
    if (a.split_len < 32 || a.n_splits < 1 || a.n_splits > 64 || a.kv.page_size != 16) return hipErrorInvalidValue;
    if (a.mode == 0) {
        // decode: pending chunk of at most 16 rows per sequence
        if (a.Q < 1 || a.Q > 16 || a.qt < a.Q || a.split_len % 16) return hipErrorInvalidValue;
        // waves per workgroup: at most one per 16-key group of a split, and
        // few enough that the whole grid is resident at once (16 waves per CU
        // at this kernel's register count)
        const int grid = a.n_tiles * a.kv.n_heads * a.n_splits;
        const int nw_split = a.split_len >= 256 ? 16 : (a.split_len >= 128 ? 8 : 4);
        const int nw_grid = grid <= 256 ? 16 : (grid <= 512 ? 8 : 4);
        const int nw = nw_split < nw_grid ? nw_split : nw_grid;
        if (nw == 16) return attn_dec_go<16>(st, a);
        if (nw == 8) return attn_dec_go<8>(st, a);
        return attn_dec_go<4>(st, a);
    }
    // prefill: tiles of at most a.qt rows (16, 32 or 64), one split
    if (a.n_splits != 1) return hipErrorInvalidValue;
    if (a.qt != 64) return hipErrorInvalidValue;
    // dynamic LDS: one page number per page of a sequence
    const size_t lds = (size_t)a.kv.max_pages_per_seq * sizeof(int);
    if (lds > 48 * 1024) return hipErrorInvalidValue;
    hipLaunchKernelGGL(attn_prefill_fa_kernel, dim3(a.n_tiles, a.kv.n_heads, 1), dim3(256), lds, st, a);
    return hipGetLastError();
}

}  // namespace mtp
