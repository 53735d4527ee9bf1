// Attention for the bf16 cache on MFMA: decode (attn_dec_kernel) and prefill
// (attn_prefill_fa_kernel), flash-style online softmax with every key product on
// the matrix cores and the probabilities kept in registers.
#include <math.h>

#include "common.h"
#include "launch.h"
#include "wave.h"

namespace mtp {

namespace {
constexpr int PSTR = 68;     // floats per partial row: max, sum, 2 pad, 64 outputs

__device__ __forceinline__ uint32_t pk2(float a, float b) {
    return (uint32_t)f32_to_bf16(a) | ((uint32_t)f32_to_bf16(b) << 16);
}
}  // namespace

// Decode attention over a bf16 cache, NW waves per workgroup: one workgroup
// per (sequence, head, key split); within a 16*NW-key chunk each wave owns 16
// consecutive keys and keeps its own online-softmax state (running max, sum,
// O^T accumulators) across the chunks of its split, so the chunk loop has no
// barrier; the NW states are merged through LDS once at the end.
//   S^T[key][q] = K[key][:] . Q[q][:] / 8    v_mfma_f32_16x16x32_bf16 (2 k-steps)
//   O^T[dim][q] += V^T[dim][key] P^T[key][q] v_mfma_f32_16x16x16_bf16: the B
//                                             operand (4 keys x query per lane)
//                                             is exactly the lane's S^T result
//                                             after exp, so P never leaves registers
// A CU streams only ~25 GB/s from HBM, so short splits spread a small batch's
// keys over many CUs (64-key splits, 4 waves, at batch 1); long splits use up
// to 16 waves.  With long splits each wave keeps PD of its 16-key groups in
// flight (a register ring, rotated by unrolling), so a CU's outstanding KV
// reads grow with PD instead of stalling on one round trip per chunk.
typedef short s16x4_t __attribute__((ext_vector_type(4)));

template <int NW, int PD>
__global__ __launch_bounds__(64 * NW) void attn_dec_kernel(AttnMfmaArgs p) {
    const int b = blockIdx.x, head = blockIdx.y, split = blockIdx.z;
    const int H = gridDim.y;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, g = lane >> 4;
    extern __shared__ float s_o[];               // [NW waves][64 dims][17]
    __shared__ float s_m[NW][16], s_l[NW][16];
    constexpr int CH = 16 * NW;                  // keys per chunk
    const bf16_t* pool = reinterpret_cast<const bf16_t*>(p.kv.pool);
    const int kb = split * p.split_len;
    const int row0 = b * p.Q;

    // Key groups start at multiples of 16 (splits and chunks are multiples of
    // 16 keys), so each wave's 16-key group is exactly one cache page; group i
    // of this wave is page (kb / 16) + wave + NW i of the sequence.  Lane j
    // holds the page number of group j (64 groups at a time, reloaded every
    // 64): a group's addresses then come from a register read, not from a
    // page-table load that, completing in order with the vector loads before
    // it, would hold each group's K / V loads behind the previous group's.
    // Page indexes are clamped to the sequence's block table, whose unused
    // entries name page 0, so loads past the context stay in the pool.
    const int maxp = p.kv.max_pages_per_seq;
    const int32_t* btab = p.kv.block_table + (size_t)b * maxp;
    const int pg0 = (kb >> 4) + wave;
    int pages = btab[min(pg0 + NW * lane, maxp - 1)];
    uint4 kf[PD][2];
    uint2 vf[PD][4];
    auto load_keys = [&](int u, int gi) {        // gi: this wave's group index (uniform)
        if ((gi & 63) == 0 && gi > 0) pages = btab[min(pg0 + NW * (gi + lane), maxp - 1)];
        const int page = __builtin_amdgcn_readlane(pages, gi & 63);
        const bf16_t* kp = pool + kv_page_block(p.kv, page, 0, head) + r * MTP_HEAD_DIM + g * 8;
        kf[u][0] = *reinterpret_cast<const uint4*>(kp);
        kf[u][1] = *reinterpret_cast<const uint4*>(kp + 32);
        const bf16_t* vp = pool + kv_page_block(p.kv, page, 1, head) + 4 * g;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) vf[u][dt] = *reinterpret_cast<const uint2*>(vp + (16 * dt + r) * 16);
    };
#pragma unroll
    for (int u = 0; u < PD; ++u) load_keys(u, u);
    float4 qa[2], qb[2];
    {
        const float* qp = p.q + (size_t)(row0 + min(r, p.Q - 1)) * p.ldq + head * 64 + g * 8;
        qa[0] = *reinterpret_cast<const float4*>(qp);
        qb[0] = *reinterpret_cast<const float4*>(qp + 4);
        qa[1] = *reinterpret_cast<const float4*>(qp + 32);
        qb[1] = *reinterpret_cast<const float4*>(qp + 36);
    }
    const int nrows = p.st[b].pend_len;
    const int pos0 = p.st[b].ctx_len;
    const int kend = pos0 + nrows;
    if (nrows <= 0 || kb >= kend) return;       // uniform over the workgroup
    const int ke = min(kb + p.split_len, kend);

    bf16x8_t qf[2];
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
        qf[h2] = __builtin_bit_cast(bf16x8_t, make_uint4(pk2(qa[h2].x * 0.125f, qa[h2].y * 0.125f),
                                                         pk2(qa[h2].z * 0.125f, qa[h2].w * 0.125f),
                                                         pk2(qb[h2].x * 0.125f, qb[h2].y * 0.125f),
                                                         pk2(qb[h2].z * 0.125f, qb[h2].w * 0.125f)));

    float m_run = -INFINITY, l_run = 0.f;       // query r, this wave's keys
    f32x4_t acc[4];                             // O^T rows 16 dt + 4 g + v, query r
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) acc[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    for (int cb = kb; cb < ke; cb += CH * PD) {
#pragma unroll
      for (int u = 0; u < PD; ++u) {
        const int c0 = cb + u * CH;
        if (c0 >= ke) break;                     // uniform over the workgroup
        const uint4 k0 = kf[u][0], k1 = kf[u][1];
        uint2 v[4];
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) v[dt] = vf[u][dt];
        if (c0 + PD * CH < ke) load_keys(u, (c0 - kb) / CH + PD);   // refill this ring slot (uniform branch)
        const int wk = c0 + 16 * wave;
        f32x4_t s = f32x4_t{0.f, 0.f, 0.f, 0.f};
        s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, k0), qf[0], s, 0, 0, 0);
        s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, k1), qf[1], s, 0, 0, 0);
        float sc[4];
        float mx = -INFINITY;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int key = wk + 4 * g + e;
            const bool ok = (key < ke) && (key <= pos0 + r) && (r < nrows);
            sc[e] = ok ? s[e] : -INFINITY;
            mx = fmaxf(mx, sc[e]);
        }
        mx = xor16_max(mx);
        mx = xor32_max(mx);
        const float m_new = fmaxf(m_run, mx);
        const float scale = (m_run == -INFINITY) ? 0.f : __expf(m_run - m_new);
        float pe[4], sum = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            pe[e] = (sc[e] == -INFINITY) ? 0.f : __expf(sc[e] - m_new);
            sum += pe[e];
        }
        sum = xor16_sum(sum);
        sum = xor32_sum(sum);
        l_run = l_run * scale + sum;
        m_run = m_new;
        const s16x4_t pf = __builtin_bit_cast(s16x4_t, make_uint2(pk2(pe[0], pe[1]), pk2(pe[2], pe[3])));
        // V^T entries of keys past the context may hold anything: zero them
        const int nvalid = ke - (wk + 4 * g);
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
            acc[dt] *= scale;
            acc[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4_t, vv), pf, acc[dt], 0, 0, 0);
        }
      }
    }

    // merge the NW waves' states
    if (g == 0) s_m[wave][r] = m_run;
    __syncthreads();
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, s_m[w][r]);
    const float wsc = (m_run == -INFINITY) ? 0.f : __expf(m_run - M);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int e = 0; e < 4; ++e) s_o[(wave * 64 + 16 * dt + 4 * g + e) * 17 + r] = acc[dt][e] * wsc;
    if (g == 0) s_l[wave][r] = l_run * wsc;
    __syncthreads();
    // output: (dim, query) pairs over the workgroup's threads
    for (int idx = tid; idx < 64 * 16; idx += 64 * NW) {
        const int dim = idx >> 4, q = idx & 15;
        if (q >= nrows) continue;
        float o = 0.f, L = 0.f, Mq = -INFINITY;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            o += s_o[(w * 64 + dim) * 17 + q];
            L += s_l[w][q];
            Mq = fmaxf(Mq, s_m[w][q]);
        }
        if (p.n_splits == 1) {
            const int row = row0 + q, col = head * 64 + dim;
            p.out[p.packed ? frag_off(row, col, p.ldo) : (size_t)row * p.ldo + col] = f32_to_bf16(o / L);
        } else {
            float* e = p.part + ((size_t)(b * H + head) * p.n_splits + split) * (p.qt * PSTR) + q * PSTR;
            e[4 + dim] = o;
            if (dim == 0) {
                e[0] = Mq;
                e[1] = L;
            }
        }
    }
}

template <int NW, int PD>
static hipError_t attn_dec_go_pd(hipStream_t st, const AttnMfmaArgs& a) {
    const size_t lds = (size_t)NW * 64 * 17 * sizeof(float);
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
