// Decode attention over a bf16 cache with 16-key pages, as a workgroup body:
// one workgroup per (sequence, head, key split), NW waves.  Shared by the
// stand-alone decode attention kernel (attn_mfma.hip) and the attention
// workgroups of the fused decode front (gemv.hip), which start before their
// head's queries exist and wait for them (FRONT).
//
// Within a 16*NW-key chunk each wave owns 16 consecutive keys and keeps its
// own online-softmax state (running max, sum, O^T accumulators) across the
// chunks of its split, so the chunk loop has no barrier; the NW states are
// merged through LDS once at the end.
//   S^T[key][q] = K[key][:] . Q[q][:] / 8    v_mfma_f32_16x16x32_bf16 (2 k-steps)
//   O^T[dim][q] += V^T[dim][key] P^T[key][q] v_mfma_f32_16x16x16_bf16: the B
//                                             operand (4 keys x query per lane)
//                                             is exactly the lane's S^T result
//                                             after exp, so P never leaves registers
// A CU streams only ~25 GB/s from HBM, so short splits spread a small batch's
// keys over many CUs; long splits use up to 16 waves.  With long splits each
// wave keeps PD of its 16-key groups in flight (a register ring, rotated by
// unrolling), so a CU's outstanding KV reads grow with PD instead of stalling
// on one round trip per chunk.
#pragma once

#include <math.h>

#include "common.h"
#include "launch.h"
#include "wave.h"

namespace mtp {

namespace attn_dec_detail {

constexpr int PSTR = 68;        // floats per partial row: max, sum, 2 pad, 64 outputs
constexpr int CPOL_SC1 = 16;    // buffer-load cache policy: device scope (misses the CU's L1)

typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pk2(float a, float b) {
    return bf16x2_bits(a, b);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// The QKV tile that stores column block w (0..11: 4 of Q, then K, then V)
// of head `head`.
__device__ __forceinline__ int front_tile(const FrontSync& fs, int head, int w) {
    return (w >> 2) * fs.tiles_per_mat + 4 * head + (w & 3);
}

// Wait until the 12 QKV tiles of `head` have stored their columns.  The
// producers and this workgroup run on one XCD (the front's workgroup
// mapping), so a plain store of theirs is visible in the XCD's L2, which a
// device-scope load reads (a plain load could hit a stale line in this CU's
// L1).  Every wave polls for itself, at most fs.spin times; a wait that
// runs out is counted (and the body goes on with whatever it then reads).
__device__ __forceinline__ void front_wait(const FrontSync& fs, int head, int lane) {
    const int t = front_tile(fs, head, min(lane, 11));
    bool ready = false;
    for (int s = 0; s < fs.spin; ++s) {
        const unsigned f = __hip_atomic_load(&fs.flags[t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (__all(f != 0u)) { ready = true; break; }
        __builtin_amdgcn_s_sleep(2);
    }
    if (!ready && lane == 0) atomicAdd(fs.err, 1u);
}

}  // namespace attn_dec_detail

// QN: query rows per sequence the LDS merge holds (the pending chunk, <= 16).
// FRONT: the head's queries (p.qh: bf16, already scaled by 1/8) and the
// pending chunk's own keys and values are being written by the same launch:
// the body prefetches the cached keys, waits for the head's QKV tiles (fs),
// then loads the queries and reloads the key groups that hold pending keys
// through the L2.
template <int NW, int PD, int QN, bool FRONT>
__device__ __forceinline__ void attn_dec_body(const AttnMfmaArgs& p, int b, int head, int split, int H,
                                              const FrontSync& fs) {
    using namespace attn_dec_detail;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, g = lane >> 4;
    extern __shared__ __attribute__((aligned(16))) float s_acc[];   // [NW waves][QN rows][64 dims]: the waves' O^T parts
    __shared__ float2 s_ml[QN][NW];              // the waves' (running max, sum) per row
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
    if constexpr (FRONT) {
        // one attention workgroup per head clears the head's flags of the
        // next launch's set (on this XCD, like every access to them)
        if (b == 0 && split == 0 && tid < 12) fs.next_flags[front_tile(fs, head, tid)] = 0u;
    }
    const int maxp = p.kv.max_pages_per_seq;
    const int32_t* btab = p.kv.block_table + (size_t)b * maxp;
    const int pg0 = (kb >> 4) + wave;
    int pages = btab[min(pg0 + NW * lane, maxp - 1)];
    uint4 kf[PD][2];
    uint2 vf[PD][4];
    // fresh (uniform): through the L2 (FRONT, after the hand-off)
    auto load_keys = [&](int u, int gi, bool fresh) {   // gi: this wave's group index (uniform)
        if ((gi & 63) == 0 && gi > 0) pages = btab[min(pg0 + NW * (gi + lane), maxp - 1)];
        const int page = __builtin_amdgcn_readlane(pages, gi & 63);
        const bf16_t* kp = pool + kv_page_block(p.kv, page, 0, head);
        const bf16_t* vp = pool + kv_page_block(p.kv, page, 1, head);
        if (FRONT && fresh) {
            const auto rk = rsrc(kp, 16 * MTP_HEAD_DIM * 2), rv = rsrc(vp, 16 * MTP_HEAD_DIM * 2);
            const int ko = (r * MTP_HEAD_DIM + g * 8) * 2;
            kf[u][0] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rk, ko, 0, CPOL_SC1));
            kf[u][1] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rk, ko + 64, 0, CPOL_SC1));
#pragma unroll
            for (int dt = 0; dt < 4; ++dt)
                vf[u][dt] = __builtin_bit_cast(
                    uint2, __builtin_amdgcn_raw_buffer_load_b64(rv, ((16 * dt + r) * 16 + 4 * g) * 2, 0, CPOL_SC1));
        } else {
            kp += r * MTP_HEAD_DIM + g * 8;
            kf[u][0] = *reinterpret_cast<const uint4*>(kp);
            kf[u][1] = *reinterpret_cast<const uint4*>(kp + 32);
            vp += 4 * g;
#pragma unroll
            for (int dt = 0; dt < 4; ++dt) vf[u][dt] = *reinterpret_cast<const uint2*>(vp + (16 * dt + r) * 16);
        }
    };
#pragma unroll
    for (int u = 0; u < PD; ++u) load_keys(u, u, false);
    // the queries of rows r (clamped to the chunk), dims 8 g .. 8 g + 7 of
    // each 32-wide k step, as bf16 after the 1/8 scale
    bf16x8_t qf[2];
    const int qrow = row0 + min(r, p.Q - 1);
    float4 qa[2], qb[2];
    const float* qp = p.q + (size_t)qrow * p.ldq + head * 64 + g * 8;
    if constexpr (!FRONT) {
        qa[0] = *reinterpret_cast<const float4*>(qp);
        qb[0] = *reinterpret_cast<const float4*>(qp + 4);
        qa[1] = *reinterpret_cast<const float4*>(qp + 32);
        qb[1] = *reinterpret_cast<const float4*>(qp + 36);
    }
    const int nrows = p.st[b].pend_len;
    const int pos0 = p.st[b].ctx_len;
    const int kend = pos0 + nrows;
    if (nrows <= 0 || kb >= kend) return;      // uniform over the workgroup
    const int ke = min(kb + p.split_len, kend);
    if constexpr (FRONT) {
        front_wait(fs, head, lane);
        // the queries, and every group in the ring that holds a pending key
        // (written by this launch's K / V tiles)
        const auto rq = rsrc(p.qh, (uint32_t)((size_t)(row0 + p.Q) * p.ldq * 2));
        const int qo = (qrow * p.ldq + head * 64 + g * 8) * 2;
        qf[0] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(rq, qo, 0, CPOL_SC1));
        qf[1] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(rq, qo + 64, 0, CPOL_SC1));
#pragma unroll
        for (int u = 0; u < PD; ++u) {
            const int gk = kb + u * CH + 16 * wave;
            if (gk + 16 > pos0 && gk < ke) load_keys(u, u, true);
        }
    } else {
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2)
            qf[h2] = __builtin_bit_cast(bf16x8_t, make_uint4(pk2(qa[h2].x * 0.125f, qa[h2].y * 0.125f),
                                                             pk2(qa[h2].z * 0.125f, qa[h2].w * 0.125f),
                                                             pk2(qb[h2].x * 0.125f, qb[h2].y * 0.125f),
                                                             pk2(qb[h2].z * 0.125f, qb[h2].w * 0.125f)));
    }

    float m_run = -INFINITY, l_run = 0.f;       // query r, this wave's keys
    f32x4_t acc[4];                             // O^T rows 16 dt + 4 g + v, query r
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) acc[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    for (int cb = kb; cb < ke; cb += CH * PD) {
#pragma unroll
      for (int u = 0; u < PD; ++u) {
        const int c0 = cb + u * CH;
        if (c0 >= ke) break;                     // uniform over the workgroup
        const int wk = c0 + 16 * wave;
        if (wk >= ke) break;                     // this wave's keys end here (uniform over the wave)
        const uint4 k0 = kf[u][0], k1 = kf[u][1];
        uint2 v[4];
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) v[dt] = vf[u][dt];
        if (c0 + PD * CH < ke) load_keys(u, (c0 - kb) / CH + PD, FRONT);   // refill this ring slot (uniform branch)
        f32x4_t s = f32x4_t{0.f, 0.f, 0.f, 0.f};
        s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, k0), qf[0], s, 0, 0, 0);
        s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, k1), qf[1], s, 0, 0, 0);
        // a group whose keys all precede the chunk and the split's end needs
        // no mask (uniform over the wave); rows past the chunk are never
        // stored and reduce only among themselves (the max and sum below
        // combine lanes of one row), so they need none either
        const bool edge = wk + 16 > min(ke, pos0 + 1);
        float sc[4];
        float mx;
        if (edge) {
            mx = -INFINITY;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int key = wk + 4 * g + e;
                sc[e] = (key < ke && key <= pos0 + r) ? s[e] : -INFINITY;
                mx = fmaxf(mx, sc[e]);
            }
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) sc[e] = s[e];
            mx = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
        }
        mx = xor16_max(mx);
        mx = xor32_max(mx);
        // the wave's first group: nothing accumulated yet (uniform)
        const bool first = c0 == kb;
        const float m_new = fmaxf(m_run, mx);
        const float scale = (first || m_run == -INFINITY) ? 0.f : __expf(m_run - m_new);
        float pe[4], sum = 0.f;
        if (edge) {
#pragma unroll
            for (int e = 0; e < 4; ++e) pe[e] = (sc[e] == -INFINITY) ? 0.f : __expf(sc[e] - m_new);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) pe[e] = __expf(sc[e] - m_new);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) sum += pe[e];
        sum = xor16_sum(sum);
        sum = xor32_sum(sum);
        l_run = first ? sum : l_run * scale + sum;
        m_run = m_new;
        const s16x4_t pf = __builtin_bit_cast(s16x4_t, make_uint2(pk2(pe[0], pe[1]), pk2(pe[2], pe[3])));
        // V^T entries of keys past the context may hold anything: zero them
        // (only a group that reaches past the split's end holds any)
        const int nvalid = ke - (wk + 4 * g);
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) {
            uint2 vv = v[dt];
            if (wk + 16 > ke && nvalid < 4) {
                uint32_t w0 = vv.x, w1 = vv.y;
                if (nvalid <= 0) w0 = 0u;
                else if (nvalid == 1) w0 &= 0x0000FFFFu;
                if (nvalid <= 2) w1 = 0u;
                else w1 &= 0x0000FFFFu;
                vv = make_uint2(w0, w1);
            }
            if (!first) acc[dt] *= scale;
            acc[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4_t, vv), pf, acc[dt], 0, 0, 0);
        }
      }
    }

    // merge the NW waves' states in one LDS pass: every wave leaves its raw
    // state (rows < QN: the other rows are never valid), then one thread per
    // (row, 4 dims) rescales each wave's part to the common maximum and sums
    // them, in wave order
    f32x4_t* s_acc4 = reinterpret_cast<f32x4_t*>(__builtin_assume_aligned(s_acc, 16));
    if (r < QN) {
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) s_acc4[(wave * QN + r) * 16 + 4 * dt + g] = acc[dt];
        if (g == 0) s_ml[r][wave] = make_float2(m_run, l_run);
    }
    __syncthreads();
    for (int idx = tid; idx < 16 * QN; idx += 64 * NW) {
        const int q = idx >> 4, d4 = idx & 15;
        if (q >= nrows) continue;
        // every LDS read first (16-byte reads, one wait), then the arithmetic
        float2 ml[NW];
        f32x4_t av[NW];
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            ml[w] = s_ml[q][w];
            av[w] = s_acc4[(w * QN + q) * 16 + d4];
        }
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < NW; ++w) M = fmaxf(M, ml[w].x);
        f32x4_t o = f32x4_t{0.f, 0.f, 0.f, 0.f};
        float L = 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            const float wsc = (ml[w].x == -INFINITY) ? 0.f : __expf(ml[w].x - M);
            o += av[w] * wsc;
            L += ml[w].y * wsc;
        }
        const int dim = 4 * d4;
        if (p.n_splits == 1) {
            const int row = row0 + q, col = head * 64 + dim;
            const uint2 y = make_uint2(pk2(o[0] / L, o[1] / L), pk2(o[2] / L, o[3] / L));
            *reinterpret_cast<uint2*>(p.out + (p.packed ? frag_off(row, col, p.ldo) : (size_t)row * p.ldo + col)) = y;
        } else {
            float* e = p.part + ((size_t)(b * H + head) * p.n_splits + split) * (p.qt * PSTR) + q * PSTR;
            *reinterpret_cast<float4*>(e + 4 + dim) = make_float4(o[0], o[1], o[2], o[3]);
            if (d4 == 0) *reinterpret_cast<float2*>(e) = make_float2(M, L);
        }
    }
}

}  // namespace mtp
