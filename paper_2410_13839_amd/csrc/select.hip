// Selection kernel: EOS mask + per-head top_k, then the lattice over the
// K positions (paper Sec. 3.3, Fig. 2) and the accept rule.
//
// Every decision is made with the same float32 operations, in the same
// association, as the plain definition: e_hat = l[c] - l[c_0];
// delta_t(j) = max_i (delta_{t-1}(i) + logQ[c_{t-1,i}][c_{t,j}]) + e_hat_t(j),
// with the lowest index winning ties in top_k (token id), in the predecessor
// scan and in the final argmax (slot).  The (value, index) max-reductions use
// a total order, so the shuffle tree cannot change their result.
//
// Sampling (top_k sampling inside the lattice, Fig. 2 caption) draws the path
// from the distribution prod_t exp(e_t / tau) * prod Q(a_{t-1}, a_t) by
// forward filtering, backward sampling.  Its arithmetic is fixed so that any
// IEEE float32 implementation reproduces every draw: one rounding per
// operation (no contraction into fused multiply-adds anywhere in this file),
// sums in ascending state order, products flushed to zero below 2^-100 (no
// result depends on subnormal handling), rescaling by exact powers of two,
// and the exp evaluation of `smp_exp`.
#include <limits.h>
#include <math.h>

#include "common.h"
#include "launch.h"
#include "wave.h"

#pragma clang fp contract(off)

namespace mtp {

namespace {
constexpr int PER_LANE = 17;   // ceil(1025 / 64): logits held per lane

__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
    return (va > vb) | ((va == vb) & (ia < ib));
}

// Philox4x64-10 (Salmon, Moraes, Dror and Shaw, SC 2011): per round, words 0
// and 2 are multiplied by the two round multipliers into 128-bit products and
// the block becomes (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0); the key then
// advances by the Weyl increments (64-bit golden ratio and sqrt(3) - 1).
__device__ __forceinline__ void philox4x64_10(uint64_t& c0, uint64_t& c1, uint64_t& c2, uint64_t& c3,
                                              uint64_t k0, uint64_t k1) {
    constexpr uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    constexpr uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t lo0 = M0 * c0, hi0 = __umul64hi(M0, c0);
        const uint64_t lo1 = M1 * c2, hi1 = __umul64hi(M1, c2);
        c0 = hi1 ^ c1 ^ k0;
        c1 = lo1;
        c2 = hi0 ^ c3 ^ k1;
        c3 = lo0;
        k0 += W0;
        k1 += W1;
    }
}

// e^x in float32 for x <= 0: x = n ln2 + r with n = rint(x log2(e)); ln 2 is
// split into a head with 16 significant bits (n * head is exact for |n| <
// 128) and a float32 tail; e^r by its Taylor series to degree 7 in Horner
// form (|r| <= ln2/2, truncation below 2^-27); then the exact scaling by 2^n.
// 0 below -64 (e^-64 ~ 2^-92) and for -inf.
__device__ __forceinline__ float smp_exp(float x) {
    if (!(x >= -64.0f)) return 0.f;
    const float n = rintf(x * __int_as_float(0x3fb8aa3b));              // log2(e)
    const float r = (x - n * __int_as_float(0x3f317200)) - n * __int_as_float(0x35bfbe8e);
    float p = 1.0f / 5040.0f;
    p = p * r + 1.0f / 720.0f;
    p = p * r + 1.0f / 120.0f;
    p = p * r + 1.0f / 24.0f;
    p = p * r + 1.0f / 6.0f;
    p = p * r + 0.5f;
    p = p * r + 1.0f;
    p = p * r + 1.0f;
    return ldexpf(p, (int)n);
}

__device__ __forceinline__ float smp_flush(float x) { return x >= 0x1p-100f ? x : 0.f; }

__device__ __forceinline__ float lane_f(float v, int i) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), i));
}

// Scale the wave's weights by the power of two that puts their maximum in
// [1/2, 1) (exact), then flush.
__device__ __forceinline__ float smp_rescale(float v) {
    const float mx = wave_max64(v);
    if (!(mx > 0.f)) return v;
    int e;
    (void)frexpf(mx, &e);
    return smp_flush(ldexpf(v, -e));
}

// Inverse-CDF draw over lanes 0..m-1 holding weights w: the first lane whose
// running sum (in lane order) exceeds u * total; the last lane of positive
// weight if none does; 0 if every weight is 0.  The result is uniform.
__device__ __forceinline__ int smp_draw(float w, float u, int m, int lane) {
    float run = 0.f, mine = 0.f;
    for (int i = 0; i < m; ++i) {
        run = run + lane_f(w, i);
        mine = (lane == i) ? run : mine;
    }
    const float thr = u * run;
    const uint64_t over = __ballot((lane < m) & (mine > thr));
    if (over) return __builtin_ctzll(over);
    const uint64_t pos = __ballot((lane < m) & (w > 0.f));
    return pos ? 63 - __builtin_clzll(pos) : 0;
}
}  // namespace

}  // namespace mtp

// ---------------------------------------------------------------- fused
// One workgroup per sequence, one wave per head: top_k of every head in
// parallel; then the lattice's emissions and transition sub-tables are
// gathered into LDS at once, and wave 0 runs the recursion, the backtrack (or
// the backward draws) and the accept rule.
//
// Two lattices (Sec. 3.3):
//   own    position t's states are head t's top_k (ordered by logit);
//   union  every position's states are the m <= K*top_k distinct tokens of
//          all heads' top_k in ascending id, scored at position t by head t
//          (e_t(c) = l_t[c] - max l_t), with the m x m sub-table of log Q.
// With `anchored`, the first position also carries the transition from the
// last emitted token.  When sampling, the gathered transitions are stored as
// probabilities (smp_exp of log Q).
namespace mtp {

namespace {
constexpr int UMAX = 64;   // union states at most (K * top_k <= 64)
}

__global__ __launch_bounds__(512) void select_fused_kernel(SelectArgs a) {
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, t = tid >> 6;
    const int K = a.K, k = a.top_k, V = a.V;
    const bool uni = a.lattice == 1;
    __shared__ int s_cand[MTP_MAX_HEADS_K][MTP_MAX_TOPK];
    __shared__ float s_ehat[MTP_MAX_HEADS_K][MTP_MAX_TOPK];
    __shared__ float s_top[MTP_MAX_HEADS_K];
    // own lattice: T[t-1][j][i] = logQ[c_{t-1,i}][c_{t,j}] (i contiguous)
    __shared__ float s_T[MTP_MAX_HEADS_K - 1][MTP_MAX_TOPK][MTP_MAX_TOPK];
    // union lattice: states, emissions [t][j], transitions [i][j] =
    // logQ[U_i][U_j] (a row per previous state, padded against bank conflicts)
    __shared__ int s_U[UMAX];
    __shared__ int s_m;
    __shared__ float s_ue[MTP_MAX_HEADS_K][UMAX];
    __shared__ float s_UT[UMAX][UMAX + 1];
    __shared__ float s_anc[UMAX];                // logQ[anchor][state of position 0]
    __shared__ int s_psi[MTP_MAX_HEADS_K][UMAX];
    __shared__ float s_alpha[MTP_MAX_HEADS_K][UMAX];   // sampling: forward weights
    const SeqState st0 = a.st[b];
    const size_t base = (size_t)b * K * k;
    const int prev = a.anchored ? st0.last_tok : -1;
    const bool smp = a.sample != 0;

    // top_k of head t (wave t)
    {
        const float* lg = a.logits + (size_t)b * a.ld_logits + (size_t)t * V;
        const bool mask_eos = (st0.gen + t) < a.eos_min;
        // unconditional loads from clamped indices (a predicated load would
        // become a branch and a full wait per element); entries past the
        // vocabulary are excluded by the idx < V test of the selection
        float v[PER_LANE];
#pragma unroll
        for (int j = 0; j < PER_LANE; ++j) v[j] = lg[min(lane + 64 * j, V - 1)];
#pragma unroll
        for (int j = 0; j < PER_LANE; ++j)
            if (lane + 64 * j == a.eos_id && mask_eos) v[j] = -INFINITY;
        // Each lane keeps the best and the second best of its values not yet
        // taken (order: value, then lower index); a round takes the wave's
        // best of the lanes' bests, and the winning lane moves its second
        // up.  A lane rescans its values only when it wins with no second
        // held, so a round costs one wave reduction instead of a scan of
        // every value.
        uint32_t taken = 0;
        float b1v, b2v;
        int b1i, b2i;
        bool have2;
        auto rescan = [&]() {
            b1v = b2v = -INFINITY;
            b1i = b2i = INT_MAX;
#pragma unroll
            for (int j = 0; j < PER_LANE; ++j) {
                const int idx = lane + 64 * j;
                const bool ok = (idx < V) & (((taken >> j) & 1u) == 0u);
                const bool n1 = ok & better(v[j], idx, b1v, b1i);
                const bool n2 = ok & !n1 & better(v[j], idx, b2v, b2i);
                b2v = n1 ? b1v : (n2 ? v[j] : b2v);
                b2i = n1 ? b1i : (n2 ? idx : b2i);
                b1v = n1 ? v[j] : b1v;
                b1i = n1 ? idx : b1i;
            }
            have2 = true;
        };
        rescan();
        float top0 = 0.f;
        int my_c = 0;
        float my_e = 0.f;
        for (int r = 0; r < k; ++r) {
            float bv = b1v;
            int bi = b1i;
            wave_argmax_uniform(bv, bi);
            if ((bi & 63) == lane) {
                taken |= 1u << (bi >> 6);
                if (have2) {
                    b1v = b2v;
                    b1i = b2i;
                    have2 = false;
                } else {
                    rescan();
                }
            }
            if (r == 0) top0 = bv;
            const float e = bv - top0;
            my_c = (lane == r) ? bi : my_c;
            my_e = (lane == r) ? e : my_e;
        }
        if (lane < k) {
            s_cand[t][lane] = my_c;
            s_ehat[t][lane] = my_e;
            a.cand[base + t * k + lane] = my_c;
            a.ehat[base + t * k + lane] = my_e;
        }
        if (lane == 0) s_top[t] = top0;
    }
    __syncthreads();

    int m = k;                                   // states per position
    if (uni) {
        // the distinct candidate ids in ascending order (wave 0): a lane keeps
        // its id if no lower lane holds the same id; its rank is the number of
        // kept ids below it
        if (t == 0) {
            const int n = K * k;
            const int id = (lane < n) ? s_cand[udiv_small(lane, k)][lane - udiv_small(lane, k) * k] : INT_MAX;
            bool dup = false;
            for (int o = 0; o < n; ++o) dup |= (__builtin_amdgcn_readlane(id, o) == id) & (o < lane);
            const bool keep = (lane < n) & !dup;
            const uint64_t kept = __ballot(keep);
            int rank = 0;
            for (int o = 0; o < n; ++o)
                rank += (int)(((kept >> o) & 1ull) != 0ull) & (__builtin_amdgcn_readlane(id, o) < id);
            if (keep) s_U[rank] = id;
            if (lane == 0) s_m = __popcll(kept);
        }
        __syncthreads();
        m = s_m;
        // emissions e_t(U_j) = l_t[U_j] - max l_t (EOS masked per head),
        // transitions T[j][i] = logQ[U_i][U_j], anchor row
        const float* lgb = a.logits + (size_t)b * a.ld_logits;
        for (int idx = tid; idx < K * m; idx += blockDim.x) {
            const int tt = udiv_small(idx, m), j = idx - tt * m;
            const int c = s_U[j];
            float l = lgb[(size_t)tt * V + c];
            if (c == a.eos_id && (st0.gen + tt) < a.eos_min) l = -INFINITY;
            s_ue[tt][j] = l - s_top[tt];
        }
        for (int idx = tid; idx < m * m; idx += blockDim.x) {
            const int i = udiv_small(idx, m), j = idx - i * m;
            const float lq = a.logq[(size_t)s_U[i] * V + s_U[j]];
            s_UT[i][j] = smp ? smp_exp(lq) : lq;
        }
        if (prev >= 0)
            for (int j = tid; j < m; j += blockDim.x) {
                const float lq = a.logq[(size_t)prev * V + s_U[j]];
                s_anc[j] = smp ? smp_exp(lq) : lq;
            }
    } else {
        const int kk = k * k;
        for (int idx = tid; idx < (K - 1) * kk; idx += blockDim.x) {
            const int t1 = udiv_small(idx, kk), rem = idx - t1 * kk;
            const int i = udiv_small(rem, k), j = rem - i * k;
            const float lq = a.logq[(size_t)s_cand[t1][i] * V + s_cand[t1 + 1][j]];
            s_T[t1][j][i] = smp ? smp_exp(lq) : lq;
        }
        if (prev >= 0)
            for (int j = tid; j < k; j += blockDim.x) {
                const float lq = a.logq[(size_t)prev * V + s_cand[0][j]];
                s_anc[j] = smp ? smp_exp(lq) : lq;
            }
    }
    __syncthreads();
    if (t != 0) return;

    // Wave 0: lane j holds state j; the other states' values come from
    // v_readlane with the (uniform) loop index, so a position costs m
    // operations in registers plus one LDS read of transitions per lane.
    const int j = lane;
    const int jc = j < m ? j : 0;
    float* out_delta = uni ? a.u_delta + (size_t)b * MTP_MAX_HEADS_K * UMAX : a.delta + base;
    int32_t* out_psi = uni ? a.u_psi + (size_t)b * MTP_MAX_HEADS_K * UMAX : a.psi + base;
    float* out_ue = a.u_ehat + (size_t)b * MTP_MAX_HEADS_K * UMAX;
    const int ostride = uni ? UMAX : k;
    // transitions into state jc of position tt from state i of position tt-1
    auto trow = [&](int tt) -> const float* { return uni ? &s_UT[0][jc] : &s_T[tt - 1][jc][0]; };
    const int tstep = uni ? UMAX + 1 : 1;
    auto emis = [&](int tt) -> float { return uni ? s_ue[tt][jc] : s_ehat[tt][jc]; };
    int my_slot = 0, my_tok = 0;

    if (!smp) {
        // Viterbi
        const float e0 = emis(0);
        float delta = (j < m) ? (prev >= 0 ? s_anc[jc] + e0 : e0) : -INFINITY;
        if (j < m) {
            out_delta[j] = delta;
            out_psi[j] = 0;
            if (uni) out_ue[j] = e0;
        }
        for (int tt = 1; tt < K; ++tt) {
            const float* T = trow(tt);
            float best = 0.f;
            int arg = 0;
            // predecessors in chunks of 8: the chunk's transition entries are
            // read from LDS together (one wait), then scanned in ascending i
            for (int i0 = 0; i0 < m; i0 += 8) {
                float tv[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) tv[u] = T[min(i0 + u, m - 1) * tstep];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int i = i0 + u;
                    if (i < m) {                                  // uniform
                        const float sc = lane_f(delta, i) + tv[u];
                        if (i == 0 || sc > best) {
                            best = sc;
                            arg = i;
                        }
                    }
                }
            }
            const float et = emis(tt);
            delta = (j < m) ? best + et : -INFINITY;
            if (j < m) {
                s_psi[tt][j] = arg;
                out_delta[tt * ostride + j] = delta;
                out_psi[tt * ostride + j] = arg;
                if (uni) out_ue[tt * UMAX + j] = et;
            }
        }
        float bestd = (j < m) ? delta : -INFINITY;
        int last = (j < m) ? j : UMAX + j;
        wave_argmax_uniform(bestd, last);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_wave_barrier();

        // backtrack with uniform state indices (state_{t-1} = psi_t(state_t));
        // lane t keeps position t
        int cur = last;
        for (int tt = K - 1; tt >= 0; --tt) {
            const int tok = uni ? s_U[cur] : s_cand[tt][cur];
            if (lane == tt) {
                my_slot = cur;
                my_tok = tok;
            }
            if (tt > 0) cur = s_psi[tt][cur];
        }
    } else {
        // Forward filtering, backward sampling.  Uniforms: lane r < K takes
        // word r % 4 of the Philox block at counter (generated count, sequence,
        // r / 4, 0), key (seed, 0); draw r decides position K-1-r.
        const float inv_tau = a.smp->inv_tau;
        float u;
        {
            uint64_t c0 = (uint64_t)st0.gen, c1 = (uint64_t)b, c2 = (uint64_t)(lane >> 2), c3 = 0;
            philox4x64_10(c0, c1, c2, c3, a.smp->seed, 0);
            const int wsel = lane & 3;
            const uint64_t x = wsel == 0 ? c0 : wsel == 1 ? c1 : wsel == 2 ? c2 : c3;
            u = (float)(uint32_t)(x >> 40) * 0x1p-24f;
        }
        if (lane < K) a.smp_u[(size_t)b * MTP_MAX_HEADS_K + lane] = u;

        const float e0 = emis(0);
        float alpha = (j < m) ? smp_exp(e0 * inv_tau) : 0.f;
        if (prev >= 0) alpha = (j < m) ? smp_flush(alpha * s_anc[jc]) : 0.f;
        alpha = smp_rescale(alpha);
        s_alpha[0][lane] = alpha;
        if (j < m) {
            out_delta[j] = alpha;
            out_psi[j] = -1;
            if (uni) out_ue[j] = e0;
        }
        for (int tt = 1; tt < K; ++tt) {
            const float* T = trow(tt);
            float sum = 0.f;
            for (int i0 = 0; i0 < m; i0 += 8) {
                float tv[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) tv[u] = T[min(i0 + u, m - 1) * tstep];
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (i0 + u < m) sum = sum + smp_flush(lane_f(alpha, i0 + u) * tv[u]);   // ascending i
            }
            const float et = emis(tt);
            alpha = (j < m) ? smp_flush(smp_exp(et * inv_tau) * sum) : 0.f;
            alpha = smp_rescale(alpha);
            s_alpha[tt][lane] = alpha;
            if (j < m) {
                out_delta[tt * ostride + j] = alpha;
                out_psi[tt * ostride + j] = -1;
                if (uni) out_ue[tt * UMAX + j] = et;
            }
        }
        // backward: position K-1 from alpha_{K-1}; position tt from
        // alpha_tt(i) * Q(state i, the state drawn at tt + 1)
        int cur = smp_draw(alpha, lane_f(u, 0), m, lane);
        if (lane == K - 1) {
            my_slot = cur;
            my_tok = uni ? s_U[cur] : s_cand[K - 1][cur];
        }
        for (int tt = K - 2; tt >= 0; --tt) {
            const float g = uni ? s_UT[jc][cur] : s_T[tt][cur][jc];
            const float w = (j < m) ? smp_flush(s_alpha[tt][jc] * g) : 0.f;
            cur = smp_draw(w, lane_f(u, K - 1 - tt), m, lane);
            if (lane == tt) {
                my_slot = cur;
                my_tok = uni ? s_U[cur] : s_cand[tt][cur];
            }
        }
    }
    if (uni) {
        if (lane < m) a.u_states[(size_t)b * UMAX + lane] = s_U[lane];
        if (lane == 0) a.u_m[b] = m;
    }
    // accept: the first min(K, budget) tokens, cut after the first EOS
    const SeqState s0 = st0;
    int n = 0;
    bool done = s0.done != 0;
    if (!done) {
        n = min(K, a.max_new - s0.gen);
        const uint64_t eos_lanes = __ballot(lane < n && my_tok == a.eos_id);
        if (eos_lanes) {
            n = __builtin_ctzll(eos_lanes) + 1;
            done = true;
        }
        if (s0.gen + n >= a.max_new) done = true;
    }
    const int last_tok = __builtin_amdgcn_readlane(my_tok, max(n - 1, 0));
    if (lane < K) {
        a.slots[(size_t)b * K + lane] = my_slot;
        a.out_tokens[(size_t)b * K + lane] = (lane < n) ? my_tok : -1;
    }
    if (lane < n) {
        a.hist[(size_t)b * a.hist_ld + s0.gen + lane] = my_tok;
        a.st[b].pend_ids[lane] = my_tok;
    }
    if (lane == 0) {
        a.out_count[b] = n;
        SeqState* sp = a.st + b;
        sp->ctx_len = s0.ctx_len + s0.pend_len;
        sp->gen = s0.gen + n;
        sp->done = done ? 1 : 0;
        sp->pend_len = done ? 0 : n;
        sp->steps = s0.steps + 1;
        if (n > 0) sp->last_tok = last_tok;
    }
}

hipError_t select_fused(hipStream_t st, const SelectArgs& a) {
    hipLaunchKernelGGL(select_fused_kernel, dim3(a.B), dim3(64 * a.K), 0, st, a);
    return hipGetLastError();
}

}  // namespace mtp
