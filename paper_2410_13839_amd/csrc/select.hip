// Selection kernels: EOS mask + per-head top_k, then the Viterbi lattice and
// the accept rule (paper Sec. 3.3, Fig. 2).
//
// Every decision is made with the same float32 operations, in the same
// association, as the plain definition: e_hat = l[c] - l[c_0];
// delta_t(j) = max_i (delta_{t-1}(i) + logQ[c_{t-1,i}][c_{t,j}]) + e_hat_t(j),
// with the lowest index winning ties in top_k (token id), in the predecessor
// scan and in the final argmax (slot).  The (value, index) max-reductions use
// a total order, so the shuffle tree cannot change their result.
#include <limits.h>
#include <math.h>

#include "common.h"
#include "launch.h"
#include "wave.h"

namespace mtp {

namespace {
constexpr int PER_LANE = 17;   // ceil(1025 / 64): logits held per lane

__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
    return (va > vb) | ((va == vb) & (ia < ib));
}
}  // namespace

// One wavefront per (sequence, head).
__global__ __launch_bounds__(64) void topk_kernel(SelectArgs a) {
    const int bt = blockIdx.x;
    const int b = bt / a.K, t = bt - b * a.K;
    const int lane = threadIdx.x;
    const float* lg = a.logits + (size_t)b * a.ld_logits + (size_t)t * a.V;
    const bool mask_eos = (a.st[b].gen + t) < a.eos_min;
    float v[PER_LANE];
#pragma unroll
    for (int j = 0; j < PER_LANE; ++j) {
        const int idx = lane + 64 * j;
        float x = (idx < a.V) ? lg[idx] : -INFINITY;
        if (idx == a.eos_id && mask_eos) x = -INFINITY;
        v[j] = x;
    }
    uint32_t taken = 0;
    float top0 = 0.f;
    const size_t out = ((size_t)b * a.K + t) * a.top_k;
    for (int r = 0; r < a.top_k; ++r) {
        float bv = -INFINITY;
        int bi = INT_MAX;
#pragma unroll
        for (int j = 0; j < PER_LANE; ++j) {
            const int idx = lane + 64 * j;
            if (idx < a.V && !((taken >> j) & 1u) && better(v[j], idx, bv, bi)) {
                bv = v[j];
                bi = idx;
            }
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            const float ov = __shfl_xor(bv, o);
            const int oi = __shfl_xor(bi, o);
            if (better(ov, oi, bv, bi)) {
                bv = ov;
                bi = oi;
            }
        }
        if ((bi & 63) == lane) taken |= 1u << (bi >> 6);
        if (r == 0) top0 = bv;
        if (lane == 0) {
            a.cand[out + r] = bi;
            a.ehat[out + r] = bv - top0;
        }
    }
}

// One wavefront per sequence: lane j owns candidate slot j.
__global__ __launch_bounds__(64) void viterbi_accept_kernel(SelectArgs a) {
    const int b = blockIdx.x, j = threadIdx.x;
    const int K = a.K, k = a.top_k, V = a.V;
    __shared__ int s_psi[MTP_MAX_HEADS_K][MTP_MAX_TOPK];
    const size_t base = (size_t)b * K * k;
    const int32_t* cand = a.cand + base;
    const float* ehat = a.ehat + base;

    float delta = (j < k) ? ehat[j] : -INFINITY;
    if (j < k) {
        a.delta[base + j] = delta;
        a.psi[base + j] = 0;
        s_psi[0][j] = 0;
    }
    for (int t = 1; t < K; ++t) {
        const int cj = (j < k) ? cand[t * k + j] : 0;
        float best = 0.f;
        int arg = 0;
        for (int i = 0; i < k; ++i) {
            const float di = __shfl(delta, i);
            const int ci = cand[(t - 1) * k + i];
            const float s = di + a.logq[(size_t)ci * V + cj];
            if (i == 0 || s > best) {
                best = s;
                arg = i;
            }
        }
        delta = (j < k) ? best + ehat[t * k + j] : -INFINITY;
        if (j < k) {
            a.delta[base + t * k + j] = delta;
            a.psi[base + t * k + j] = arg;
            s_psi[t][j] = arg;
        }
    }
    int last = 0;
    float bestd = __shfl(delta, 0);
    for (int i = 1; i < k; ++i) {
        const float di = __shfl(delta, i);
        if (di > bestd) {
            bestd = di;
            last = i;
        }
    }
    __syncthreads();
    if (j != 0) return;

    int slots[MTP_MAX_HEADS_K], toks[MTP_MAX_HEADS_K];
    slots[K - 1] = last;
    for (int t = K - 1; t > 0; --t) slots[t - 1] = s_psi[t][slots[t]];
    for (int t = 0; t < K; ++t) {
        toks[t] = cand[t * k + slots[t]];
        a.slots[(size_t)b * K + t] = slots[t];
    }

    SeqState s = a.st[b];
    int n = 0;
    bool done = s.done != 0;
    if (!done) {
        n = min(K, a.max_new - s.gen);
        for (int p = 0; p < n; ++p) {
            if (toks[p] == a.eos_id) {
                n = p + 1;
                done = true;
                break;
            }
        }
        if (s.gen + n >= a.max_new) done = true;
    }
    for (int t = 0; t < K; ++t) a.out_tokens[(size_t)b * K + t] = (t < n) ? toks[t] : -1;
    a.out_count[b] = n;
    for (int t = 0; t < n; ++t) a.hist[(size_t)b * a.hist_ld + s.gen + t] = toks[t];
    s.ctx_len += s.pend_len;
    s.gen += n;
    s.done = done ? 1 : 0;
    s.pend_len = done ? 0 : n;
    for (int t = 0; t < n && t < MTP_MAX_HEADS_K; ++t) s.pend_ids[t] = toks[t];
    s.steps += 1;
    a.st[b] = s;
}

hipError_t topk(hipStream_t st, const SelectArgs& a) {
    hipLaunchKernelGGL(topk_kernel, dim3(a.B * a.K), dim3(64), 0, st, a);
    return hipGetLastError();
}

hipError_t viterbi_accept(hipStream_t st, const SelectArgs& a) {
    hipLaunchKernelGGL(viterbi_accept_kernel, dim3(a.B), dim3(64), 0, st, a);
    return hipGetLastError();
}

}  // namespace mtp

// ---------------------------------------------------------------- fused
// One workgroup per sequence, one wave per head: top_k of every head in
// parallel; then the lattice's emissions and transition sub-tables are
// gathered into LDS at once, and wave 0 runs the recursion, the backtrack and
// the accept rule.  Same arithmetic and tie rules as the two kernels above.
//
// Two lattices (Sec. 3.3):
//   own    position t's states are head t's top_k (ordered by logit);
//   union  every position's states are the m <= K*top_k distinct tokens of
//          all heads' top_k in ascending id, scored at position t by head t
//          (e_t(c) = l_t[c] - max l_t), with the m x m sub-table of log Q.
// With `anchored`, delta_0 also carries logQ[last emitted token][c].
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
    // union lattice: states, emissions [t][j], transitions [j][i]
    __shared__ int s_U[UMAX];
    __shared__ int s_m;
    __shared__ float s_ue[MTP_MAX_HEADS_K][UMAX];
    __shared__ float s_UT[UMAX][UMAX];
    __shared__ float s_anc[UMAX];                // logQ[anchor][state of position 0]
    __shared__ int s_psi[MTP_MAX_HEADS_K][UMAX];
    const SeqState st0 = a.st[b];
    const size_t base = (size_t)b * K * k;
    const int prev = a.anchored ? st0.last_tok : -1;

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
        uint32_t taken = 0;
        float top0 = 0.f;
        int my_c = 0;
        float my_e = 0.f;
        for (int r = 0; r < k; ++r) {
            float bv = -INFINITY;
            int bi = INT_MAX;
#pragma unroll
            for (int j = 0; j < PER_LANE; ++j) {
                const int idx = lane + 64 * j;
                const bool ok = (idx < V) & (((taken >> j) & 1u) == 0u);
                const bool bt = ok & better(v[j], idx, bv, bi);
                bv = bt ? v[j] : bv;
                bi = bt ? idx : bi;
            }
            wave_argmax_uniform(bv, bi);
            taken |= ((bi & 63) == lane) ? (1u << (bi >> 6)) : 0u;
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
            const int j = udiv_small(idx, m), i = idx - j * m;
            s_UT[j][i] = a.logq[(size_t)s_U[i] * V + s_U[j]];
        }
        if (prev >= 0)
            for (int j = tid; j < m; j += blockDim.x) s_anc[j] = a.logq[(size_t)prev * V + s_U[j]];
    } else {
        const int kk = k * k;
        for (int idx = tid; idx < (K - 1) * kk; idx += blockDim.x) {
            const int t1 = udiv_small(idx, kk), rem = idx - t1 * kk;
            const int i = udiv_small(rem, k), j = rem - i * k;
            s_T[t1][j][i] = a.logq[(size_t)s_cand[t1][i] * V + s_cand[t1 + 1][j]];
        }
        if (prev >= 0)
            for (int j = tid; j < k; j += blockDim.x) s_anc[j] = a.logq[(size_t)prev * V + s_cand[0][j]];
    }
    __syncthreads();
    if (t != 0) return;

    // Viterbi on wave 0: lane j holds state j's score; the scores of the other
    // states come from v_readlane with the (uniform) loop index, so a step is
    // m adds and compares in registers plus one LDS row of transitions.
    const int j = lane;
    const int jc = j < m ? j : 0;
    const int ld = uni ? UMAX : MTP_MAX_TOPK;    // row strides of the emission / delta outputs
    float e0 = uni ? s_ue[0][jc] : s_ehat[0][jc];
    float delta = (j < m) ? (prev >= 0 ? s_anc[jc] + e0 : e0) : -INFINITY;
    float* out_delta = uni ? a.u_delta + (size_t)b * MTP_MAX_HEADS_K * UMAX : a.delta + base;
    int32_t* out_psi = uni ? a.u_psi + (size_t)b * MTP_MAX_HEADS_K * UMAX : a.psi + base;
    const int ostride = uni ? UMAX : k;
    if (j < m) {
        out_delta[j] = delta;
        out_psi[j] = 0;
        if (uni) a.u_ehat[(size_t)b * MTP_MAX_HEADS_K * UMAX + j] = e0;
    }
    for (int tt = 1; tt < K; ++tt) {
        const float* Trow = uni ? &s_UT[jc][0] : &s_T[tt - 1][jc][0];
        float best = 0.f;
        int arg = 0;
        for (int i = 0; i < m; ++i) {
            const float di = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(delta), i));
            const float sc = di + Trow[i];
            if (i == 0 || sc > best) {
                best = sc;
                arg = i;
            }
        }
        const float et = uni ? s_ue[tt][jc] : s_ehat[tt][jc];
        delta = (j < m) ? best + et : -INFINITY;
        if (j < m) {
            s_psi[tt][j] = arg;
            out_delta[tt * ostride + j] = delta;
            out_psi[tt * ostride + j] = arg;
            if (uni) a.u_ehat[(size_t)b * MTP_MAX_HEADS_K * UMAX + tt * UMAX + j] = et;
        }
    }
    (void)ld;
    float bestd = (j < m) ? delta : -INFINITY;
    int last = (j < m) ? j : UMAX + j;
    wave_argmax_uniform(bestd, last);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();

    // backtrack with uniform state indices (state_{t-1} = psi_t(state_t));
    // lane t keeps position t
    int my_slot = 0, my_tok = 0;
    int cur = last;
    for (int tt = K - 1; tt >= 0; --tt) {
        const int tok = uni ? s_U[cur] : s_cand[tt][cur];
        if (lane == tt) {
            my_slot = cur;
            my_tok = tok;
        }
        if (tt > 0) cur = s_psi[tt][cur];
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
