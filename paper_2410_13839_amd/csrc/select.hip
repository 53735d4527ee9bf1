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
// parallel, then all (K-1) x top_k x top_k transition entries are gathered
// into LDS at once, then wave 0 runs the recursion, the backtrack and the
// accept rule.  Same arithmetic and tie rules as the two kernels above.
namespace mtp {

__global__ __launch_bounds__(512) void select_fused_kernel(SelectArgs a) {
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, t = tid >> 6;
    const int K = a.K, k = a.top_k, V = a.V;
    __shared__ int s_cand[MTP_MAX_HEADS_K][MTP_MAX_TOPK];
    __shared__ float s_ehat[MTP_MAX_HEADS_K][MTP_MAX_TOPK];
    __shared__ float s_T[MTP_MAX_HEADS_K - 1][MTP_MAX_TOPK][MTP_MAX_TOPK];   // [t-1][j][i] (i contiguous)
    __shared__ int s_psi[MTP_MAX_HEADS_K][MTP_MAX_TOPK];
    __shared__ float s_delta[MTP_MAX_TOPK];
    const SeqState st0 = a.st[b];
    const size_t base = (size_t)b * K * k;

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
    }
    __syncthreads();
    // transition sub-tables T[t-1][j][i] = logQ[c_{t-1,i}][c_{t,j}] (stored
    // with i contiguous: the recursion reads one row per slot j)
    const int kk = k * k;
    for (int idx = tid; idx < (K - 1) * kk; idx += blockDim.x) {
        const int t1 = idx / kk, rem = idx - t1 * kk;
        const int i = rem / k, j = rem - i * k;
        s_T[t1][j][i] = a.logq[(size_t)s_cand[t1][i] * V + s_cand[t1 + 1][j]];
    }
    __syncthreads();
    if (t != 0) return;

    // Viterbi on wave 0: lane j holds slot j's score; the scores of the other
    // slots come from v_readlane with the (uniform) loop index, so a step is k
    // adds and compares in registers plus one LDS row of transitions.
    const int j = lane;
    const int jc = j < k ? j : 0;
    float delta = (j < k) ? s_ehat[0][jc] : -INFINITY;
    if (j < k) {
        a.delta[base + j] = delta;
        a.psi[base + j] = 0;
    }
    for (int tt = 1; tt < K; ++tt) {
        const float* Trow = &s_T[tt - 1][jc][0];
        float best = 0.f;
        int arg = 0;
        for (int i = 0; i < k; ++i) {
            const float di = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(delta), i));
            const float sc = di + Trow[i];
            if (i == 0 || sc > best) {
                best = sc;
                arg = i;
            }
        }
        delta = (j < k) ? best + s_ehat[tt][jc] : -INFINITY;
        if (j < k) {
            s_psi[tt][j] = arg;
            a.delta[base + tt * k + j] = delta;
            a.psi[base + tt * k + j] = arg;
        }
    }
    float bestd = (j < k) ? delta : -INFINITY;
    int last = (j < k) ? j : MTP_MAX_TOPK + j;
    wave_argmax_uniform(bestd, last);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();

    // backtrack with uniform slot indices (slot_{t-1} = psi_t(slot_t));
    // lane t keeps position t
    int my_slot = 0, my_tok = 0;
    int cur = last;
    for (int tt = K - 1; tt >= 0; --tt) {
        const int tok = s_cand[tt][cur];
        if (lane == tt) {
            my_slot = cur;
            my_tok = tok;
        }
        if (tt > 0) cur = s_psi[tt][cur];
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
    }
}

hipError_t select_fused(hipStream_t st, const SelectArgs& a) {
    hipLaunchKernelGGL(select_fused_kernel, dim3(a.B), dim3(64 * a.K), 0, st, a);
    return hipGetLastError();
}

}  // namespace mtp
