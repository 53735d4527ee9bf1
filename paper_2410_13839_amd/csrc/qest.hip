// Transition-table estimation (paper Sec. 3.3: Q is derived from the
// training corpus): bigram counts C[prev][next] over utterances (no pair
// spans two utterances; optionally each non-empty utterance adds (last
// token, EOS)), then log Q.
//
// Device-scope atomics run at only ~27 G/s on this part whatever the address
// pattern, so one global atomic per pair (4 ms for LibriTTS' ~105 M tokens)
// is replaced by a partition of the pairs by key range and workgroup-private
// LDS histograms.  A key is prev * V + next; keys are split into buckets of
// 2^15 consecutive keys (one bucket's histogram fills 128 KB of LDS).
//
//   q_bucket_count    utterance ranges per workgroup: validate, count each
//                     range's pairs per bucket (LDS), row per workgroup;
//   q_column_scan     per bucket: exclusive scan over workgroups (the
//                     workgroups' write offsets inside the bucket), total;
//   q_bucket_plan     bucket bases, slices of at most S keys per bucket,
//                     overflow check (more pairs than tokens: nothing counted);
//   q_bucket_scatter  the same pairs again, each key written to its bucket
//                     at an LDS cursor (every range reads its tokens twice);
//   q_slice_hist      one workgroup per slice: LDS histogram of its keys,
//                     written whole to a partial row;
//   q_reduce          per key: counts += the partials of its bucket's slices.
// Only a few hundred global atomics remain (input-error tallies).  Every
// count is an integer sum, so the result does not depend on scheduling.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <mutex>

#include "../../include/mtp.h"

namespace mtp {
namespace {

constexpr int QB_LOG = 15;
constexpr uint32_t QB_BIN = 1u << QB_LOG;       // keys per bucket
constexpr int QB_MAX_NB = 2048;                 // buckets for vocab <= 8192
constexpr int QB_MAX_WG = 4096;                 // utterance-range workgroups
constexpr int QB_THREADS = 256;                 // count / scatter workgroups
constexpr int QH_THREADS = 1024;                // histogram workgroups
constexpr int QS_THREADS = 1024;                // scans

struct QPlan {
    int V, NB, NWG, upw;        // vocab, buckets, range workgroups, utterances per range
    int64_t S;                  // keys per slice
    int64_t max_slices;         // n_tokens / S + NB
};

struct QWs {
    uint32_t* wg_cnt;           // [NWG][NB] counts, then write offsets within the bucket
    uint32_t* b_cnt;            // [NB]
    uint32_t* b_base;           // [NB + 1]
    uint32_t* s_base;           // [NB + 1] first slice of each bucket
    uint32_t* ctl;              // [0] 1 when the pairs exceed the key buffer
    uint32_t* keys;             // [n_tokens]
    uint32_t* part;             // [max_slices][QB_BIN]
};

struct QArgs {
    const int32_t* tok; int64_t n_tokens;
    const int64_t* off; int64_t n_seqs;
    int eos; int count_eos;
    uint32_t* counts;
    unsigned long long* status;
    QPlan p;
    QWs w;
};

uint64_t align256(uint64_t x) { return (x + 255) & ~uint64_t(255); }

QPlan make_plan(int64_t n_tokens, int64_t n_seqs, int V) {
    QPlan p{};
    p.V = V;
    const uint64_t keys = (uint64_t)V * V;
    p.NB = (int)((keys + QB_BIN - 1) >> QB_LOG);
    int64_t nwg = (n_seqs + 15) / 16;
    p.NWG = (int)(nwg < 1 ? 1 : nwg > QB_MAX_WG ? QB_MAX_WG : nwg);
    p.upw = (int)((n_seqs + p.NWG - 1) / p.NWG);
    const int64_t s = (n_tokens + 447) / 448;
    p.S = s < 65536 ? 65536 : s;
    p.max_slices = n_tokens / p.S + p.NB;
    return p;
}

// Workspace carve-up; returns the bytes needed.
uint64_t carve(const QPlan& p, int64_t n_tokens, char* base, QWs* w) {
    uint64_t o = 0;
    auto take = [&](uint64_t bytes) { char* r = base ? base + o : nullptr; o = align256(o + bytes); return r; };
    QWs t{};
    t.wg_cnt = (uint32_t*)take((uint64_t)p.NWG * p.NB * 4);
    t.b_cnt = (uint32_t*)take((uint64_t)p.NB * 4);
    t.b_base = (uint32_t*)take((uint64_t)(p.NB + 1) * 4);
    t.s_base = (uint32_t*)take((uint64_t)(p.NB + 1) * 4);
    t.ctl = (uint32_t*)take(16);
    const int64_t cap = (n_tokens + 3) / 4 * 4;   // whole 16-byte groups for the vector loads
    t.keys = (uint32_t*)take((uint64_t)(cap > 0 ? cap : 4) * 4);
    t.part = (uint32_t*)take((uint64_t)p.max_slices * QB_BIN * 4);
    if (w) *w = t;
    return o;
}

// The pairs of workgroup `wg`'s utterance range.  The range's offsets are
// staged in LDS.  When they are valid and non-decreasing, the range is one
// contiguous span of tokens; if the span is at most QB_FLAT positions, the
// whole workgroup sweeps it in 16-byte aligned groups of four positions
// (one vector load per group, the fifth token from the next lane), and an
// LDS bitmap marks each utterance's last position, where the pair is
// (last, EOS) or none.  Otherwise each wave walks whole utterances (wave i
// takes utterances i, i+4, ...).  Positions are 32-bit (n_tokens < 2^31).
// Both passes over a range make the same choice, so they see the same pairs.
constexpr int QB_MAX_UPW = 256;
constexpr int QB_FLAT = 65536;

struct QLds {
    int64_t off[QB_MAX_UPW + 1];
    uint32_t last[QB_FLAT / 32];
};

struct QRange {
    int64_t u0, u1;
    bool staged, flat;
    int32_t S0, S1;              // the span when flat
};

__device__ __forceinline__ bool pair_key(const QArgs& a, int x, int y, uint32_t* key) {
    const uint32_t V = (uint32_t)a.p.V;
    if ((uint32_t)x >= V || (uint32_t)y >= V) return false;
    *key = (uint32_t)x * V + (uint32_t)y;
    return true;
}

// Stages the offsets, decides flat or not, builds the bitmap.  All threads
// of the workgroup call it (it synchronises).
__device__ QRange range_setup(const QArgs& a, int wg, QLds& L) {
    const int tid = threadIdx.x;
    QRange r{};
    r.u0 = (int64_t)wg * a.p.upw;
    r.u1 = r.u0 + a.p.upw < a.n_seqs ? r.u0 + a.p.upw : a.n_seqs;
    const int nu = (int)(r.u1 - r.u0);
    r.staged = a.p.upw <= QB_MAX_UPW;
    if (nu <= 0 || !r.staged) return r;            // nu: uniform; no range or too many utterances to stage
    for (int i = tid; i <= nu; i += QB_THREADS) L.off[i] = a.off[r.u0 + i];
    __syncthreads();
    bool ok = true;
    for (int i = tid; i < nu; i += QB_THREADS) ok &= L.off[i] <= L.off[i + 1];
    ok &= L.off[0] >= 0 && L.off[nu] <= a.n_tokens && L.off[nu] - L.off[0] <= QB_FLAT;
    r.flat = __syncthreads_and(ok) != 0;
    if (r.flat) {
        r.S0 = (int32_t)L.off[0];
        r.S1 = (int32_t)L.off[nu];
        for (int i = tid; i < QB_FLAT / 32; i += QB_THREADS) L.last[i] = 0u;
        __syncthreads();
        for (int i = tid; i < nu; i += QB_THREADS) {
            const int32_t e = (int32_t)L.off[i + 1];
            if (e > (int32_t)L.off[i]) atomicOr(&L.last[(e - 1 - r.S0) >> 5], 1u << ((e - 1 - r.S0) & 31));
        }
        __syncthreads();
    }
    return r;
}

// The four positions g .. g+3 (g a multiple of 4; every lane of the wave
// calls it): key[j] and bit j of the returned mask for each counted pair,
// *bad += the pairs with an id outside [0, V).
__device__ __forceinline__ uint32_t sweep_group(const QArgs& a, const QLds& L, const QRange& r, int32_t g,
                                                uint32_t key[4], uint32_t* bad) {
    const int32_t n = (int32_t)a.n_tokens;
    const int32_t* tok = a.tok;
    int t0 = 0, t1 = 0, t2 = 0, t3 = 0;
    if (g + 4 <= n) {
        const int4 v = *reinterpret_cast<const int4*>(tok + g);
        t0 = v.x; t1 = v.y; t2 = v.z; t3 = v.w;
    } else if (g < n) {
        t0 = tok[g];
        t1 = tok[min(g + 1, n - 1)];
        t2 = tok[min(g + 2, n - 1)];
        t3 = tok[min(g + 3, n - 1)];
    }
    int t4 = __shfl_down(t0, 1);
    if ((threadIdx.x & 63) == 63) t4 = tok[min(g + 4, n - 1)];
    const int t[5] = {t0, t1, t2, t3, t4};
    uint32_t mask = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int32_t pos = g + j;
        if (pos >= r.S0 && pos < r.S1) {
            const int32_t q = pos - r.S0;
            const bool last = (L.last[q >> 5] >> (q & 31)) & 1u;
            if (!last || a.count_eos) {
                if (pair_key(a, t[j], last ? a.eos : t[j + 1], &key[j]))
                    mask |= 1u << j;
                else
                    ++*bad;
            }
        }
    }
    return mask;
}

// The range's pairs utterance by utterance (the range is not flat): f(key)
// per counted pair; returns this lane's (bad pairs, bad utterances).
template <typename F>
__device__ __forceinline__ uint2 per_utterance(const QArgs& a, const QLds& L, const QRange& r, F&& f) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int32_t* tok = a.tok;
    uint2 bad = {0u, 0u};
    for (int64_t u = r.u0 + wave; u < r.u1; u += QB_THREADS / 64) {
        const int64_t s64 = r.staged ? L.off[u - r.u0] : a.off[u];
        const int64_t e64 = r.staged ? L.off[u - r.u0 + 1] : a.off[u + 1];
        if (s64 < 0 || e64 < s64 || e64 > a.n_tokens) {
            bad.y += lane == 0;
            continue;
        }
        const int32_t S = (int32_t)s64, E = (int32_t)e64;
        const int32_t pend = a.count_eos ? E : E - 1;       // pairs start at S .. pend-1
        for (int32_t pos = S + lane; pos < pend; pos += 64) {
            const int x = tok[pos];
            const int y = pos + 1 == E ? a.eos : tok[min(pos + 1, E - 1)];
            uint32_t key;
            if (pair_key(a, x, y, &key))
                f(key);
            else
                ++bad.x;
        }
    }
    return bad;
}

__global__ __launch_bounds__(QB_THREADS) void q_bucket_count_kernel(QArgs a) {
    __shared__ uint32_t h[QB_MAX_NB];
    __shared__ QLds L;
    const int wg = blockIdx.x, NB = a.p.NB;
    for (int i = threadIdx.x; i < NB; i += QB_THREADS) h[i] = 0;
    __syncthreads();
    const QRange r = range_setup(a, wg, L);
    uint2 bad = {0u, 0u};
    if (r.flat) {
        for (int32_t g0 = r.S0 & ~3; g0 < r.S1; g0 += 4 * QB_THREADS) {
            uint32_t key[4];
            const uint32_t m = sweep_group(a, L, r, g0 + 4 * (int)threadIdx.x, key, &bad.x);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if ((m >> j) & 1u) atomicAdd(&h[key[j] >> QB_LOG], 1u);
        }
    } else {
        bad = per_utterance(a, L, r, [&](uint32_t key) { atomicAdd(&h[key >> QB_LOG], 1u); });
    }
    for (int o = 32; o >= 1; o >>= 1) {
        bad.x += __shfl_xor(bad.x, o);
        bad.y += __shfl_xor(bad.y, o);
    }
    if ((threadIdx.x & 63) == 0 && bad.x)
        __hip_atomic_fetch_add(a.status, (unsigned long long)bad.x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((threadIdx.x & 63) == 0 && bad.y)
        __hip_atomic_fetch_add(a.status + 1, (unsigned long long)bad.y, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    uint32_t* row = a.w.wg_cnt + (size_t)wg * NB;
    for (int i = threadIdx.x; i < NB; i += QB_THREADS) row[i] = h[i];
}

// Exclusive block scan of one value per thread (1024 threads); returns the
// thread's exclusive prefix and sets *total.
__device__ __forceinline__ uint32_t block_scan_excl(uint32_t v, uint32_t* s_w, uint32_t* total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t x = v;
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == 63) s_w[wave] = x;
    __syncthreads();
    if (wave == 0) {
        uint32_t t = lane < QS_THREADS / 64 ? s_w[lane] : 0u;
        for (int o = 1; o < 64; o <<= 1) {
            const uint32_t y = __shfl_up(t, o);
            if (lane >= o) t += y;
        }
        if (lane < QS_THREADS / 64) s_w[lane] = t;     // inclusive wave totals
    }
    __syncthreads();
    const uint32_t before = wave ? s_w[wave - 1] : 0u;
    *total = s_w[QS_THREADS / 64 - 1];
    __syncthreads();
    return before + x - v;
}

// One workgroup per bucket: prefix over the range workgroups.
__global__ __launch_bounds__(QS_THREADS) void q_column_scan_kernel(QArgs a) {
    __shared__ uint32_t s_w[QS_THREADS / 64];
    const int b = blockIdx.x, NB = a.p.NB, NWG = a.p.NWG;
    uint32_t carry = 0;
    for (int w0 = 0; w0 < NWG; w0 += QS_THREADS) {
        const int w = w0 + threadIdx.x;
        uint32_t* cell = a.w.wg_cnt + (size_t)w * NB + b;
        const uint32_t v = w < NWG ? *cell : 0u;
        uint32_t tot;
        const uint32_t ex = block_scan_excl(v, s_w, &tot);
        if (w < NWG) *cell = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) a.w.b_cnt[b] = carry;
}

// One workgroup: bucket bases, slice bases, overflow flag.
__global__ __launch_bounds__(QS_THREADS) void q_bucket_plan_kernel(QArgs a) {
    __shared__ uint32_t s_w[QS_THREADS / 64];
    const int NB = a.p.NB;
    uint64_t carry = 0, scarry = 0;
    for (int b0 = 0; b0 < NB; b0 += QS_THREADS) {
        const int b = b0 + threadIdx.x;
        const uint32_t c = b < NB ? a.w.b_cnt[b] : 0u;
        const uint32_t ns = (uint32_t)((c + a.p.S - 1) / a.p.S);
        uint32_t tot, stot;
        const uint32_t ex = block_scan_excl(c, s_w, &tot);
        const uint32_t sex = block_scan_excl(ns, s_w, &stot);
        if (b < NB) {
            a.w.b_base[b] = (uint32_t)(carry + ex);
            a.w.s_base[b] = (uint32_t)(scarry + sex);
        }
        carry += tot;
        scarry += stot;
    }
    if (threadIdx.x == 0) {
        a.w.b_base[NB] = (uint32_t)carry;
        a.w.s_base[NB] = (uint32_t)scarry;
        const bool over = carry > (uint64_t)a.n_tokens || scarry > (uint64_t)a.p.max_slices;
        a.w.ctl[0] = over ? 1u : 0u;
        if (over)
            __hip_atomic_fetch_add(a.status + 2, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Writes each pair's key into its bucket.  A flat range with at most 64
// buckets is written in rounds of 2048 positions sorted by bucket in LDS
// first (rank of a key inside its bucket by an LDS atomic, bases by a
// one-wave scan), so every bucket gets one contiguous run per round; other
// ranges write key by key at an LDS cursor.
constexpr int QS_LOCAL_NB = 64;
constexpr int QS_GROUPS = 2;                        // 4-position groups per thread per round

__global__ __launch_bounds__(QB_THREADS) void q_bucket_scatter_kernel(QArgs a) {
    __shared__ uint32_t cur[QB_MAX_NB];
    __shared__ QLds L;
    __shared__ uint32_t s_sorted[QB_THREADS * 4 * QS_GROUPS];
    __shared__ uint32_t s_cnt[QS_LOCAL_NB], s_lb[QS_LOCAL_NB + 1];
    if (a.w.ctl[0]) return;
    const int wg = blockIdx.x, NB = a.p.NB, tid = threadIdx.x;
    const uint32_t* row = a.w.wg_cnt + (size_t)wg * NB;
    for (int i = tid; i < NB; i += QB_THREADS) cur[i] = a.w.b_base[i] + row[i];
    if (tid < QS_LOCAL_NB) s_cnt[tid] = 0;
    __syncthreads();
    const QRange r = range_setup(a, wg, L);
    uint32_t* keys = a.w.keys;
    if (!r.flat) {
        (void)per_utterance(a, L, r, [&](uint32_t key) { keys[atomicAdd(&cur[key >> QB_LOG], 1u)] = key; });
        return;
    }
    uint32_t dummy = 0;
    if (NB > QS_LOCAL_NB) {
        for (int32_t g0 = r.S0 & ~3; g0 < r.S1; g0 += 4 * QB_THREADS) {
            uint32_t key[4];
            const uint32_t m = sweep_group(a, L, r, g0 + 4 * tid, key, &dummy);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if ((m >> j) & 1u) keys[atomicAdd(&cur[key[j] >> QB_LOG], 1u)] = key[j];
        }
        return;
    }
    for (int32_t g0 = r.S0 & ~3; g0 < r.S1; g0 += 4 * QB_THREADS * QS_GROUPS) {
        uint32_t key[QS_GROUPS][4], rank[QS_GROUPS][4], m[QS_GROUPS];
#pragma unroll
        for (int q = 0; q < QS_GROUPS; ++q) {
            m[q] = sweep_group(a, L, r, g0 + 4 * QB_THREADS * q + 4 * tid, key[q], &dummy);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if ((m[q] >> j) & 1u) rank[q][j] = atomicAdd(&s_cnt[key[q][j] >> QB_LOG], 1u);
        }
        __syncthreads();
        if (tid < 64) {                              // bases of this round's runs
            const uint32_t c = tid < NB ? s_cnt[tid] : 0u;
            uint32_t x = c;
            for (int o = 1; o < 64; o <<= 1) {
                const uint32_t y = __shfl_up(x, o);
                if (tid >= o) x += y;
            }
            if (tid < NB) s_lb[tid] = x - c;
            if (tid == 63) s_lb[QS_LOCAL_NB] = x;
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < QS_GROUPS; ++q)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if ((m[q] >> j) & 1u) s_sorted[s_lb[key[q][j] >> QB_LOG] + rank[q][j]] = key[q][j];
        __syncthreads();
        const uint32_t total = s_lb[QS_LOCAL_NB];
        for (uint32_t i = tid; i < total; i += QB_THREADS) {
            const uint32_t k = s_sorted[i], b = k >> QB_LOG;
            keys[cur[b] + (i - s_lb[b])] = k;
        }
        __syncthreads();
        if (tid < NB) {
            cur[tid] += s_cnt[tid];
            s_cnt[tid] = 0;
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(QH_THREADS) void q_slice_hist_kernel(QArgs a) {
    extern __shared__ uint32_t hist[];            // QB_BIN entries
    if (a.w.ctl[0]) return;
    const int s = blockIdx.x, NB = a.p.NB;
    if ((uint32_t)s >= a.w.s_base[NB]) return;
    // the bucket holding slice s: the last b with s_base[b] <= s
    int lo = 0, hi = NB;                          // s_base[lo] <= s < s_base[hi]
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (a.w.s_base[mid] <= (uint32_t)s) lo = mid; else hi = mid;
    }
    const int b = lo;
    const uint64_t k0 = a.w.b_base[b] + (uint64_t)(s - a.w.s_base[b]) * a.p.S;
    uint64_t k1 = k0 + a.p.S;
    if (k1 > a.w.b_base[b + 1]) k1 = a.w.b_base[b + 1];
    const uint4 z = {0u, 0u, 0u, 0u};
    for (uint32_t i = threadIdx.x; i < QB_BIN / 4; i += QH_THREADS) reinterpret_cast<uint4*>(hist)[i] = z;
    __syncthreads();
    // aligned 16-byte loads over [k0 & ~3, k1): the key buffer is padded to a
    // multiple of 4 keys, entries outside [k0, k1) are skipped
    const uint32_t K0 = (uint32_t)k0, K1 = (uint32_t)k1;
    constexpr int U = 4;                          // vector loads in flight per thread
    for (uint32_t blk = (K0 & ~3u) + 4 * threadIdx.x; blk < K1; blk += 4 * QH_THREADS * U) {
        uint4 v[U];
#pragma unroll
        for (int j = 0; j < U; ++j) {
            const uint32_t b4 = blk + 4 * QH_THREADS * j;
            v[j] = *reinterpret_cast<const uint4*>(a.w.keys + (b4 < K1 ? b4 : blk));
        }
#pragma unroll
        for (int j = 0; j < U; ++j) {
            const uint32_t b4 = blk + 4 * QH_THREADS * j;
            const uint32_t kv[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if (b4 + c >= K0 && b4 + c < K1) atomicAdd(&hist[kv[c] & (QB_BIN - 1)], 1u);
        }
    }
    __syncthreads();
    uint4* out = reinterpret_cast<uint4*>(a.w.part + (size_t)s * QB_BIN);
    for (uint32_t i = threadIdx.x; i < QB_BIN / 4; i += QH_THREADS) out[i] = reinterpret_cast<const uint4*>(hist)[i];
}

__global__ __launch_bounds__(256) void q_reduce_kernel(QArgs a) {
    if (a.w.ctl[0]) return;
    const uint64_t nk = (uint64_t)a.p.V * a.p.V;
    const uint64_t k = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    if (k >= nk) return;
    const uint32_t b = (uint32_t)(k >> QB_LOG), bin = (uint32_t)(k & (QB_BIN - 1));
    uint32_t sum = 0;
    for (uint32_t s = a.w.s_base[b]; s < a.w.s_base[b + 1]; ++s) sum += a.w.part[(size_t)s * QB_BIN + bin];
    if (sum) a.counts[k] += sum;
}

constexpr int QN_THREADS = 256;

// One workgroup per row.
__global__ __launch_bounds__(QN_THREADS) void q_normalize_kernel(const uint32_t* counts, int V, float alpha,
                                                                 float* logq) {
    __shared__ unsigned long long s_sum[QN_THREADS];
    const int row = blockIdx.x, tid = threadIdx.x;
    const uint32_t* cr = counts + (size_t)row * V;
    unsigned long long s = 0;
    for (int j = tid; j < V; j += QN_THREADS) s += cr[j];
    s_sum[tid] = s;
    __syncthreads();
    for (int h = QN_THREADS / 2; h > 0; h >>= 1) {
        if (tid < h) s_sum[tid] += s_sum[tid + h];
        __syncthreads();
    }
    const double av = (double)alpha;
    const double den = (double)s_sum[0] + av * (double)V;
    float* out = logq + (size_t)row * V;
    if (den == 0.0) {
        const float uni = (float)(-log((double)V));
        for (int j = tid; j < V; j += QN_THREADS) out[j] = uni;
        return;
    }
    const double lden = log(den);
    for (int j = tid; j < V; j += QN_THREADS) out[j] = (float)(log((double)cr[j] + av) - lden);
}

bool q_sizes_ok(int64_t n_tokens, int64_t n_seqs, int vocab) {
    return n_tokens >= 0 && n_tokens < (int64_t(1) << 31) && n_seqs >= 0 && vocab >= 1 && vocab <= 8192;
}

// Argument checks shared by both count entry points (the workspace aside).
int q_count_check(const int32_t* tokens, int64_t n_tokens, const int64_t* offsets, int64_t n_seqs, int vocab,
                  int eos_id, int flags, const uint32_t* counts, const uint64_t* status) {
    if (!q_sizes_ok(n_tokens, n_seqs, vocab) || eos_id < 0 || eos_id >= vocab) return MTP_EINVAL;
    if ((flags & ~MTP_Q_COUNT_EOS) != 0) return MTP_EINVAL;
    if (!counts || !status || !offsets || (n_tokens > 0 && !tokens)) return MTP_EINVAL;
    if (((uintptr_t)tokens & 15) != 0) return MTP_EINVAL;
    return MTP_OK;
}

// Validation and the six launches of a count over a workspace of ws_bytes.
int q_count_run(const int32_t* tokens, int64_t n_tokens, const int64_t* offsets, int64_t n_seqs, int vocab,
                int eos_id, int flags, uint32_t* counts, uint64_t* status, void* workspace, uint64_t ws_bytes,
                hipStream_t st) {
    const int rc = q_count_check(tokens, n_tokens, offsets, n_seqs, vocab, eos_id, flags, counts, status);
    if (rc != MTP_OK) return rc;
    if (!workspace || ((uintptr_t)workspace & 255) != 0) return MTP_EINVAL;
    const QPlan p = make_plan(n_tokens, n_seqs, vocab);
    QWs w{};
    if (carve(p, n_tokens, (char*)workspace, &w) > ws_bytes) return MTP_ENOMEM;
    if (n_seqs == 0) return MTP_OK;
    QArgs a{tokens, n_tokens, offsets, n_seqs, eos_id, (flags & MTP_Q_COUNT_EOS) ? 1 : 0, counts,
            reinterpret_cast<unsigned long long*>(status), p, w};
    hipLaunchKernelGGL(q_bucket_count_kernel, dim3(p.NWG), dim3(QB_THREADS), 0, st, a);
    hipLaunchKernelGGL(q_column_scan_kernel, dim3(p.NB), dim3(QS_THREADS), 0, st, a);
    hipLaunchKernelGGL(q_bucket_plan_kernel, dim3(1), dim3(QS_THREADS), 0, st, a);
    hipLaunchKernelGGL(q_bucket_scatter_kernel, dim3(p.NWG), dim3(QB_THREADS), 0, st, a);
    // 128 KB of dynamic LDS: raise the function's limit (per device, cheap)
    if (hipFuncSetAttribute((const void*)q_slice_hist_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                            QB_BIN * 4) != hipSuccess)
        return MTP_EHIP;
    hipLaunchKernelGGL(q_slice_hist_kernel, dim3((unsigned)p.max_slices), dim3(QH_THREADS), QB_BIN * 4, st, a);
    const uint64_t nk = (uint64_t)vocab * vocab;
    hipLaunchKernelGGL(q_reduce_kernel, dim3((unsigned)((nk + 255) / 256)), dim3(256), 0, st, a);
    return hipGetLastError() == hipSuccess ? MTP_OK : MTP_EHIP;
}

}  // namespace
}  // namespace mtp

// Fixed scratch of mtp_q_count_noalloc (callers that cannot allocate): one
// copy per device, part of the code object.  In host code `scratch` names a
// host-side stand-in, not the device array: kernels receive the device
// address that hipGetSymbolAddress returns, looked up once per device.
static __device__ __align__(256) char scratch[MTP_Q_NOALLOC_SCRATCH_BYTES];

namespace mtp {
namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// Device address of `scratch` on the current device.
int noalloc_scratch(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return MTP_EHIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MTP_EHIP;
        g_scratch_dev[dev] = p;
    }
    *out = g_scratch_dev[dev];
    return MTP_OK;
}
}  // namespace
}  // namespace mtp

extern "C" {

int mtp_q_workspace_size(int64_t n_tokens, int64_t n_seqs, int vocab, uint64_t* bytes) {
    if (!bytes || !mtp::q_sizes_ok(n_tokens, n_seqs, vocab)) return MTP_EINVAL;
    *bytes = mtp::carve(mtp::make_plan(n_tokens, n_seqs, vocab), n_tokens, nullptr, nullptr);
    return MTP_OK;
}

int mtp_q_count(const int32_t* tokens, int64_t n_tokens, const int64_t* offsets, int64_t n_seqs, int vocab,
                int eos_id, int flags, uint32_t* counts, uint64_t* status, void* workspace, uint64_t ws_bytes,
                void* hip_stream) {
    return mtp::q_count_run(tokens, n_tokens, offsets, n_seqs, vocab, eos_id, flags, counts, status, workspace,
                            ws_bytes, (hipStream_t)hip_stream);
}

int mtp_q_count_noalloc(const int32_t* tokens, int64_t n_tokens, const int64_t* offsets, int64_t n_seqs, int vocab,
                        int eos_id, int flags, uint32_t* counts, uint64_t* status, void* hip_stream) {
    using namespace mtp;
    // the same checks as mtp_q_count, then the size limit of the fixed scratch
    const int rc = q_count_check(tokens, n_tokens, offsets, n_seqs, vocab, eos_id, flags, counts, status);
    if (rc != MTP_OK) return rc;
    const uint64_t need = carve(make_plan(n_tokens, n_seqs, vocab), n_tokens, nullptr, nullptr);
    if (need > (uint64_t)MTP_Q_NOALLOC_SCRATCH_BYTES) return MTP_ENOMEM;
    void* ws = nullptr;
    const int rs = noalloc_scratch(&ws);
    if (rs != MTP_OK) return rs;
    return q_count_run(tokens, n_tokens, offsets, n_seqs, vocab, eos_id, flags, counts, status, ws,
                       (uint64_t)MTP_Q_NOALLOC_SCRATCH_BYTES, (hipStream_t)hip_stream);
}

int mtp_q_normalize(const uint32_t* counts, int vocab, float alpha, float* logq, void* hip_stream) {
    if (!counts || !logq || vocab < 1 || vocab > 8192) return MTP_EINVAL;
    if (!(alpha >= 0.f) || !isfinite(alpha)) return MTP_EINVAL;
    hipLaunchKernelGGL(mtp::q_normalize_kernel, dim3(vocab), dim3(mtp::QN_THREADS), 0, (hipStream_t)hip_stream,
                       counts, vocab, alpha, logq);
    return hipGetLastError() == hipSuccess ? MTP_OK : MTP_EHIP;
}

}  // extern "C"
