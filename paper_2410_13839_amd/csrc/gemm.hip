// GEMM kernels of the decoder trunk and the fused K-head projection.
//
// All products are "NT": C[m][n] = sum_k X[m][k] * W[n][k], with X the
// activations ([M][K], row-major) and W a Linear weight ([N][K], row-major),
// so both operands are K-contiguous.  Outputs go through an epilogue functor
// that receives 4 consecutive n of one row m.
//
//  * gemm_med_bf16: M <= 256 (decode rows of the batched path, the heads).
//    A weight stream (M = 128 rows is ~128 flop per weight byte, below the
//    MFMA / HBM ridge), so W fragments go straight from HBM into MFMA
//    registers (no LDS round trip), 16 waves per workgroup split the K range,
//    each wave loading its own activation fragments from L2 (no LDS staging:
//    no two waves read the same k), and one LDS reduction over the waves
//    precedes the epilogue.  The grid is sized so every CU streams.
//  * gemm_big_bf16: M > 256 (prefill, NAR).  256 x 256 tiles on MFMA with
//    both operands streamed global -> LDS in fragment order.
//  * gemm_f32: the fp32 model; LDS-tiled VALU FMA.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "launch.h"

namespace mtp {

// ---------------------------------------------------------------- epilogues
// An epilogue stores 4 consecutive n of one row m.  Its operands come in
// three groups, so that a kernel storing many (m, n) issues their loads
// ahead of its stores:
//   RowKey  row_key(m)   one per output row (EpiQKV: its sequence and position)
//   RowPre  row(key)     one per output row (EpiQKV: its cache page, a load
//                        that depends on the key: all keys of a kernel's rows
//                        are loaded before any of these)
//   ColPre  col(n)       one per 4-column group (the biases)
//   ElemPre elem(m, n)   one per 4 outputs (EpiResid: the residual values)
//   store(rp, cp, ep, m, n, v, split, nvalid)
// A load that follows a store it may alias cannot move above it, and vmcnt
// counts stores as well as loads, so an epilogue that loads inside each
// store4 waits one full memory round trip per store (32-64 per wave in the
// large kernel).  The loads take clamped, valid m and n (the callers pass
// m < M and n < N or the last valid ones); only the stores are guarded.
// ok(rp) says whether a row is stored at all (EpiQKV: not a padding row);
// store<true> may assume it is, so that a kernel whose wave holds only such
// rows issues the same stores on every lane (a lane-dependent branch around
// a store leaves the compiler unable to count the stores in flight, and it
// then waits for all of them before the next one).
struct EpiNoPre {};

template <class Epi>
__device__ __forceinline__ void epi_store4(const Epi& e, int m, int n, const float (&v)[4], int split, int nvalid) {
    e.template store<false>(e.row(e.row_key(m)), e.col(n), e.elem(m, n), m, n, v, split, nvalid);
}

__device__ __forceinline__ uint32_t epi_pk2(float a, float b) {
    return bf16x2_bits(a, b);
}

template <typename KVT>
struct EpiQKV {
    float* q;            // [M][d] queries (fp32)
    const float* bias;   // [3d]
    const RowInfo* rows;
    KVView kv;
    int d;
    using RowKey = RowInfo;
    struct RowPre { int page, pos; };        // pos < 0: a padding row (no cache write)
    using ColPre = float4;
    using ElemPre = EpiNoPre;
    __device__ __forceinline__ RowKey row_key(int m) const { return rows[m]; }
    // the page stays as loaded (nothing computed from it before the stores)
    __device__ __forceinline__ RowPre row(const RowKey& ri) const {
        const int pos = max(ri.pos, 0), seq = max(ri.seq, 0);
        return RowPre{kv.block_table[(size_t)seq * kv.max_pages_per_seq + (pos >> kv.page_shift)], ri.pos};
    }
    __device__ __forceinline__ ColPre col(int n) const { return *reinterpret_cast<const float4*>(bias + n); }
    __device__ __forceinline__ ElemPre elem(int, int) const { return {}; }
    __device__ __forceinline__ bool ok(const RowPre& rp) const { return rp.pos >= 0; }
    // every caller's wave holds 16 consecutive columns inside one section
    // (d is a multiple of 64), so the section is wave-uniform
    template <bool ROWS_OK>
    __device__ __forceinline__ void store(const RowPre& rp, const ColPre& bv, const ElemPre&, int m, int n,
                                          const float (&v)[4], int, int) const {
        const float r0 = v[0] + bv.x, r1 = v[1] + bv.y, r2 = v[2] + bv.z, r3 = v[3] + bv.w;
        const int sec = __builtin_amdgcn_readfirstlane((n >= d) + (n >= 2 * d));   // q, k or v
        if (sec == 0) {
            *reinterpret_cast<float4*>(q + (size_t)m * d + n) = make_float4(r0, r1, r2, r3);
            return;
        }
        if (!ROWS_OK && rp.pos < 0) return;
        const int c = n - sec * d;
        const int slot = rp.pos & (kv.page_size - 1);
        KVT* blk = reinterpret_cast<KVT*>(kv.pool) + kv_page_block(kv, rp.page, sec - 1, c >> 6);
        if constexpr (sizeof(KVT) == 2) {
            if (sec == 2) {   // transposed V block: [dim][slot]
                bf16_t* vt = blk + (size_t)(c & 63) * kv.page_size + slot;
                vt[0] = f32_to_bf16(r0);
                vt[kv.page_size] = f32_to_bf16(r1);
                vt[2 * kv.page_size] = f32_to_bf16(r2);
                vt[3 * kv.page_size] = f32_to_bf16(r3);
                return;
            }
            *reinterpret_cast<uint2*>(blk + (size_t)slot * MTP_HEAD_DIM + (c & 63)) =
                make_uint2(epi_pk2(r0, r1), epi_pk2(r2, r3));
        } else {
            *reinterpret_cast<float4*>(blk + (size_t)slot * MTP_HEAD_DIM + (c & 63)) = make_float4(r0, r1, r2, r3);
        }
    }
};

template <typename OutT>
struct EpiGelu {
    OutT* out;
    const float* bias;
    int ldo;
    int pk;               // bf16 output in fragment order (K = ldo)
    using RowKey = EpiNoPre;
    using RowPre = EpiNoPre;
    using ColPre = float4;
    using ElemPre = EpiNoPre;
    __device__ __forceinline__ RowKey row_key(int) const { return {}; }
    __device__ __forceinline__ RowPre row(const RowKey&) const { return {}; }
    __device__ __forceinline__ ColPre col(int n) const { return *reinterpret_cast<const float4*>(bias + n); }
    __device__ __forceinline__ ElemPre elem(int, int) const { return {}; }
    __device__ __forceinline__ bool ok(const RowPre&) const { return true; }
    template <bool ROWS_OK>
    __device__ __forceinline__ void store(const RowPre&, const ColPre& bv, const ElemPre&, int m, int n,
                                          const float (&v)[4], int, int) const {
        const float r[4] = {gelu_erf(v[0] + bv.x), gelu_erf(v[1] + bv.y), gelu_erf(v[2] + bv.z), gelu_erf(v[3] + bv.w)};
        OutT* p = out + (pk ? frag_off(m, n, ldo) : (size_t)m * ldo + n);
        if constexpr (sizeof(OutT) == 2) {
            *reinterpret_cast<uint2*>(p) = make_uint2(epi_pk2(r[0], r[1]), epi_pk2(r[2], r[3]));
        } else {
            *reinterpret_cast<float4*>(p) = make_float4(r[0], r[1], r[2], r[3]);
        }
    }
};

struct EpiPartial {
    float* part;          // [split][M][ldo]
    int ldo;
    size_t split_stride;  // elements between splits
    using RowKey = EpiNoPre;
    using RowPre = EpiNoPre;
    using ColPre = EpiNoPre;
    using ElemPre = EpiNoPre;
    __device__ __forceinline__ RowKey row_key(int) const { return {}; }
    __device__ __forceinline__ RowPre row(const RowKey&) const { return {}; }
    __device__ __forceinline__ ColPre col(int) const { return {}; }
    __device__ __forceinline__ ElemPre elem(int, int) const { return {}; }
    __device__ __forceinline__ bool ok(const RowPre&) const { return true; }
    template <bool ROWS_OK>
    __device__ __forceinline__ void store(const RowPre&, const ColPre&, const ElemPre&, int m, int n,
                                          const float (&v)[4], int split, int) const {
        *reinterpret_cast<float4*>(part + split * split_stride + (size_t)m * ldo + n) =
            make_float4(v[0], v[1], v[2], v[3]);
    }
};

// h[m][n..n+3] += product + bias: the residual stream updated in place by a
// projection with no K split (every (m, n) belongs to one workgroup, so the
// read-modify-write is race free); the same association as resid_ln_kernel.
struct EpiResid {
    float* h;             // [M][ldh]
    const float* bias;    // [N]
    int ldh;
    using RowKey = EpiNoPre;
    using RowPre = EpiNoPre;
    using ColPre = float4;
    using ElemPre = float4;
    __device__ __forceinline__ RowKey row_key(int) const { return {}; }
    __device__ __forceinline__ RowPre row(const RowKey&) const { return {}; }
    __device__ __forceinline__ ColPre col(int n) const { return *reinterpret_cast<const float4*>(bias + n); }
    __device__ __forceinline__ ElemPre elem(int m, int n) const {
        return *reinterpret_cast<const float4*>(h + (size_t)m * ldh + n);
    }
    __device__ __forceinline__ bool ok(const RowPre&) const { return true; }
    template <bool ROWS_OK>
    __device__ __forceinline__ void store(const RowPre&, const ColPre& bv, const ElemPre& x, int m, int n,
                                          const float (&v)[4], int, int) const {
        *reinterpret_cast<float4*>(h + (size_t)m * ldh + n) =
            make_float4(x.x + (v[0] + bv.x), x.y + (v[1] + bv.y), x.z + (v[2] + bv.z), x.w + (v[3] + bv.w));
    }
};

struct EpiLogits {
    float* out;           // [M][ldo]
    const float* bias;    // [N]
    int ldo;
    int N;
    using RowKey = EpiNoPre;
    using RowPre = EpiNoPre;
    using ColPre = float4;
    using ElemPre = EpiNoPre;
    __device__ __forceinline__ RowKey row_key(int) const { return {}; }
    __device__ __forceinline__ RowPre row(const RowKey&) const { return {}; }
    __device__ __forceinline__ ColPre col(int n) const {
        return make_float4(bias[min(n, N - 1)], bias[min(n + 1, N - 1)], bias[min(n + 2, N - 1)], bias[min(n + 3, N - 1)]);
    }
    __device__ __forceinline__ ElemPre elem(int, int) const { return {}; }
    __device__ __forceinline__ bool ok(const RowPre&) const { return true; }
    template <bool ROWS_OK>
    __device__ __forceinline__ void store(const RowPre&, const ColPre& bv, const ElemPre&, int m, int n,
                                          const float (&v)[4], int, int nvalid) const {
        float* p = out + (size_t)m * ldo + n;
        const float b[4] = {bv.x, bv.y, bv.z, bv.w};
        for (int i = 0; i < nvalid; ++i) p[i] = v[i] + b[i];
    }
};

// ---------------------------------------------------------------- medium bf16
// Workgroup (x, y, z) = (NT 16-column tiles, 16*MT-row group, K split).  Wave
// w takes k steps w, w + 16, ... of its split (32 k per step), up to MAXST at
// a time, all loads of a round in flight together: NT weight fragments
// (packed order, each one contiguous 1 KB wave load) and one 16 x 32
// activation fragment per row tile, which serves all NT column tiles (the
// activations are re-read from L2 once per column group, so wider groups
// cut that traffic).  Rows beyond M read the last valid row and column tiles
// beyond N the last valid tile; neither is stored.  The wave index is made
// scalar so the step guards are uniform branches.
constexpr int GM_NW = 16;

template <int MT, int NT, int MAXST, int XP, class Epi>
__global__ __launch_bounds__(64 * GM_NW) void gemm_med_bf16(const bf16_t* __restrict__ X, int ldx, int M,
                                                            const bf16_t* __restrict__ W, int N, int K,
                                                            int k_per_split, Epi epi) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r = lane & 15, g = lane >> 4;
    const int ntiles = (N + 15) >> 4;
    const int nt0 = blockIdx.x * NT;
    const int m0 = blockIdx.y * 16 * MT;
    const int split = blockIdx.z;
    const int kb = split * k_per_split;
    const int nsteps = k_per_split >> 5;
    const bf16_t* wp[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j)
        wp[j] = W + ((size_t)min(nt0 + j, ntiles - 1) * (K >> 5) + (kb >> 5)) * 512 + lane * 8;
    // XP: X in fragment order (one contiguous 1 KB block per row tile and k
    // step, rows padded to 16), else row-major
    const bf16_t* xp[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        if (XP) {
            const int t = min(m0 / 16 + mt, (M - 1) >> 4);
            xp[mt] = X + ((size_t)t * (K >> 5) + (kb >> 5)) * 512 + lane * 8;
        } else {
            const int m = min(m0 + 16 * mt + r, M - 1);
            xp[mt] = X + (size_t)m * ldx + kb + g * 8;
        }
    }
    f32x4_t acc[NT][MT];
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[j][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    for (int s0 = wave; s0 < nsteps; s0 += GM_NW * MAXST) {
        uint4 wv[MAXST][NT];
        uint4 xv[MAXST][MT];
#pragma unroll
        for (int u = 0; u < MAXST; ++u) {
            const int ss = s0 + GM_NW * u;
            if (ss < nsteps) {
#pragma unroll
                for (int j = 0; j < NT; ++j) wv[u][j] = *reinterpret_cast<const uint4*>(wp[j] + (size_t)ss * 512);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    xv[u][mt] = *reinterpret_cast<const uint4*>(xp[mt] + (XP ? (size_t)ss * 512 : (size_t)ss * 32));
            }
        }
#pragma unroll
        for (int u = 0; u < MAXST; ++u) {
            if (s0 + GM_NW * u < nsteps) {
#pragma unroll
                for (int j = 0; j < NT; ++j)
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
                        acc[j][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wv[u][j]),
                                                                             __builtin_bit_cast(bf16x8_t, xv[u][mt]),
                                                                             acc[j][mt], 0, 0, 0);
            }
        }
    }

    // one output item (4 columns of one row) per thread: its epilogue
    // operands load while the waves' sums go through LDS
    static_assert(NT * MT * 64 <= 64 * GM_NW, "one epilogue item per thread");
    const int t = threadIdx.x;
    const int jm = min(t >> 6, NT * MT - 1), l = t & 63;
    const int j = jm / MT, mt = jm - j * MT;
    const int m = m0 + 16 * mt + (l & 15);
    const int n = (nt0 + j) * 16 + 4 * (l >> 4);
    const int mc = min(m, M - 1), nc = n < N ? n : ((N - 1) & ~3);
    const typename Epi::RowPre rp = epi.row(epi.row_key(mc));
    const typename Epi::ColPre cp = epi.col(nc);
    const typename Epi::ElemPre ep = epi.elem(mc, nc);
    __shared__ f32x4_t red[GM_NW][NT * MT][64];
#pragma unroll
    for (int j2 = 0; j2 < NT; ++j2)
#pragma unroll
        for (int mt2 = 0; mt2 < MT; ++mt2) red[wave][j2 * MT + mt2][lane] = acc[j2][mt2];
    __syncthreads();
    if (t < NT * MT * 64) {
        f32x4_t s = red[0][jm][l];
#pragma unroll
        for (int w = 1; w < GM_NW; ++w) s += red[w][jm][l];
        if (m < M && n < N) {
            const float v[4] = {s[0], s[1], s[2], s[3]};
            epi.template store<false>(rp, cp, ep, m, n, v, split, min(4, N - n));
        }
    }
}

// Column tiles per workgroup: two, so every activation fragment serves two
// weight fragments (the activations are re-read once per workgroup), with
// the LDS reduction holding 16 waves x NT x MT tiles (at most 8).
constexpr int GM_NT = 2;

template <int MT, int XP, class Epi>
static void launch_med(hipStream_t st, const bf16_t* X, int ldx, int M, const bf16_t* W, int N, int K, int splits,
                       Epi epi) {
    constexpr int NT = GM_NT;
    static_assert(NT * MT <= 8, "LDS reduction");
    const int kps = K / splits;
    const int per_wave = ((kps >> 5) + GM_NW - 1) / GM_NW;   // k steps per wave
    dim3 grid(((N + 15) / 16 + NT - 1) / NT, (M + 16 * MT - 1) / (16 * MT), splits);
    dim3 block(64 * GM_NW);
    // one round of loads holds at most MAXST x (NT + MT) fragments per wave
    constexpr int CAP = NT * MT >= 8 ? 2 : 4;
    if (per_wave <= 1)
        hipLaunchKernelGGL((gemm_med_bf16<MT, NT, 1, XP, Epi>), grid, block, 0, st, X, ldx, M, W, N, K, kps, epi);
    else if (per_wave == 2 || CAP == 2)
        hipLaunchKernelGGL((gemm_med_bf16<MT, NT, 2, XP, Epi>), grid, block, 0, st, X, ldx, M, W, N, K, kps, epi);
    else if (per_wave == 3)
        hipLaunchKernelGGL((gemm_med_bf16<MT, NT, 3, XP, Epi>), grid, block, 0, st, X, ldx, M, W, N, K, kps, epi);
    else
        hipLaunchKernelGGL((gemm_med_bf16<MT, NT, CAP, XP, Epi>), grid, block, 0, st, X, ldx, M, W, N, K, kps, epi);
}

template <int MT, class Epi>
static void launch_med_x(hipStream_t st, const bf16_t* X, int ldx, int M, const bf16_t* W, int N, int K, int splits,
                         int xpk, Epi epi) {
    if (xpk) launch_med<MT, 1>(st, X, ldx, M, W, N, K, splits, epi);
    else launch_med<MT, 0>(st, X, ldx, M, W, N, K, splits, epi);
}

// ---------------------------------------------------------------- large bf16
// M > 256 (prefill, NAR).  Tiles of BM rows x BN columns (256 x 256 and
// 256 x 128 with 8 waves in a 2 x 4 grid, each wave owning 128 x BN/4
// outputs as 8 x BN/64 v_mfma_f32_16x16x32_bf16 tiles; 128 x 128 with 4
// waves in a 2 x 2 grid, 64 x 64 outputs each, for products too small to
// give the CUs enough of the larger tiles).  Both
// operands are in fragment order (activations written so by their producers,
// weights packed at load), so a 16 x 32 fragment is one contiguous 1 KB; it
// travels global -> LDS by one global_load_lds_dwordx4 per wave (lane l's 16
// bytes land at byte 16 l, the order the MFMA operand read wants: every
// ds_read_b128 is conflict free) with no register staging.  K advances 32 per
// stage through NS = 4 LDS stages, NS - 1 of them in flight while one is
// consumed.  Each stage buffer is its own LDS object and the stage loop is
// unrolled by NS, so the compiler's LDS-DMA waits see which buffer a read
// touches.  Workgroups are numbered so that the ones sharing an XCD (the
// dispatcher deals workgroups to the 8 XCDs in turn) take neighbouring tiles
// of one row band, which they share through that XCD's L2.
constexpr int GB_NS = 4;

__device__ __forceinline__ constexpr int vmcnt_imm(int n) {
    // s_waitcnt immediate: vmcnt = n, expcnt and lgkmcnt not waited on
    return (n & 15) | (((n >> 4) & 3) << 14) | (7 << 4) | (15 << 8);
}

// Workgroup barrier without the memory fence __syncthreads() adds: that
// fence waits for every outstanding global load, the stages still in flight
// included.  The explicit vmcnt wait before it covers the stage consumed.
__device__ __forceinline__ void gb_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <int BM, int BN, int NWV, class Epi>
__global__ __launch_bounds__(64 * NWV) void gemm_big_bf16(const bf16_t* __restrict__ X, int M,
                                                          const bf16_t* __restrict__ W, int N, int K, int k_per_split,
                                                          int tiles_m, int tiles_n, Epi epi) {
    constexpr int FM = BM / 16, FN = BN / 16;   // 16-row fragments of a stage
    constexpr int NF = FM + FN;                 // fragments per stage (one 32-k step)
    constexpr int NL = NF / NWV;                // global_load_lds per wave per stage
    constexpr int WGN = NWV / 2;                // waves along n (two along m)
    constexpr int WFM = FM / 2, WFN = FN / WGN; // fragments per wave
    static_assert(NF % NWV == 0 && (WFM == 8 || WFM == 4) && WFN >= 1, "tile shape");
    typedef __attribute__((address_space(3))) void lds_void;
    __shared__ __attribute__((aligned(1024))) bf16_t s0[NF * 512];
    __shared__ __attribute__((aligned(1024))) bf16_t s1[NF * 512];
    __shared__ __attribute__((aligned(1024))) bf16_t s2[NF * 512];
    __shared__ __attribute__((aligned(1024))) bf16_t s3[NF * 512];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave / WGN, wn = wave - wm * WGN;
    // tiles of this workgroup: XCD x (= bid % 8) takes the x-th eighth of the
    // tiles in row-band order (n fastest), and its workgroups take them in
    // turn (workgroup j of the XCD: tiles j, j + wgx, ...), so the ones in
    // flight on an XCD are neighbours in a row band
    const int ntile = tiles_m * tiles_n;
    const int bid = blockIdx.x;
    const int per = (ntile + 7) >> 3;
    const int wgx = gridDim.x >> 3;             // workgroups per XCD
    const int t_end = min(((bid & 7) + 1) * per, ntile);
    int t = (bid & 7) * per + (bid >> 3);
    if (t >= t_end) return;                     // uniform: whole workgroup
    const int mfr_last = ((M + 15) >> 4) - 1, nfr_last = ((N + 15) >> 4) - 1;
    const int split = blockIdx.y;
    const int ks0 = (split * k_per_split) >> 5; // first 32-k step
    const int nst = k_per_split >> 5;
    const int K32 = K >> 5;

    // fragment f of a stage: f < FM is activation rows 16 f.., else weight
    // rows 16 (f - FM)..; wave w issues f = w, w + NWV, ...
    int mfr0 = 0, nfr0 = 0;                     // first 16-row fragment of each operand
    const bf16_t* src[NL];
    auto set_tile = [&](int tt) {
        const int tm = tt / tiles_n, tn = tt - tm * tiles_n;
        mfr0 = tm * FM;
        nfr0 = tn * FN;
#pragma unroll
        for (int i = 0; i < NL; ++i) {
            const int f = wave + NWV * i;
            const bf16_t* base;
            if (f < FM) base = X + (size_t)min(mfr0 + f, mfr_last) * K32 * 512;
            else base = W + (size_t)min(nfr0 + f - FM, nfr_last) * K32 * 512;
            src[i] = base + (size_t)ks0 * 512 + lane * 8;
        }
    };
    set_tile(t);
    auto issue = [&](bf16_t* buf, int st) {
#pragma unroll
        for (int i = 0; i < NL; ++i)
            __builtin_amdgcn_global_load_lds((const void*)(src[i] + (size_t)st * 512),
                                             (lds_void*)(buf + (wave + NWV * i) * 512), 16, 0, 0);
    };

    f32x4_t acc[WFN][WFM];
#pragma unroll
    for (int i = 0; i < WFN; ++i)
#pragma unroll
        for (int j = 0; j < WFM; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // Operand reads are ds_read_b128 in asm: the compiler cannot tell the
    // stage being read from the stages the LDS DMA is still filling and would
    // wait for every load in flight before each read.  The stage read is
    // complete (the vmcnt wait and barrier before it).  Each asm block issues
    // its reads and waits for them itself, so its outputs are valid when it
    // ends whatever the compiler does with the registers afterwards.
    auto compute = [&](const bf16_t* buf) {
        const uint32_t lb = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) bf16_t*)buf + lane * 16;
        const uint32_t la = lb + (FM + wn * WFN) * 1024, lbm = lb + wm * WFM * 1024;
        bf16x8_t a[WFN], b[WFM];
        static_assert((WFN == 8 || WFN == 4 || WFN == 2), "operand counts");
        if constexpr (WFN == 8) {
            asm volatile(
                "ds_read_b128 %0, %8 offset:0\n\tds_read_b128 %1, %8 offset:1024\n\t"
                "ds_read_b128 %2, %8 offset:2048\n\tds_read_b128 %3, %8 offset:3072\n\t"
                "ds_read_b128 %4, %8 offset:4096\n\tds_read_b128 %5, %8 offset:5120\n\t"
                "ds_read_b128 %6, %8 offset:6144\n\tds_read_b128 %7, %8 offset:7168\n\t"
                "s_waitcnt lgkmcnt(0)"
                : "=&v"(a[0]), "=&v"(a[1]), "=&v"(a[2]), "=&v"(a[3]), "=&v"(a[4]), "=&v"(a[5]), "=&v"(a[6]),
                  "=&v"(a[7])
                : "v"(la)
                : "memory");
        } else if constexpr (WFN == 4) {
            asm volatile(
                "ds_read_b128 %0, %4 offset:0\n\tds_read_b128 %1, %4 offset:1024\n\t"
                "ds_read_b128 %2, %4 offset:2048\n\tds_read_b128 %3, %4 offset:3072\n\t"
                "s_waitcnt lgkmcnt(0)"
                : "=&v"(a[0]), "=&v"(a[1]), "=&v"(a[2]), "=&v"(a[3])
                : "v"(la)
                : "memory");
        } else {
            asm volatile(
                "ds_read_b128 %0, %2 offset:0\n\tds_read_b128 %1, %2 offset:1024\n\t"
                "s_waitcnt lgkmcnt(0)"
                : "=&v"(a[0]), "=&v"(a[1])
                : "v"(la)
                : "memory");
        }
        if constexpr (WFM == 8) {
            asm volatile(
                "ds_read_b128 %0, %8 offset:0\n\tds_read_b128 %1, %8 offset:1024\n\t"
                "ds_read_b128 %2, %8 offset:2048\n\tds_read_b128 %3, %8 offset:3072\n\t"
                "ds_read_b128 %4, %8 offset:4096\n\tds_read_b128 %5, %8 offset:5120\n\t"
                "ds_read_b128 %6, %8 offset:6144\n\tds_read_b128 %7, %8 offset:7168\n\t"
                "s_waitcnt lgkmcnt(0)"
                : "=&v"(b[0]), "=&v"(b[1]), "=&v"(b[2]), "=&v"(b[3]), "=&v"(b[4]), "=&v"(b[5]), "=&v"(b[6]),
                  "=&v"(b[7])
                : "v"(lbm)
                : "memory");
        } else {
            asm volatile(
                "ds_read_b128 %0, %4 offset:0\n\tds_read_b128 %1, %4 offset:1024\n\t"
                "ds_read_b128 %2, %4 offset:2048\n\tds_read_b128 %3, %4 offset:3072\n\t"
                "s_waitcnt lgkmcnt(0)"
                : "=&v"(b[0]), "=&v"(b[1]), "=&v"(b[2]), "=&v"(b[3])
                : "v"(lbm)
                : "memory");
        }
#pragma unroll
        for (int i = 0; i < WFN; ++i)
#pragma unroll
            for (int j = 0; j < WFM; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    };

    // prologue: stages 0 .. NS-2 in flight
    if (0 < nst) issue(s0, 0);
    if (1 < nst) issue(s1, 1);
    if (2 < nst) issue(s2, 2);
    const int r = lane & 15, g = lane >> 4;
    for (bool later = false;; later = true) {
        // step st: wait for stage st (the NS-2 later stages may stay in
        // flight; on a later tile the first step waits for everything, the
        // previous tile's output stores included), barrier (stage st visible
        // to all waves, and every wave is done with the buffer stage st +
        // NS - 1 refills), refill, consume
#define GB_STEP(BUF, NEXT, U)                                                          \
        {                                                                              \
            const int st = st0 + (U);                                                  \
            if (st < nst) {                                                            \
                if (later && st == 0) __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));        \
                else if (st + 2 < nst) __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * NL));  \
                else if (st + 1 < nst) __builtin_amdgcn_s_waitcnt(vmcnt_imm(NL));      \
                else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));                         \
                gb_barrier();                                                          \
                if (st + GB_NS - 1 < nst) issue(NEXT, st + GB_NS - 1);                 \
                compute(BUF);                                                          \
            }                                                                          \
        }
        for (int st0 = 0; st0 < nst; st0 += GB_NS) {
            GB_STEP(s0, s3, 0)
            GB_STEP(s1, s0, 1)
            GB_STEP(s2, s1, 2)
            GB_STEP(s3, s2, 3)
        }
#undef GB_STEP
        // the next tile's first stages go out before this tile's outputs are
        // stored, once every wave is done reading the stage buffers
        const int em0 = mfr0, en0 = nfr0;
        const int t_next = t + wgx;
        const bool more = t_next < t_end;      // uniform
        if (more) {
            gb_barrier();
            set_tile(t_next);
            if (0 < nst) issue(s0, 0);
            if (1 < nst) issue(s1, 1);
            if (2 < nst) issue(s2, 2);
        }
        // epilogue: lane (r, g) of tile (i, j) holds outputs n = 4 g .. 4 g + 3
        // of weight fragment i, row m = r of activation fragment j.  The
        // rows' operands load once; each column fragment's operands load
        // while the previous fragment's outputs are stored, so a wave waits
        // about WFN + 1 memory round trips, not one per store.  A wave whose
        // outputs all lie inside the product (and whose rows are all stored)
        // stores without guards.
        int em[WFM], emc[WFM];
        typename Epi::RowKey rk[WFM];
        typename Epi::RowPre rp[WFM];
        bool rows_ok = true;
#pragma unroll
        for (int j = 0; j < WFM; ++j) {
            em[j] = (em0 + wm * WFM + j) * 16 + r;
            emc[j] = min(em[j], M - 1);
            rk[j] = epi.row_key(emc[j]);
        }
#pragma unroll
        for (int j = 0; j < WFM; ++j) rp[j] = epi.row(rk[j]);
#pragma unroll
        for (int j = 0; j < WFM; ++j) rows_ok = rows_ok && epi.ok(rp[j]);
        const bool inside = (em0 + wm * WFM + WFM) * 16 <= M && (en0 + wn * WFN + WFN) * 16 <= N;   // uniform
        const bool fast = inside && __all(rows_ok);
        // column operands (biases) go out one fragment ahead; per-output
        // operands (the residual values) one fragment at a time, after the
        // previous fragment's stores, for want of registers (the 128 of the
        // accumulators are still live)
        typename Epi::ColPre cp[2];
        typename Epi::ElemPre ep[WFM];
        auto col_n = [&](int i) {
            const int n = (en0 + wn * WFN + i) * 16 + 4 * g;
            return n < N ? n : ((N - 1) & ~3);
        };
        auto store_all = [&](auto guarded) {
            constexpr bool GUARD = decltype(guarded)::value;
            cp[0] = epi.col(col_n(0));
#pragma unroll
            for (int j = 0; j < WFM; ++j) ep[j] = epi.elem(emc[j], col_n(0));
#pragma unroll
            for (int i = 0; i < WFN; ++i) {
                if (i + 1 < WFN) cp[(i + 1) & 1] = epi.col(col_n(i + 1));
                const int n = (en0 + wn * WFN + i) * 16 + 4 * g;
#pragma unroll
                for (int j = 0; j < WFM; ++j) {
                    const float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
                    if (!GUARD) {
                        epi.template store<true>(rp[j], cp[i & 1], ep[j], em[j], n, v, split, 4);
                    } else if (em[j] < M && n < N) {
                        epi.template store<false>(rp[j], cp[i & 1], ep[j], em[j], n, v, split, min(4, N - n));
                    }
                }
                if (i + 1 < WFN) {
#pragma unroll
                    for (int j = 0; j < WFM; ++j) ep[j] = epi.elem(emc[j], col_n(i + 1));
                }
            }
        };
        if (fast) store_all(std::false_type{});
        else store_all(std::true_type{});
#pragma unroll
        for (int i = 0; i < WFN; ++i)
#pragma unroll
            for (int j = 0; j < WFM; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        if (!more) break;
        t = t_next;
    }
}

template <int BM, int BN, int NWV, class Epi>
static hipError_t launch_big(hipStream_t st, const bf16_t* X, int M, const bf16_t* W, int N, int K, int splits,
                             Epi epi) {
    const int kps = K / splits;
    if (kps % 32) return hipErrorInvalidValue;
    const int tm = (M + BM - 1) / BM, tn = (N + BN - 1) / BN;
    const int ntile = tm * tn;
    // the tile numbering deals eighths of the tiles to the XCDs; each XCD
    // gets at most as many workgroups as it holds at once (its CUs times the
    // workgroups per CU the LDS stages allow), and those take its tiles in
    // turn, so a workgroup's next tile streams in while it stores the last
    static int n_cu = 0;
    if (n_cu == 0) {
        int dev = 0, v = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v < 8)
            v = 256;
        n_cu = v;
    }
    constexpr int lds_kb = GB_NS * (BM / 16 + BN / 16);   // 1 KB per fragment per stage
    const int per_cu = lds_kb <= 80 ? 2 : 1;               // 160 KB of LDS per CU
    const int per_xcd = std::min((ntile + 7) / 8, std::max(1, n_cu / 8) * per_cu);
    dim3 grid(8 * per_xcd, splits);
    hipLaunchKernelGGL((gemm_big_bf16<BM, BN, NWV, Epi>), grid, dim3(64 * NWV), 0, st, X, M, W, N, K, kps, tm, tn, epi);
    return hipGetLastError();
}

// ----------------------------------------------------------------- fp32 VALU
template <class Epi>
__global__ __launch_bounds__(256) void gemm_f32(const float* __restrict__ X, int ldx, int M,
                                                const float* __restrict__ W, int N, int K,
                                                int k_per_split, Epi epi) {
    __shared__ float Xs[16][33];
    __shared__ float Ws[64][33];
    const int tid = threadIdx.x;
    const int mi = tid >> 4, n4 = tid & 15;
    const int m0 = blockIdx.y * 16, n0 = blockIdx.x * 64;
    const int split = blockIdx.z;
    const int kb = split * k_per_split;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int k0 = kb; k0 < kb + k_per_split; k0 += 32) {
        for (int e = tid; e < 16 * 32; e += 256) {
            int row = e >> 5, col = e & 31;
            int m = m0 + row;
            Xs[row][col] = (m < M) ? X[(size_t)m * ldx + k0 + col] : 0.f;
        }
        for (int e = tid; e < 64 * 32; e += 256) {
            int row = e >> 5, col = e & 31;
            int n = n0 + row;
            Ws[row][col] = (n < N) ? W[(size_t)n * K + k0 + col] : 0.f;
        }
        __syncthreads();
#pragma unroll 8
        for (int kk = 0; kk < 32; ++kk) {
            float x = Xs[mi][kk];
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] = fmaf(x, Ws[n4 * 4 + i][kk], acc[i]);
        }
        __syncthreads();
    }
    const int m = m0 + mi, n = n0 + n4 * 4;
    if (m < M && n < N) epi_store4(epi, m, n, acc, split, min(4, N - n));
}

// ------------------------------------------------------------------ launchers
// Tile of the large-M kernel for an M x N product (M > 256): 256 x 256 when
// that gives at least 128 tiles (half the CUs), 256 x 128 when that gives
// 192, else 128 x 128 when that gives 96 (64 for a split-K product, whose
// K splits multiply the workgroups), else 256 x 128 when that gives 64;
// otherwise {0, 0}: the product is too small for any and goes to the medium
// kernel (64-row groups, one workgroup per 32 columns).  Measured at M =
// 325 and 1,075: 72-81 tiles of 128 x 128 without K splits lose to the
// medium kernel, 96 and more win against it and against 256 x 128.
struct BigTile { int bm, bn; };
static int tile_count(int M, int N, int bm, int bn) { return ((M + bm - 1) / bm) * ((N + bn - 1) / bn); }
static BigTile big_tile(int M, int N, bool splittable) {
    if (tile_count(M, N, 256, 256) >= 128) return {256, 256};
    if (tile_count(M, N, 256, 128) >= 192) return {256, 128};
    if (tile_count(M, N, 128, 128) >= (splittable ? 64 : 96)) return {128, 128};
    if (tile_count(M, N, 256, 128) >= 64) return {256, 128};
    return {0, 0};
}
template <class Epi>
static hipError_t launch_bf16(hipStream_t st, const bf16_t* X, int ldx, int M, const bf16_t* W, int N, int K,
                              int splits, int xpk, Epi epi) {
    if (splits < 1 || K % (32 * splits)) return hipErrorInvalidValue;
    if (M <= 16) {
        launch_med_x<1>(st, X, ldx, M, W, N, K, splits, xpk, epi);
    } else if (M <= 32) {
        launch_med_x<2>(st, X, ldx, M, W, N, K, splits, xpk, epi);
    } else {
        const BigTile bt = big_tile(M, N, std::is_same<Epi, EpiPartial>::value);
        if (bt.bm == 0) {
            launch_med_x<4>(st, X, ldx, M, W, N, K, splits, xpk, epi);
        } else {
            if (!xpk) return hipErrorInvalidValue;   // large products take fragment-order activations only
            if (bt.bm == 128) return launch_big<128, 128, 4>(st, X, M, W, N, K, splits, epi);
            return bt.bn == 256 ? launch_big<256, 256, 8>(st, X, M, W, N, K, splits, epi)
                                : launch_big<256, 128, 8>(st, X, M, W, N, K, splits, epi);
        }
    }
    return hipGetLastError();
}

template <class Epi>
static hipError_t launch_f32(hipStream_t st, const float* X, int ldx, int M, const float* W, int N, int K,
                             int splits, Epi epi) {
    dim3 grid((N + 63) / 64, (M + 15) / 16, splits);
    hipLaunchKernelGGL((gemm_f32<Epi>), grid, dim3(256), 0, st, X, ldx, M, W, N, K, K / splits, epi);
    return hipGetLastError();
}

int gemm_split_granule(int dtype, int M) {
    (void)dtype;
    (void)M;
    return 32;   // one k step of the bf16 kernels, one LDS tile of the fp32 one
}

// Whether an M x N bf16 product takes the large-M kernel (the prefill and
// NAR trunk), where a residual projection updates the residual stream in its
// epilogue (EPI_RESID) instead of writing split-K partial sums.
int gemm_resid_in_place(int M, int N) {
    return M > 256 && big_tile(M, N, false).bm != 0;
}

// Workgroups of one split-K-able (partial-sum) bf16 launch for M rows and N
// columns before K splitting.
int gemm_tiles(int M, int N) {
    const int groups = ((N + 15) / 16 + GM_NT - 1) / GM_NT;
    if (M <= 32) return groups;
    const BigTile bt = M <= 256 ? BigTile{0, 0} : big_tile(M, N, true);
    if (bt.bm == 0) return groups * ((M + 63) / 64);
    return tile_count(M, N, bt.bm, bt.bn);
}

hipError_t gemm(hipStream_t st, const GemmArgs& a) {
    const bool bf = a.dtype == 1;
    switch (a.epi) {
    case EPI_QKV: {
        if (bf) {
            EpiQKV<bf16_t> e{a.q, a.bias, a.rows, a.kv, a.d};
            return launch_bf16(st, (const bf16_t*)a.X, a.ldx, a.M, (const bf16_t*)a.W, a.N, a.K, 1, a.xpk, e);
        }
        EpiQKV<float> e{a.q, a.bias, a.rows, a.kv, a.d};
        return launch_f32(st, (const float*)a.X, a.ldx, a.M, (const float*)a.W, a.N, a.K, 1, e);
    }
    case EPI_GELU: {
        if (bf) {
            EpiGelu<bf16_t> e{(bf16_t*)a.out, a.bias, a.ldo, a.opk};
            return launch_bf16(st, (const bf16_t*)a.X, a.ldx, a.M, (const bf16_t*)a.W, a.N, a.K, 1, a.xpk, e);
        }
        EpiGelu<float> e{(float*)a.out, a.bias, a.ldo, 0};
        return launch_f32(st, (const float*)a.X, a.ldx, a.M, (const float*)a.W, a.N, a.K, 1, e);
    }
    case EPI_PARTIAL: {
        EpiPartial e{(float*)a.out, a.ldo, a.split_stride};
        if (bf) return launch_bf16(st, (const bf16_t*)a.X, a.ldx, a.M, (const bf16_t*)a.W, a.N, a.K, a.splits, a.xpk, e);
        return launch_f32(st, (const float*)a.X, a.ldx, a.M, (const float*)a.W, a.N, a.K, a.splits, e);
    }
    case EPI_RESID: {
        // large-M bf16 products only, no K split
        if (!bf || a.splits != 1 || !gemm_resid_in_place(a.M, a.N) || a.N % 4) return hipErrorInvalidValue;
        EpiResid e{(float*)a.out, a.bias, a.ldo};
        return launch_bf16(st, (const bf16_t*)a.X, a.ldx, a.M, (const bf16_t*)a.W, a.N, a.K, 1, a.xpk, e);
    }
    case EPI_LOGITS: {
        EpiLogits e{(float*)a.out, a.bias, a.ldo, a.N};
        if (bf) return launch_bf16(st, (const bf16_t*)a.X, a.ldx, a.M, (const bf16_t*)a.W, a.N, a.K, 1, a.xpk, e);
        return launch_f32(st, (const float*)a.X, a.ldx, a.M, (const float*)a.W, a.N, a.K, 1, e);
    }
    }
    return hipErrorInvalidValue;
}

}  // namespace mtp
