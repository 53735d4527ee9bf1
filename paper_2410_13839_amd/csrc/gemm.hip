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
//  * gemm_tiled_bf16: M > 256 (prefill).  LDS double-buffered
//    BMxBN tiles, BK = 64, 2x2 waves of v_mfma_f32_16x16x32_bf16.
//  * gemm_f32: the fp32 model; LDS-tiled VALU FMA.
#include "common.h"
#include "launch.h"

namespace mtp {

// ---------------------------------------------------------------- epilogues
template <typename KVT>
struct EpiQKV {
    float* q;            // [M][d] queries (fp32)
    const float* bias;   // [3d]
    const RowInfo* rows;
    KVView kv;
    int d;
    __device__ __forceinline__ void store4(int m, int n, const float (&v)[4], int, int) const {
        float r0 = v[0] + bias[n], r1 = v[1] + bias[n + 1], r2 = v[2] + bias[n + 2], r3 = v[3] + bias[n + 3];
        int sec = n / d;
        if (sec == 0) {
            *reinterpret_cast<float4*>(q + (size_t)m * d + n) = make_float4(r0, r1, r2, r3);
            return;
        }
        RowInfo ri = rows[m];
        if (ri.pos < 0) return;
        int c = n - sec * d;
        if constexpr (sizeof(KVT) == 2) {
            if (sec == 2) {   // transposed V block
                bf16_t* vt = reinterpret_cast<bf16_t*>(kv.pool) + kv.vt_offset(ri.seq, ri.pos, c >> 6);
                const int dim = c & 63;
                vt[(size_t)(dim + 0) * kv.page_size] = f32_to_bf16(r0);
                vt[(size_t)(dim + 1) * kv.page_size] = f32_to_bf16(r1);
                vt[(size_t)(dim + 2) * kv.page_size] = f32_to_bf16(r2);
                vt[(size_t)(dim + 3) * kv.page_size] = f32_to_bf16(r3);
                return;
            }
        }
        KVT* dst = reinterpret_cast<KVT*>(kv.pool) + kv.offset(ri.seq, ri.pos, sec - 1, c >> 6) + (c & 63);
        if constexpr (sizeof(KVT) == 2) {
            uint2 pk;
            pk.x = (uint32_t)f32_to_bf16(r0) | ((uint32_t)f32_to_bf16(r1) << 16);
            pk.y = (uint32_t)f32_to_bf16(r2) | ((uint32_t)f32_to_bf16(r3) << 16);
            *reinterpret_cast<uint2*>(dst) = pk;
        } else {
            *reinterpret_cast<float4*>(dst) = make_float4(r0, r1, r2, r3);
        }
    }
};

template <typename OutT>
struct EpiGelu {
    OutT* out;
    const float* bias;
    int ldo;
    int pk;               // bf16 output in fragment order (K = ldo)
    __device__ __forceinline__ void store4(int m, int n, const float (&v)[4], int, int) const {
        float r[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) r[i] = gelu_erf(v[i] + bias[n + i]);
        OutT* p = out + (pk ? frag_off(m, n, ldo) : (size_t)m * ldo + n);
        if constexpr (sizeof(OutT) == 2) {
            uint2 pk;
            pk.x = (uint32_t)f32_to_bf16(r[0]) | ((uint32_t)f32_to_bf16(r[1]) << 16);
            pk.y = (uint32_t)f32_to_bf16(r[2]) | ((uint32_t)f32_to_bf16(r[3]) << 16);
            *reinterpret_cast<uint2*>(p) = pk;
        } else {
            *reinterpret_cast<float4*>(p) = make_float4(r[0], r[1], r[2], r[3]);
        }
    }
};

struct EpiPartial {
    float* part;          // [split][M][ldo]
    int ldo;
    size_t split_stride;  // elements between splits
    __device__ __forceinline__ void store4(int m, int n, const float (&v)[4], int split, int) const {
        *reinterpret_cast<float4*>(part + split * split_stride + (size_t)m * ldo + n) =
            make_float4(v[0], v[1], v[2], v[3]);
    }
};

struct EpiLogits {
    float* out;           // [M][ldo]
    const float* bias;    // [N]
    int ldo;
    __device__ __forceinline__ void store4(int m, int n, const float (&v)[4], int, int nvalid) const {
        float* p = out + (size_t)m * ldo + n;
        for (int i = 0; i < nvalid; ++i) p[i] = v[i] + bias[n + i];
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

    __shared__ f32x4_t red[GM_NW][NT * MT][64];
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) red[wave][j * MT + mt][lane] = acc[j][mt];
    __syncthreads();
    for (int t = threadIdx.x; t < NT * MT * 64; t += 64 * GM_NW) {
        const int jm = t >> 6, l = t & 63;
        const int j = jm / MT, mt = jm - j * MT;
        f32x4_t s = red[0][jm][l];
#pragma unroll
        for (int w = 1; w < GM_NW; ++w) s += red[w][jm][l];
        const int m = m0 + 16 * mt + (l & 15);
        const int n = (nt0 + j) * 16 + 4 * (l >> 4);
        if (m < M && n < N) {
            float v[4] = {s[0], s[1], s[2], s[3]};
            epi.store4(m, n, v, split, min(4, N - n));
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
        hipLaunchKernelGGL((gemm_med_bf16<MT, NT, 4, XP, Epi>), grid, block, 0, st, X, ldx, M, W, N, K, kps, epi);
}

template <int MT, class Epi>
static void launch_med_x(hipStream_t st, const bf16_t* X, int ldx, int M, const bf16_t* W, int N, int K, int splits,
                         int xpk, Epi epi) {
    if (xpk) launch_med<MT, 1>(st, X, ldx, M, W, N, K, splits, epi);
    else launch_med<MT, 0>(st, X, ldx, M, W, N, K, splits, epi);
}

// ---------------------------------------------------------------- tiled bf16
template <int BM, int BN, class Epi>
__global__ __launch_bounds__(256) void gemm_tiled_bf16(const bf16_t* __restrict__ X, int ldx, int M,
                                                       const bf16_t* __restrict__ W, int N, int K,
                                                       int k_per_split, Epi epi) {
    constexpr int BK = 64;
    constexpr int LDSK = BK + 8;           // padded row (bf16 elements)
    constexpr int TM = BM / 32;            // 16-row MFMA tiles per wave along m
    constexpr int TN = BN / 32;            // along n
    constexpr int XCH = BM * BK / 8 / 256; // 16-byte chunks per thread per stage
    constexpr int WCH = BN * BK / 8 / 256;
    static_assert(XCH >= 1 && WCH >= 1, "tile too small");
    __shared__ __attribute__((aligned(16))) bf16_t Xs[2][BM][LDSK];
    __shared__ __attribute__((aligned(16))) bf16_t Ws[2][BN][LDSK];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = blockIdx.y * BM;
    const int n0 = blockIdx.x * BN;
    const int split = blockIdx.z;
    const int kb = split * k_per_split;
    const int nk = k_per_split / BK;

    uint4 xr[XCH], wr[WCH];
    auto gload = [&](int kt) {
        const int k0 = kb + kt * BK;
#pragma unroll
        for (int c = 0; c < XCH; ++c) {
            int ch = tid + c * 256;
            int row = ch >> 3, col = (ch & 7) * 8;
            int m = m0 + row;
            xr[c] = (m < M) ? *reinterpret_cast<const uint4*>(X + (size_t)m * ldx + k0 + col) : make_uint4(0, 0, 0, 0);
        }
        // W tile in the packed fragment order: each wave load is one 1 KB
        // fragment (16 rows x 32 columns); fragment t of the tile is row block
        // t / 2, column block t % 2 (the row-block test is uniform per wave)
#pragma unroll
        for (int c = 0; c < WCH; ++c) {
            const int ch = tid + c * 256;
            const int t = ch >> 6, l = ch & 63;
            const int rt = t >> 1, fk = t & 1;
            wr[c] = (n0 + rt * 16 < N)
                        ? *reinterpret_cast<const uint4*>(W + ((size_t)((n0 >> 4) + rt) * (K >> 5) + (k0 >> 5) + fk) * 512 + l * 8)
                        : make_uint4(0, 0, 0, 0);
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int c = 0; c < XCH; ++c) {
            int ch = tid + c * 256;
            *reinterpret_cast<uint4*>(&Xs[buf][ch >> 3][(ch & 7) * 8]) = xr[c];
        }
#pragma unroll
        for (int c = 0; c < WCH; ++c) {
            const int ch = tid + c * 256;
            const int t = ch >> 6, l = ch & 63;
            *reinterpret_cast<uint4*>(&Ws[buf][(t >> 1) * 16 + (l & 15)][(t & 1) * 32 + (l >> 4) * 8]) = wr[c];
        }
    };

    f32x4_t acc[TN][TM];
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
        for (int kk = 0; kk < BK / 32; ++kk) {
            bf16x8_t a[TN], b[TM];
#pragma unroll
            for (int i = 0; i < TN; ++i)
                a[i] = *reinterpret_cast<const bf16x8_t*>(&Ws[buf][wn * (BN / 2) + i * 16 + r][kk * 32 + g * 8]);
#pragma unroll
            for (int j = 0; j < TM; ++j)
                b[j] = *reinterpret_cast<const bf16x8_t*>(&Xs[buf][wm * (BM / 2) + j * 16 + r][kk * 32 + g * 8]);
#pragma unroll
            for (int i = 0; i < TN; ++i)
#pragma unroll
                for (int j = 0; j < TM; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) {
            sstore(buf ^ 1);
        }
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j) {
            const int n = n0 + wn * (BN / 2) + i * 16 + 4 * g;
            const int m = m0 + wm * (BM / 2) + j * 16 + r;
            if (m < M && n < N) {
                float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
                epi.store4(m, n, v, split, min(4, N - n));
            }
        }
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
    if (m < M && n < N) epi.store4(m, n, acc, split, min(4, N - n));
}

// ------------------------------------------------------------------ launchers
template <class Epi>
static hipError_t launch_bf16(hipStream_t st, const bf16_t* X, int ldx, int M, const bf16_t* W, int N, int K,
                              int splits, int xpk, Epi epi) {
    const int kps = K / splits;
    if (M <= 16) {
        launch_med_x<1>(st, X, ldx, M, W, N, K, splits, xpk, epi);
    } else if (M <= 32) {
        launch_med_x<2>(st, X, ldx, M, W, N, K, splits, xpk, epi);
    } else if (M <= 256) {
        launch_med_x<4>(st, X, ldx, M, W, N, K, splits, xpk, epi);
    } else {
        if (xpk) return hipErrorInvalidValue;
        dim3 grid((N + 127) / 128, (M + 127) / 128, splits);
        hipLaunchKernelGGL((gemm_tiled_bf16<128, 128, Epi>), grid, dim3(256), 0, st, X, ldx, M, W, N, K, kps, epi);
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
    if (dtype == 0) return 32;
    if (M <= 256) return 32;
    return 64;
}

// Workgroups of one bf16 launch for M rows and N columns before K splitting.
int gemm_tiles(int M, int N) {
    const int groups = ((N + 15) / 16 + GM_NT - 1) / GM_NT;
    if (M <= 32) return groups;
    if (M <= 256) return groups * ((M + 63) / 64);
    return ((N + 127) / 128) * ((M + 127) / 128);
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
    case EPI_LOGITS: {
        EpiLogits e{(float*)a.out, a.bias, a.ldo};
        if (bf) return launch_bf16(st, (const bf16_t*)a.X, a.ldx, a.M, (const bf16_t*)a.W, a.N, a.K, 1, a.xpk, e);
        return launch_f32(st, (const float*)a.X, a.ldx, a.M, (const float*)a.W, a.N, a.K, 1, e);
    }
    }
    return hipErrorInvalidValue;
}

}  // namespace mtp
