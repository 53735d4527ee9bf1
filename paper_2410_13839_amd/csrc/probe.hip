// Measurement probes behind the design of the decode path (libmtp_probe.so,
// a separate library: the decode library itself allocates nothing and
// never runs these).  They measure what a launch boundary costs and what the
// in-kernel alternatives cost, which decides whether a decode step is a
// chain of launches or one persistent kernel:
//
//  * mtp_probe_launch_floor: back-to-back launches of a kernel that stores
//    one value per thread, captured in a hipGraph and replayed;
//  * mtp_probe_stream: back-to-back launches that each read `bytes` bytes
//    (16-byte loads, a grid-stride loop), captured and replayed: a launch
//    plus one weight stream, the shape of an FFN2 GEMV;
//  * mtp_probe_flag_barrier: a grid barrier among co-resident workgroups
//    (cooperative launch) built from device-coherent flag stores and loads
//    only (no cache writeback or invalidate), every wait bounded: mode 0,
//    every workgroup polls every flag; mode 1, workgroup 0 polls them and
//    publishes one go word the others poll.  With `data`, each workgroup
//    also stores 256 bytes before its flag and checks a neighbour's after
//    the barrier (stale reads are counted).
//
//  * mtp_probe_xcc_map: the XCD (the XCC_ID hardware register) that each
//    workgroup of an ordinary launch runs on, to check the round-robin
//    dealing of workgroups to the 8 XCDs that the decode kernels' tile
//    mappings assume;
//  * mtp_probe_handoff: the latency of one producer -> consumer hand-off
//    between two co-resident workgroups (a ping-pong of data + flag), with
//    the workgroups on one XCD or on two, for each combination of the
//    stores' and the loads' cache bits (below): which of them make a store
//    of one CU visible to the loads of another, and how soon.
//  * mtp_probe_bf16_round: the gfx950 float -> bfloat16 conversion
//    instruction against round-to-nearest-even written out on the bits, for
//    every finite float (2^32 patterns less Inf / NaN).
//
// Each returns 0, or a negative value on a HIP error (its message on
// stderr).  All memory is allocated and freed inside the call.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>

namespace {

#define PCK(x)                                                                                  \
    do {                                                                                        \
        hipError_t e_ = (x);                                                                    \
        if (e_ != hipSuccess) {                                                                 \
            fprintf(stderr, "probe: %s at %s:%d\n", hipGetErrorString(e_), __FILE__, __LINE__); \
            return -1;                                                                          \
        }                                                                                       \
    } while (0)

__global__ void probe_store_kernel(float* out, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) out[i] = (float)i;
}

__global__ __launch_bounds__(1024) void probe_stream_kernel(const uint4* __restrict__ src, size_t n16, float* out) {
    uint32_t acc = 0;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x) {
        const uint4 v = src[i];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    // one store per workgroup that depends on every load (nothing is elided)
    if (acc == 0x9E3779B9u) out[blockIdx.x] = (float)acc;
}

constexpr int SPIN = 200000;     // bounded waits: about 0.1 s of polling at most

__device__ __forceinline__ void st_dev(unsigned* p, unsigned v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned ld_dev(const unsigned* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// err[0]: a wait ran out (the kernel then returns); err[1]: stale reads
template <int MODE, bool DATA>
__global__ __launch_bounds__(1024) void probe_flag_barrier_kernel(unsigned* flags, unsigned* go, unsigned* data,
                                                                  unsigned* err, int rounds) {
    const int nb = gridDim.x, bid = blockIdx.x, tid = threadIdx.x;
    __shared__ int bad;
    if (tid == 0) bad = 0;
    __syncthreads();
    for (int r = 1; r <= rounds; ++r) {
        if (DATA && tid < 64) st_dev(&data[((size_t)(r & 1) * nb + bid) * 64 + tid], (unsigned)(r * 1000 + bid));
        __builtin_amdgcn_s_waitcnt(0);          // this wave's stores are complete
        __syncthreads();                        // ... and every wave's
        if (tid == 0) st_dev(&flags[bid], (unsigned)r);
        if (tid < 64) {
            if (MODE == 0 || bid == 0) {
                int s = 0;
                while (true) {
                    bool ok = true;
                    for (int f = tid; f < nb; f += 64) ok &= ld_dev(&flags[f]) >= (unsigned)r;
                    if (__all(ok) || ++s >= SPIN) break;
                    __builtin_amdgcn_s_sleep(1);
                }
                if (s >= SPIN && tid == 0) {
                    bad = 1;
                    atomicExch(err, 1u);
                }
                if (MODE == 1 && tid == 0) st_dev(go, (unsigned)r);
            } else {
                int s = 0;
                while (ld_dev(go) < (unsigned)r && ++s < SPIN) __builtin_amdgcn_s_sleep(1);
                if (s >= SPIN && tid == 0) {
                    bad = 1;
                    atomicExch(err, 1u);
                }
            }
        }
        __syncthreads();
        if (bad) {
            // release the others: workgroup 0's go word (mode 1) and this
            // workgroup's flag move past every round, so every wait ends
            if (tid == 0) {
                st_dev(&flags[bid], 0x7FFFFFFFu);
                if (MODE == 1 && bid == 0) st_dev(go, 0x7FFFFFFFu);
            }
            return;
        }
        if (DATA && tid < 64) {
            const int nbr = (bid + 37) % nb;
            const unsigned v = ld_dev(&data[((size_t)(r & 1) * nb + nbr) * 64 + tid]);
            if (v != (unsigned)(r * 1000 + nbr)) atomicAdd(err + 1, 1u);
        }
    }
}

__device__ __forceinline__ unsigned xcc_id() {
    unsigned v;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
    return v & 0xFu;
}

__global__ void probe_xcc_kernel(unsigned* xcc, int spin) {
    if (threadIdx.x == 0) xcc[blockIdx.x] = xcc_id();
    // stay resident for a while, as a decode workgroup does
    for (int i = 0; i < spin; ++i) __builtin_amdgcn_s_sleep(8);
}

// Cache bits of the hand-off's stores (ST) and loads (LD); every load waits
// for its own data.
//   ST 0: plain; 1: sc0; 2: sc1 (device scope); 3: nt
//   LD 0: sc0; 1: plain after buffer_inv sc0 (the CU's L1 invalidated);
//      2: sc1 (device scope); 3: plain after buffer_inv sc1; 4: nt
template <int LD>
__device__ __forceinline__ unsigned ld_bits(const unsigned* p) {
    unsigned v;
    if constexpr (LD == 0)
        asm volatile("global_load_dword %0, %1, off sc0\n\ts_waitcnt vmcnt(0)" : "=v"(v) : "v"(p) : "memory");
    else if constexpr (LD == 1)
        asm volatile("buffer_inv sc0\n\tglobal_load_dword %0, %1, off\n\ts_waitcnt vmcnt(0)" : "=v"(v) : "v"(p) : "memory");
    else if constexpr (LD == 2)
        asm volatile("global_load_dword %0, %1, off sc1\n\ts_waitcnt vmcnt(0)" : "=v"(v) : "v"(p) : "memory");
    else if constexpr (LD == 3)
        asm volatile("buffer_inv sc1\n\tglobal_load_dword %0, %1, off\n\ts_waitcnt vmcnt(0)" : "=v"(v) : "v"(p) : "memory");
    else
        asm volatile("global_load_dword %0, %1, off nt\n\ts_waitcnt vmcnt(0)" : "=v"(v) : "v"(p) : "memory");
    return v;
}
template <int ST>
__device__ __forceinline__ void st_bits(unsigned* p, unsigned v) {
    if constexpr (ST == 0)
        asm volatile("global_store_dword %0, %1, off" : : "v"(p), "v"(v) : "memory");
    else if constexpr (ST == 1)
        asm volatile("global_store_dword %0, %1, off sc0" : : "v"(p), "v"(v) : "memory");
    else if constexpr (ST == 2)
        asm volatile("global_store_dword %0, %1, off sc1" : : "v"(p), "v"(v) : "memory");
    else
        asm volatile("global_store_dword %0, %1, off nt" : : "v"(p), "v"(v) : "memory");
}

// One wave per workgroup.  Workgroups b and b + stride form a pair (b with
// (b / stride) even is the pinger).  Round r: the pinger stores 64 data
// words and, once they are complete, its flag r; the ponger waits for the
// flag, checks the data words and stores its own flag r, which the pinger
// waits for.  err[0]: waits that ran out (the workgroup then stops, and its
// partner's next wait runs out too); err[1]: stale data words; err[2]:
// pairs on one XCD.
template <int ST, int LD>
__global__ __launch_bounds__(64) void probe_handoff_kernel(unsigned* flags, unsigned* data, unsigned* err, int stride,
                                                           int rounds) {
    const int b = blockIdx.x, lane = threadIdx.x;
    const bool ping = ((b / stride) & 1) == 0;
    const int pair = (b / (2 * stride)) * stride + b % stride;
    unsigned* f_ab = flags + pair * 128;         // separate 256-byte blocks
    unsigned* f_ba = f_ab + 64;
    unsigned* dp = data + pair * 64 + lane;
    if (ping && lane == 0) {
        // the pair's XCDs, compared once
        st_bits<2>(&flags[64 * 128 + b], xcc_id());
    }
    for (int r = 1; r <= rounds; ++r) {
        if (ping) {
            st_bits<ST>(dp, (unsigned)(r * 1000 + lane));
            __builtin_amdgcn_s_waitcnt(0);
            if (lane == 0) st_bits<ST>(f_ab, (unsigned)r);
            int s = 0;
            while (ld_bits<LD>(f_ba) < (unsigned)r && ++s < SPIN) __builtin_amdgcn_s_sleep(1);
            if (s >= SPIN) {
                if (lane == 0) atomicAdd(err, 1u);
                return;
            }
        } else {
            int s = 0;
            while (ld_bits<LD>(f_ab) < (unsigned)r && ++s < SPIN) __builtin_amdgcn_s_sleep(1);
            if (s >= SPIN) {
                if (lane == 0) atomicAdd(err, 1u);
                return;
            }
            if (ld_bits<LD>(dp) != (unsigned)(r * 1000 + lane)) atomicAdd(err + 1, 1u);
            if (lane == 0) st_bits<ST>(f_ba, (unsigned)r);
        }
    }
    if (!ping && lane == 0) {
        const unsigned mine = xcc_id();
        // the pinger stored its XCD before its first flag, which this
        // workgroup has seen (or the round loop ended on a timeout)
        if (ld_bits<2>(&flags[64 * 128 + b - stride]) == mine) atomicAdd(err + 2, 1u);
    }
}

// round to nearest even on the bits (finite inputs)
__device__ __forceinline__ uint32_t bf16_rne_bits(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return u >> 16;
}

__global__ __launch_bounds__(256) void probe_bf16_kernel(unsigned long long* out) {
    unsigned long long mism = 0, checked = 0;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < (1ull << 32); i += stride) {
        const uint32_t u = (uint32_t)i;
        if (((u >> 23) & 0xFFu) == 0xFFu) continue;   // Inf, NaN
        const float f = __uint_as_float(u);
        const uint32_t h = __builtin_bit_cast(uint16_t, (__bf16)f);
        ++checked;
        mism += h != bf16_rne_bits(f);
    }
    atomicAdd(&out[0], mism);
    atomicAdd(&out[1], checked);
}

template <class F>
int time_graph(hipStream_t st, int launches, F launch_one, double* us) {
    hipGraph_t g;
    hipGraphExec_t ge;
    PCK(hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal));
    for (int i = 0; i < launches; ++i) launch_one();
    PCK(hipStreamEndCapture(st, &g));
    PCK(hipGraphInstantiate(&ge, g, nullptr, nullptr, 0));
    for (int w = 0; w < 3; ++w) PCK(hipGraphLaunch(ge, st));
    PCK(hipStreamSynchronize(st));
    hipEvent_t a, b;
    PCK(hipEventCreate(&a));
    PCK(hipEventCreate(&b));
    const int reps = 10;
    PCK(hipEventRecord(a, st));
    for (int w = 0; w < reps; ++w) PCK(hipGraphLaunch(ge, st));
    PCK(hipEventRecord(b, st));
    PCK(hipEventSynchronize(b));
    float ms = 0.f;
    PCK(hipEventElapsedTime(&ms, a, b));
    *us = (double)ms * 1000.0 / ((double)reps * launches);
    PCK(hipEventDestroy(a));
    PCK(hipEventDestroy(b));
    PCK(hipGraphExecDestroy(ge));
    PCK(hipGraphDestroy(g));
    return 0;
}

template <int ST, int LD>
const void* handoff_fn() { return (const void*)probe_handoff_kernel<ST, LD>; }
template <int ST>
const void* handoff_fn_ld(int ld) {
    switch (ld) {
    case 0: return handoff_fn<ST, 0>();
    case 1: return handoff_fn<ST, 1>();
    case 2: return handoff_fn<ST, 2>();
    case 3: return handoff_fn<ST, 3>();
    default: return handoff_fn<ST, 4>();
    }
}

}  // namespace

extern "C" {

int mtp_probe_launch_floor(int grid, int block, int launches, double* us_per_launch) {
    if (grid < 1 || block < 1 || block > 1024 || launches < 1 || !us_per_launch) return -2;
    float* out = nullptr;
    hipStream_t st;
    PCK(hipMalloc(&out, (size_t)grid * block * sizeof(float)));
    PCK(hipStreamCreate(&st));
    const int n = grid * block;
    const int rc = time_graph(st, launches, [&] {
        hipLaunchKernelGGL(probe_store_kernel, dim3(grid), dim3(block), 0, st, out, n);
    }, us_per_launch);
    PCK(hipStreamDestroy(st));
    PCK(hipFree(out));
    return rc;
}

int mtp_probe_stream(int grid, uint64_t bytes, int launches, double* us_per_launch) {
    if (grid < 1 || bytes < 16 || bytes % 16 || launches < 1 || !us_per_launch) return -2;
    // `launches` separate buffers, so each launch streams its own bytes
    // from HBM as a decode step's projections stream their own weights
    const size_t total = (size_t)bytes * launches;
    char* src = nullptr;
    float* out = nullptr;
    hipStream_t st;
    PCK(hipMalloc(&src, total));
    PCK(hipMemset(src, 1, total));
    PCK(hipMalloc(&out, (size_t)grid * sizeof(float)));
    PCK(hipStreamCreate(&st));
    int i = 0;
    const int rc = time_graph(st, launches, [&] {
        const uint4* p = reinterpret_cast<const uint4*>(src + (size_t)(i++) * bytes);
        hipLaunchKernelGGL(probe_stream_kernel, dim3(grid), dim3(1024), 0, st, p, (size_t)(bytes / 16), out);
    }, us_per_launch);
    PCK(hipStreamDestroy(st));
    PCK(hipFree(src));
    PCK(hipFree(out));
    return rc;
}

int mtp_probe_flag_barrier(int mode, int data, int rounds, double* us_per_barrier, uint32_t* timeouts,
                           uint32_t* stale) {
    if ((mode != 0 && mode != 1) || rounds < 1 || !us_per_barrier || !timeouts || !stale) return -2;
    int dev = 0, coop = 0, occ = 0, n_cu = 0;
    PCK(hipGetDevice(&dev));
    PCK(hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev));
    PCK(hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev));
    const void* fn = mode == 0 ? (data ? (const void*)probe_flag_barrier_kernel<0, true> : (const void*)probe_flag_barrier_kernel<0, false>)
                               : (data ? (const void*)probe_flag_barrier_kernel<1, true> : (const void*)probe_flag_barrier_kernel<1, false>);
    PCK(hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, 1024, 0));
    if (!coop || occ < 1 || n_cu < 1) return -3;      // every workgroup must be resident at once
    const int nb = n_cu;                              // one workgroup per CU
    unsigned *flags = nullptr, *go = nullptr, *buf = nullptr, *err = nullptr;
    PCK(hipMalloc(&flags, (size_t)nb * 4));
    PCK(hipMalloc(&go, 256));
    PCK(hipMalloc(&buf, (size_t)2 * nb * 64 * 4));
    PCK(hipMalloc(&err, 8));
    PCK(hipMemset(flags, 0, (size_t)nb * 4));
    PCK(hipMemset(go, 0, 256));
    PCK(hipMemset(buf, 0, (size_t)2 * nb * 64 * 4));
    PCK(hipMemset(err, 0, 8));
    PCK(hipDeviceSynchronize());
    void* args[] = {&flags, &go, &buf, &err, &rounds};
    hipEvent_t a, b;
    PCK(hipEventCreate(&a));
    PCK(hipEventCreate(&b));
    PCK(hipEventRecord(a, 0));
    PCK(hipLaunchCooperativeKernel(fn, dim3(nb), dim3(1024), args, 0, 0));
    PCK(hipEventRecord(b, 0));
    PCK(hipEventSynchronize(b));
    float ms = 0.f;
    PCK(hipEventElapsedTime(&ms, a, b));
    unsigned h[2];
    PCK(hipMemcpy(h, err, 8, hipMemcpyDeviceToHost));
    *us_per_barrier = (double)ms * 1000.0 / rounds;
    *timeouts = h[0];
    *stale = h[1];
    PCK(hipEventDestroy(a));
    PCK(hipEventDestroy(b));
    PCK(hipFree(flags));
    PCK(hipFree(go));
    PCK(hipFree(buf));
    PCK(hipFree(err));
    return 0;
}

int mtp_probe_bf16_round(uint64_t* mismatches, uint64_t* checked) {
    if (!mismatches || !checked) return -2;
    unsigned long long* d = nullptr;
    PCK(hipMalloc(&d, 16));
    PCK(hipMemset(d, 0, 16));
    hipLaunchKernelGGL(probe_bf16_kernel, dim3(2048), dim3(256), 0, 0, d);
    PCK(hipGetLastError());
    unsigned long long h[2];
    PCK(hipMemcpy(h, d, 16, hipMemcpyDeviceToHost));
    PCK(hipFree(d));
    *mismatches = h[0];
    *checked = h[1];
    return 0;
}

int mtp_probe_xcc_map(int grid, int block, uint32_t* xcc_out) {
    if (grid < 1 || grid > 65536 || block < 1 || block > 1024 || !xcc_out) return -2;
    unsigned* xcc = nullptr;
    PCK(hipMalloc(&xcc, (size_t)grid * 4));
    PCK(hipMemset(xcc, 0xFF, (size_t)grid * 4));
    hipLaunchKernelGGL(probe_xcc_kernel, dim3(grid), dim3(block), 0, 0, xcc, 64);
    PCK(hipGetLastError());
    PCK(hipDeviceSynchronize());
    PCK(hipMemcpy(xcc_out, xcc, (size_t)grid * 4, hipMemcpyDeviceToHost));
    PCK(hipFree(xcc));
    return 0;
}

int mtp_probe_handoff(int st_bits_sel, int ld_bits_sel, int stride, int rounds, double* us_per_handoff,
                      uint32_t* timeouts, uint32_t* stale, uint32_t* pairs_same_xcd) {
    if (st_bits_sel < 0 || st_bits_sel > 3 || ld_bits_sel < 0 || ld_bits_sel > 4 || (stride != 1 && stride != 8) ||
        rounds < 1 || !us_per_handoff || !timeouts || !stale || !pairs_same_xcd)
        return -2;
    int dev = 0, coop = 0;
    PCK(hipGetDevice(&dev));
    PCK(hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev));
    if (!coop) return -3;                            // both sides of a pair must be resident at once
    const int nb = 16;                               // 8 pairs
    unsigned *flags = nullptr, *data = nullptr, *err = nullptr;
    const size_t fbytes = (size_t)(64 * 128 + nb) * 4;
    PCK(hipMalloc(&flags, fbytes));
    PCK(hipMalloc(&data, (size_t)8 * 64 * 4));
    PCK(hipMalloc(&err, 16));
    PCK(hipMemset(flags, 0, fbytes));
    PCK(hipMemset(data, 0, (size_t)8 * 64 * 4));
    PCK(hipMemset(err, 0, 16));
    PCK(hipDeviceSynchronize());
    void* args[] = {&flags, &data, &err, &stride, &rounds};
    const void* fn = st_bits_sel == 0   ? handoff_fn_ld<0>(ld_bits_sel)
                     : st_bits_sel == 1 ? handoff_fn_ld<1>(ld_bits_sel)
                     : st_bits_sel == 2 ? handoff_fn_ld<2>(ld_bits_sel)
                                        : handoff_fn_ld<3>(ld_bits_sel);
    hipEvent_t a, b;
    PCK(hipEventCreate(&a));
    PCK(hipEventCreate(&b));
    PCK(hipEventRecord(a, 0));
    PCK(hipLaunchCooperativeKernel(fn, dim3(nb), dim3(64), args, 0, 0));
    PCK(hipEventRecord(b, 0));
    PCK(hipEventSynchronize(b));
    float ms = 0.f;
    PCK(hipEventElapsedTime(&ms, a, b));
    unsigned h[4];
    PCK(hipMemcpy(h, err, 16, hipMemcpyDeviceToHost));
    *us_per_handoff = (double)ms * 1000.0 / (2.0 * rounds);
    *timeouts = h[0];
    *stale = h[1];
    *pairs_same_xcd = h[2];
    PCK(hipEventDestroy(a));
    PCK(hipEventDestroy(b));
    PCK(hipFree(flags));
    PCK(hipFree(data));
    PCK(hipFree(err));
    return 0;
}

}  // extern "C"
