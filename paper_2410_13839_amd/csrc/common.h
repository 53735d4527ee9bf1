// Shared device-side definitions for the MTP decode kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define MTP_HEAD_DIM 64
#define MTP_MAX_HEADS_K 8      // prediction heads a step may use
#define MTP_MAX_TOPK 32
#define MTP_PREFILL_ROWS 64    // query rows per prefill attention tile (bf16)
#define MTP_ATTN_QT 8          // query rows per attention tile
#define MTP_SPLITK_MAX 8

typedef uint16_t bf16_t;  // raw bfloat16 bits

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Per-sequence decode state, device resident (int32 fields).
// x / d for 0 <= x < 2^20 and d >= 1: a float reciprocal estimate (error
// below 1/4 for such x) corrected by one step, so the quotient is exact.  The
// integer division the compiler emits for a run-time divisor costs ~40 VALU
// instructions per lane.
__device__ __forceinline__ int udiv_small(int x, int d) {
    int q = (int)((float)x * __builtin_amdgcn_rcpf((float)d));
    const int r = x - q * d;
    q += (r >= d) ? 1 : 0;
    q -= (r < 0) ? 1 : 0;
    return q;
}

struct SeqState {
    int32_t ctx_len;     // tokens whose K/V are in the cache
    int32_t pend_len;    // accepted tokens not yet run through the trunk
    int32_t gen;         // tokens emitted so far
    int32_t done;        // 1 once EOS was emitted or the budget is used
    int32_t phon_len;    // phoneme prefix length
    int32_t prompt_len;  // phonemes + acoustic prompt
    int32_t steps;       // decode steps taken
    int32_t last_tok;    // last emitted codec token (the prompt's last one before any), -1 if none
    int32_t pend_ids[MTP_MAX_HEADS_K];
};
static_assert(sizeof(SeqState) == 64, "SeqState layout");

// Row metadata of a packed activation row: sequence and absolute position
// (pos < 0 marks a padding row that must not touch the KV cache).
struct RowInfo {
    int32_t seq;
    int32_t pos;
};

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
    return __uint_as_float(((uint32_t)b) << 16);
}

// Round-to-nearest-even float -> bfloat16 bits, by gfx950's conversion
// instruction (v_cvt_pk_bf16_f32), which gives exactly the RNE result on the
// bits for every finite float (all 2^32 - 2^24 of them checked on the GPU).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
    return __builtin_bit_cast(uint16_t, (__bf16)f);
}
// Two floats -> two bfloat16 in one word (lo in the low half), one instruction.
__device__ __forceinline__ uint32_t bf16x2_bits(float lo, float hi) {
    typedef __bf16 b2_t __attribute__((ext_vector_type(2)));
    typedef float f2_t __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2_t){lo, hi}, b2_t));
}

// Split-K partial rows of the small-M projections (four K ranges, `rows`
// rows of `ld` floats each): [4][rows][ld] float32; or, for more than 4
// rows (partials_bf16), the first range, which carries the residual input
// and the bias, in float32 at `part` and ranges 1..3 in bfloat16 after it
// ([3][rows][ld]): the LayerNorm prologues that read all four then hold
// fewer registers, so that at 8 rows the chained FFN fits two workgroups
// per CU.  (At 4 rows and fewer the float32 form measured faster.)  The
// kernels take the form as a template argument BF = partials_bf16(rows).
__host__ __device__ __forceinline__ bool partials_bf16(int rows) { return rows > 4; }
template <bool BF>
__device__ __forceinline__ void store_partial4(float* part, int split, int rows, int ld, int m, int n,
                                               float4 o) {
    if (!BF || split == 0) {
        *reinterpret_cast<float4*>(part + ((size_t)split * rows + m) * ld + n) = o;
    } else {
        bf16_t* ph = reinterpret_cast<bf16_t*>(part + (size_t)rows * ld);
        *reinterpret_cast<uint2*>(ph + ((size_t)(split - 1) * rows + m) * ld + n) =
            make_uint2(bf16x2_bits(o.x, o.y), bf16x2_bits(o.z, o.w));
    }
}
// Range s of row m, columns c .. c + 3, as float32: range 0, or any range
// of the float32 form
__device__ __forceinline__ float4 load_partial_f32(const float* part, int s, int rows, int ld, int m, int c) {
    return *reinterpret_cast<const float4*>(part + ((size_t)s * rows + m) * ld + c);
}
// Range s (1..3) of row m of the bfloat16 form, columns c .. c + 3, as the
// raw bits (converted where the values are used, so the load needs no wait)
__device__ __forceinline__ uint2 load_partial_bits(const float* part, int s, int rows, int ld, int m, int c) {
    const bf16_t* ph = reinterpret_cast<const bf16_t*>(part + (size_t)rows * ld);
    return *reinterpret_cast<const uint2*>(ph + ((size_t)(s - 1) * rows + m) * ld + c);
}
__device__ __forceinline__ float4 bf16x4_to_f32(uint2 u) {
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u), __uint_as_float(u.y << 16),
                       __uint_as_float(u.y & 0xFFFF0000u));
}

// Element (row, k) of a bf16 activation matrix with K columns (K a multiple
// of 32) stored in MFMA fragment order, the order of the packed weights: 16 x
// 32 blocks of 1 KB, block (row / 16, k / 32) at ((row / 16) * (K / 32) +
// k / 32) * 512 elements, inside which lane r + 16 g holds row r's k = 8 g ..
// 8 g + 7.  A wave loads one block as one contiguous 1 KB read (row-major
// rows would be 16 separate 64-byte pieces).  Rows are padded to 16.
__device__ __forceinline__ size_t frag_off(int row, int k, int K) {
    return ((((size_t)(row >> 4) * (K >> 5) + (k >> 5)) * 64 + (row & 15) + 16 * ((k >> 3) & 3)) << 3) + (k & 7);
}

template <typename T> struct ActIO;
template <> struct ActIO<float> {
    __device__ static __forceinline__ float load(const float* p) { return *p; }
    __device__ static __forceinline__ void store(float* p, float v) { *p = v; }
};
template <> struct ActIO<bf16_t> {
    __device__ static __forceinline__ float load(const bf16_t* p) { return bf16_to_f32(*p); }
    __device__ static __forceinline__ void store(bf16_t* p, float v) { *p = f32_to_bf16(v); }
};

// erf by Abramowitz & Stegun, Handbook of Mathematical Functions, 7.1.26:
// erf(x) = 1 - (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) exp(-x^2),
// t = 1 / (1 + p x) for x >= 0, odd extension; |error| <= 1.5e-7, below one
// float32 ulp of GELU's 0.5 x (1 + erf) wherever that exceeds 1e-6 and far
// below the bf16 rounding of its output.  A quarter of the cost of the
// library erff in the GELU epilogues.
__device__ __forceinline__ float erf_as(float x) {
    const float ax = fabsf(x);
    const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, ax, 1.0f));
    float y = fmaf(1.061405429f, t, -1.453152027f);
    y = fmaf(y, t, 1.421413741f);
    y = fmaf(y, t, -0.284496736f);
    y = fmaf(y, t, 0.254829592f);
    const float r = 1.0f - (y * t) * __expf(-ax * ax);
    return copysignf(r, x);
}

// GELU with the Gaussian CDF, x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2)).
__device__ __forceinline__ float gelu_erf(float x) {
    return 0.5f * x * (1.0f + erf_as(x * 0.70710678118654752f));
}

// Paged KV addressing.  Pool layout: [layer][page][kv(0=K,1=V)][head][P*64]
// where the K block is [slot][64] (one key per row) and the V block is
// [slot][64] for fp32 caches but transposed, [64][slot], for bf16 caches, so
// that 8 consecutive keys of one dimension are one 16-byte MFMA operand.
struct KVView {
    void* pool;
    const int32_t* block_table;  // [batch][max_pages_per_seq]
    int32_t max_pages_per_seq;
    int32_t num_pages;
    int32_t page_size;           // power of two
    int32_t page_shift;
    int32_t n_heads;
    int32_t layer;

    __device__ __forceinline__ size_t offset(int seq, int pos, int kv, int head) const {
        int page = block_table[(size_t)seq * max_pages_per_seq + (pos >> page_shift)];
        int slot = pos & (page_size - 1);
        size_t base = (((size_t)layer * num_pages + page) * 2 + kv) * (size_t)n_heads;
        return ((base + head) * page_size + slot) * MTP_HEAD_DIM;
    }
    // element (dim) of the transposed V block of key `pos`: base + dim * page_size
    __device__ __forceinline__ size_t vt_offset(int seq, int pos, int head) const {
        int page = block_table[(size_t)seq * max_pages_per_seq + (pos >> page_shift)];
        int slot = pos & (page_size - 1);
        size_t base = (((size_t)layer * num_pages + page) * 2 + 1) * (size_t)n_heads;
        return (base + head) * page_size * MTP_HEAD_DIM + slot;
    }
};

// Element offset of the K (sec 0) or transposed V (sec 1) block of one head
// in cache page `page` (the page table already looked up).
__device__ __forceinline__ size_t kv_page_block(const KVView& kv, int page, int sec, int head) {
    return ((((size_t)kv.layer * kv.num_pages + page) * 2 + sec) * kv.n_heads + head) * (size_t)kv.page_size *
           MTP_HEAD_DIM;
}
