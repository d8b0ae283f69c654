// amsim_common.h -- types, constants and device helpers shared by the library's translation
// units: the pre-pass and host code (amsim_kernels.hip) and the table kernels (amsim_tab.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace amsim_detail __attribute__((visibility("hidden"))) {

constexpr uint32_t kIdxMask = 0x003FFFFFu;
constexpr uint32_t kHeadMask = 0xFFC00000u;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x3 __attribute__((ext_vector_type(3)));  // buffer_load_dwordx3 results only
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ------------------------------------------------------------------ device helpers -------

// The decode of one operand for a (1, e, m) multiplier (Sec. "AMSim": e can range from 1 to 8 given
// an exponent-casting function).  The cast maps an FP32 value into the e-bit format: fields
// [lo, hi] of the FP32 exponent are the format's normal range (unbiased exponents 1 - beta ..
// beta, beta = 2^(e-1) - 1); below it the value is a signed zero (the format's denormals read as
// zero, as Algorithm 2 reads FP32's); above it a signed Inf, or with `sat` the format's largest
// finite value (exponent beta, top-M mantissa bits all ones).  The head of a value in range has
// its exponent field lowered by `delta` = (127 - beta) / 2, so that the FP32 product of two
// heads underflows exactly when the e-bit exponent sum Ea + Eb - beta is <= 0 (Algorithm 2's zero
// rule in the format's constants).  e = 8 is the identity: lo = 1, hi = 254, delta = 0.
struct DecFmt {
    int m;          // mantissa bits of the table index (the paper's M)
    int shift;      // the index field's shift
    uint32_t zidx;  // index field of zeros
    int lo, hi;     // FP32 exponent fields of the format's normal range
    int delta;      // exponent offset of in-range heads
    int sat;        // overflow saturates to the largest finite value (else Inf)
    int raw;        // native multiply: operands kept as they are (no decode)
};

// Every case is formed and the right one selected, so that the decode passes run it without
// branches (measured on MI355X: the step's convolution decodes 5-9% faster than with a branch per
// case).
__device__ __forceinline__ uint32_t amsim_decode_fmt(uint32_t u, const DecFmt &f)
{
    if (f.raw) return u;
    const uint32_t e = (u >> 23) & 0xFFu, sign = u & 0x80000000u;
    const uint32_t mfield = ((1u << f.m) - 1u);
    const bool special = e == 0xFFu;
    const bool zero = e == 0u || (!special && int(e) < f.lo);  // +-0, denormals, underflow
    const bool over = !special && int(e) > f.hi;
    const uint32_t idx = ((u >> (23 - f.m)) & mfield) << f.shift;
    const uint32_t h_in = sign | (uint32_t(int(e) - f.delta) << 23);                   // +-2^(E-127-delta)
    const uint32_t h_special = (u & 0xFF800000u) | ((u & 0x007FFFFFu) ? 0x00400000u : 0u);  // +-Inf / qNaN
    const uint32_t over_word = f.sat ? (sign | (uint32_t(f.hi - f.delta) << 23) | (mfield << f.shift))
                                     : (sign | 0x7F800000u);
    const uint32_t r = over ? over_word : ((special ? h_special : h_in) | idx);
    return zero ? (sign | f.zidx) : r;
}

// The FP32 format (e = 8): the decode of Algorithm 2's operands as they are.
__host__ __device__ constexpr DecFmt fp32_fmt(int m, int shift, uint32_t zidx = 0u)
{
    return DecFmt{m, shift, zidx, 1, 254, 0, 0, 0};
}

// zidx: the index field given to zeros and denormals (their mantissa bits never matter: every
// product with a zero is a signed zero, whatever table entry it reads).
__device__ __forceinline__ uint32_t amsim_decode(uint32_t u, int m, int shift, uint32_t zidx = 0u)
{
    return amsim_decode_fmt(u, fp32_fmt(m, shift, zidx));
}

__device__ __forceinline__ float head_value(uint32_t w) { return __uint_as_float(w & kHeadMask); }

__device__ __forceinline__ float table_value(uint32_t entry)
{
    return __uint_as_float((entry & 0x00FFFFFFu) + 0x3F800000u);
}

template <int TM, int TN>
__device__ __forceinline__ void init_acc(float (&acc)[TM][TN])
{
#pragma unroll
    for (int r = 0; r < TM; ++r)
#pragma unroll
        for (int t = 0; t < TN; ++t) acc[r][t] = -0.0f;
}

__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// Exponent range of the operands a decode pass has seen, for the table kernels' bf16 path
// (which is exact only while no product can leave the normal range).  Finite non-zero operands
// count; zeros and denormals (read as zeros) do not.  One packed word per workgroup:
//   bits 0..7 smallest exponent field, 8..15 largest, bit 16 set if an Inf or NaN was seen.
constexpr int kStatSlots = 8192;  // most workgroups of a decode job that records them

struct ExpStats {
    uint32_t lo = 255u, hi = 0u, special = 0u;
    __device__ __forceinline__ void add(uint32_t u)
    {
        const uint32_t e = (u >> 23) & 0xFFu;
        if (e == 0xFFu) {
            special = 1u;
        } else if (e != 0u) {
            lo = min(lo, e);
            hi = max(hi, e);
        }
    }
};

__device__ __forceinline__ uint32_t wave_min(uint32_t v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = min(v, uint32_t(__shfl_xor(int(v), o)));
    return v;
}

__device__ __forceinline__ uint32_t wave_max(uint32_t v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, uint32_t(__shfl_xor(int(v), o)));
    return v;
}

// Workgroup reduction of the threads' statistics into stats[slot] (every thread of a workgroup
// of at most 1024 threads must call it).  Reduced within each wave first: same-address LDS
// atomics from every thread would serialise.  Once an Inf or NaN is seen the largest exponent no
// longer matters, so it travels with the special flag in one maximum.
__device__ __forceinline__ void store_stats(const ExpStats &s, uint32_t *stats, int slot)
{
    __shared__ uint32_t s_lo[16], s_hs[16];
    if (stats == nullptr) return;  // uniform: the whole launch records or none of it
    const uint32_t lo = wave_min(s.lo), hs = wave_max((s.special << 8) | s.hi);
    const int wave = int(threadIdx.x) >> 6, nwaves = int(blockDim.x + 63) >> 6;
    if ((threadIdx.x & 63) == 0) {
        s_lo[wave] = lo;
        s_hs[wave] = hs;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t l = 255u, h = 0u;
        for (int i = 0; i < nwaves; ++i) {
            l = min(l, s_lo[i]);
            h = max(h, s_hs[i]);
        }
        stats[slot] = l | ((h & 0xFFu) << 8) | ((h >> 8) << 16);
    }
}

// ------------------------------------------------------------------ table rows
constexpr int kTabRowEntries = 128;  // rows padded to 2^7 entries
// Table row kZeroRow (after the 2^M rows) holds zeros: the table path decodes second-operand
// zeros, and names padding steps, with its index, so that a zero's row needs no test.
constexpr int kZeroRow = kTabRowEntries;
constexpr uint32_t kZeroRowWord = uint32_t(kZeroRow) << 7;  // decoded +0 of the second operand

// A table entry as the factor v = 2^carry * 1.mantissa of the product: 1-byte entries hold the
// entry's bits 23..16 (carry and the top 7 mantissa bits), 2-byte entries bits 23..8, 4-byte
// entries the rebiased float itself.
template <int EB>
__device__ __forceinline__ float tab_value(const unsigned char *p)
{
    if constexpr (EB == 1)
        return __uint_as_float((uint32_t(*p) << 16) + 0x3F800000u);
    else if constexpr (EB == 2)
        return __uint_as_float((uint32_t(*reinterpret_cast<const uint16_t *>(p)) << 8) + 0x3F800000u);
    else
        return *reinterpret_cast<const float *>(p);
}

// The same factor times 2^k, vadd = k << 23 (0 <= k <= 126: v * 2^k stays finite).
template <int EB>
__device__ __forceinline__ float tab_value_scaled(const unsigned char *p, uint32_t vadd)
{
    if constexpr (EB == 1)
        return __uint_as_float((uint32_t(*p) << 16) + (0x3F800000u + vadd));
    else if constexpr (EB == 2)
        return __uint_as_float((uint32_t(*reinterpret_cast<const uint16_t *>(p)) << 8) + (0x3F800000u + vadd));
    else
        return __uint_as_float(*reinterpret_cast<const uint32_t *>(p) + vadd);
}

// Convolution geometry: batch, input height and width, input and output channels, kernel height
// and width, strides, top and left padding, output height and width.
struct ConvShape {
    int n, h, w, ci, co, kh, kw, sh, sw, pt, pl, oh, ow;
};

}  // namespace amsim_detail
