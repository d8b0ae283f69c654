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

// zidx: the index field given to zeros and denormals (their mantissa bits never matter: every
// product with a zero is a signed zero, whatever table entry it reads).
__device__ __forceinline__ uint32_t amsim_decode(uint32_t u, int m, int shift, uint32_t zidx = 0u)
{
    const uint32_t e = (u >> 23) & 0xFFu;
    if (e == 0u) return (u & 0x80000000u) | zidx;                      // +-0 (denormals too)
    uint32_t head;
    if (e == 0xFFu)
        head = (u & 0xFF800000u) | ((u & 0x007FFFFFu) ? 0x00400000u : 0u);  // +-Inf / qNaN
    else
        head = u & 0xFF800000u;                                        // +-2^(E-127)
    const uint32_t idx = ((u >> (23 - m)) & ((1u << m) - 1u)) << shift;
    return head | idx;
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
constexpr int kStatSlots = 8192;  // most workgroups of a decode launch that records them

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

// Convolution geometry: batch, input height and width, input and output channels, kernel height
// and width, strides, top and left padding, output height and width.
struct ConvShape {
    int n, h, w, ci, co, kh, kw, sh, sw, pt, pl, oh, ow;
};

}  // namespace amsim_detail
