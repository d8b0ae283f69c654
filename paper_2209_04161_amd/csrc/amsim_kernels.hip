// amsim_kernels.hip -- HIP kernels for gfx950 and the device-side C entry points of the
// approximate-multiplier library (ApproxTrain's AMSim, arXiv 2209.04161, Algorithms 2-4).
//
// How a product is evaluated (Algorithm 2, rewritten for the vector ALU):
//   Each operand is decoded once into a 32-bit word
//     head (bits 31..22): sign | exponent field | quiet-NaN bit   (mantissa cleared)
//     idx  (bits 21..0) : the operand's top-M mantissa bits, pre-shifted into its part of
//                         the table offset
//   head read as a float is +-2^(E-127) for a normal operand, +-0 for a zero/denormal one,
//   +-Inf or NaN for the specials.  The product is
//     c = v * (pa * pb),   v = float((entry & 0xFFFFFF) + 0x3F800000) = 2^carry * 1.mantissa
//   with f32 denormals flushed to zero: pa*pb underflows to a signed zero exactly when
//   Ea + Eb - 127 <= 0 (the zero rule, before the carry), overflows to a signed Inf when it
//   is >= 255, and v * (pa*pb) is exact, or Inf when the carry lifts the exponent to 255.
//   IEEE arithmetic gives the NaN/Inf policy for special operands.  Where the operands'
//   exponents rule that last case out (Ea + Eb <= 380 for every finite pair, known from the
//   decode statistics), the sum uses fma(v, pa*pb, acc), which then equals acc + c rounded once;
//   otherwise c is rounded on its own first, so that an overflowing product is Inf whatever the
//   sum it is added to.
//
// The table kernels (the hot path) live in amsim_tab.h / amsim_tab.hip; this file holds the
// decode and table-preparation pre-passes, the split reduction, the direct-evaluation GEMM,
// the host-side planning and the C entry points.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <iterator>
#include <mutex>
#include <type_traits>
#include <vector>

#include "amsim.h"

#include "amsim_plan.h"
#include "amsim_tab.h"

namespace {

using namespace amsim_detail;

// ------------------------------------------------------------------ pre-pass kernels -----

// r / d for 0 <= r and 1 <= d, given inv_d = 1.0f / d.  Below 2^24 (small, uniform) the float
// quotient is within one of the true one, which a remainder test corrects; above, the integer
// division.
__device__ __forceinline__ int div_small(int r, int d, float inv_d, bool small)
{
    if (!small) return r / d;
    int q = int(float(r) * inv_d);
    const int rem = r - q * d;
    if (rem < 0)
        --q;
    else if (rem >= d)
        ++q;
    return q;
}

// A step-pair record from the decoded words of its two steps: {index field of the first, the two
// heads as bf16 (the first in the low half), index field of the second}; with raw operands
// (native multiply) {first, 0, second}.
__device__ __forceinline__ void store_record(uint32_t *d, uint32_t w0, uint32_t w1, int raw)
{
    d[0] = raw ? w0 : (w0 & 0xFFFFu);
    d[1] = raw ? 0u : ((w0 >> 16) | (w1 & 0xFFFF0000u));
    d[2] = raw ? w1 : (w1 & 0xFFFFu);
}

// The pre-pass jobs below are workgroup bodies: `bid` of `nblk` workgroups of 256 threads take
// the place of blockIdx.x and gridDim.x (see prepass_kernel).

// The second operand's decode, dst[(b * rows + r) * dld + c] = decode(src[b * sb + r * sr + c * sc])
// for r < vrows, c < cols; padding columns c in [cols, dld) and padding rows r in [vrows, rows)
// (whose source is not read) are written as decoded +0.  dld is a multiple of 4 and
// batches * rows * dld / 4 < 2^31: each thread takes groups of 4 columns (16-byte stores), two
// groups per iteration so that 8 loads are in flight.  vec: sc == 1 and every row start is
// 16-byte aligned, so a full group is one 16-byte load.
struct DecRows {
    const float *src;
    int64_t sb, sr, sc;
    int batches, rows, vrows, cols;
    uint32_t *dst;
    int dld;
    int vec;
};

__device__ __forceinline__ void decode_rows_body(const DecRows &d, DecFmt f, uint32_t *__restrict__ stats, uint32_t bid,
                                                 uint32_t nblk)
{
    const float *__restrict__ src = d.src;
    uint32_t *__restrict__ dst = d.dst;
    const int64_t sb = d.sb, sr = d.sr, sc = d.sc;
    const int rows = d.rows, vrows = d.vrows, cols = d.cols, dld = d.dld, vec = d.vec;
    const uint32_t qpr = uint32_t(dld) / 4u;
    const uint32_t total = uint32_t(d.batches) * uint32_t(rows) * qpr;
    const uint32_t step = nblk * 256u;
    ExpStats st;
    for (uint32_t q0 = bid * 256u + threadIdx.x; q0 < total; q0 += 2u * step) {
        uint32_t w[2][4];
        uint32_t row[2], c[2];
        bool live[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const uint32_t q = q0 + uint32_t(h) * step;
            live[h] = q < total;
            row[h] = live[h] ? q / qpr : 0u;
            c[h] = (q - row[h] * qpr) * 4u;
            const uint32_t b = row[h] / uint32_t(rows), r = row[h] - b * uint32_t(rows);
            const float *base = src + int64_t(b) * sb + int64_t(r) * sr;
            const uint32_t ncols = r < uint32_t(vrows) ? uint32_t(cols) : 0u;
            if (vec && live[h] && c[h] + 4u <= ncols) {
                const u32x4 q4 = *reinterpret_cast<const u32x4 *>(base + c[h]);
#pragma unroll
                for (int e = 0; e < 4; ++e) w[h][e] = q4[e];
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t ce = c[h] + uint32_t(e);
                    w[h][e] = (live[h] && ce < ncols) ? __float_as_uint(base[int64_t(ce) * sc]) : 0u;
                }
            }
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            if (!live[h]) continue;
            u32x4 o;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                // padding columns and +0 operands both decode to 0 and leave the statistics alone
                st.add(w[h][e]);
                o[e] = amsim_decode_fmt(w[h][e], f);
            }
            *reinterpret_cast<u32x4 *>(dst + int64_t(row[h]) * dld + c[h]) = o;
        }
    }
    store_stats(st, stats, int(bid));
}

// The backward-weight pass's first operand: the NHWC tensor inside its zero border as step-pair
// records [n][hp][wp][c], record (b, y, x, ci) = the record of the decoded elements at columns x and
// x + sw of padded row y (a column past the border, or outside x, a decoded +0).  A workgroup takes
// one padded image row at a time; consecutive threads write consecutive records.  With row_lds
// (rows of at most kPairsRowWords elements) the row is decoded once into LDS, with 16-byte loads
// where vec allows, and the records are read from there (measured on MI355X: the ResNet 3x3
// decode 19% faster than with each element loaded from memory for both of its records).
constexpr int kPairsRowWords = 8192;

struct DecPairs {
    const float *src;
    int n, h, w, c, top, left, hp, wp, sw;
    uint32_t *dst;
    int row_lds, vec;
};

__device__ __forceinline__ void decode_a_body(const DecPairs &d, DecFmt f, uint32_t *__restrict__ stats, int bid,
                                              int nblk)
{
    const float *__restrict__ src = d.src;
    uint32_t *__restrict__ dst = d.dst;
    const int n = d.n, h = d.h, w = d.w, c = d.c, top = d.top, left = d.left, hp = d.hp, wp = d.wp, sw = d.sw;
    const int len = wp * c;
    const float inv_c = 1.0f / float(c);
    const bool small = len < (1 << 24);
    ExpStats st;
    if (d.row_lds) {  // uniform
        extern __shared__ uint32_t row[];  // w * c decoded words (the launch sizes it)
        const int wc = w * c;
        for (int rr = bid; rr < n * hp; rr += nblk) {
            const int b = rr / hp, y = rr - b * hp, ih = y - top;
            const bool inside = unsigned(ih) < unsigned(h);  // uniform over the workgroup
            const float *srow = src + (int64_t(b) * h + ih) * w * c;
            uint32_t *drow = dst + int64_t(rr) * len * 3;
            __syncthreads();  // the previous row's records have read the row
            if (inside) {
                if (d.vec) {
                    for (int g = threadIdx.x; g < wc / 4; g += 256) {
                        const u32x4 v = reinterpret_cast<const u32x4 *>(srow)[g];
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
                            st.add(v[k]);
                            row[4 * g + k] = amsim_decode_fmt(v[k], f);
                        }
                    }
                } else {
                    for (int e = threadIdx.x; e < wc; e += 256) {
                        const uint32_t v = __float_as_uint(srow[e]);
                        st.add(v);
                        row[e] = amsim_decode_fmt(v, f);
                    }
                }
            }
            __syncthreads();
            for (int i = threadIdx.x; i < len; i += 256) {
                const int x = div_small(i, c, inv_c, small), ci = i - x * c, x1 = x + sw;
                const int ix0 = x - left, ix1 = x1 - left;
                uint32_t w0 = 0u, w1 = 0u;
                if (inside) {
                    if (unsigned(ix0) < unsigned(w)) w0 = row[ix0 * c + ci];
                    if (x1 < wp && unsigned(ix1) < unsigned(w)) w1 = row[ix1 * c + ci];
                }
                store_record(drow + int64_t(i) * 3, w0, w1, f.raw);
            }
        }
        store_stats(st, stats, bid);
        return;
    }
    for (int rr = bid; rr < n * hp; rr += nblk) {
        const int b = rr / hp, y = rr - b * hp, ih = y - top;
        const bool inside = unsigned(ih) < unsigned(h);  // uniform over the workgroup
        const float *srow = src + (int64_t(b) * h + ih) * w * c;
        uint32_t *drow = dst + int64_t(rr) * len * 3;
        for (int i = threadIdx.x; i < len; i += 256) {
            const int x = div_small(i, c, inv_c, small), ci = i - x * c, x1 = x + sw;
            const int ix0 = x - left, ix1 = x1 - left;
            uint32_t u0 = 0u, u1 = 0u;
            if (inside) {
                if (unsigned(ix0) < unsigned(w)) u0 = __float_as_uint(srow[ix0 * c + ci]);
                if (x1 < wp && unsigned(ix1) < unsigned(w)) u1 = __float_as_uint(srow[ix1 * c + ci]);
            }
            st.add(u0);  // every element is the first of exactly one record
            store_record(drow + int64_t(i) * 3, amsim_decode_fmt(u0, f), amsim_decode_fmt(u1, f), f.raw);
        }
    }
    store_stats(st, stats, bid);
}

// Decoded NHWC tensor as step-pair records [n][hp][cp][wp] (cp = ceil(c / 2)) inside a zero
// border: record (b, y, q, x) = {index word of channel 2q, heads of channels 2q and 2q + 1 as bf16
// (2q in the low half), index word of channel 2q + 1} of pixel (y - top, x - left) where it
// exists, zeros elsewhere; a channel past the end is a decoded +0.  A workgroup takes one padded
// image row at a time: the source row (w pixels x cc channels at a time, cc even, contiguous
// loads) goes through LDS as [channel][x] (row pitch w | 1, odd, so the transposing stores do not
// collide in banks), then the workgroup writes the chunk's records, one per thread.  With vec
// (c and cc multiples of 4, a 16-byte aligned source) each load takes four channels of a pixel
// (measured on MI355X: the ResNet 3x3 decode 14% faster than with single-channel loads).

struct DecNhcw {
    const float *src;
    int n, h, w, c, top, left, hp, wp;
    uint32_t *dst;
    int cc, cp;
    int vec;
};

__device__ __forceinline__ void decode_a_body(const DecNhcw &d, DecFmt f, uint32_t *__restrict__ stats, int bid,
                                              int nblk)
{
    extern __shared__ uint32_t tile[];  // cc * (w | 1) words (the launch sizes it)
    const float *__restrict__ src = d.src;
    uint32_t *__restrict__ dst = d.dst;
    const int n = d.n, h = d.h, w = d.w, c = d.c, top = d.top, left = d.left, hp = d.hp, wp = d.wp;
    const int cc = d.cc, cp = d.cp;
    const int ws = w | 1;
    const int nch = (c + cc - 1) / cc;  // channel chunks per row: a work item is (padded row, chunk)
    ExpStats st;
    for (int item = bid; item < n * hp * nch; item += nblk) {
        const int rr = item / nch, c0 = (item - rr * nch) * cc;
        const int b = rr / hp, y = rr - b * hp, ih = y - top;
        const int ccn = min(cc, c - c0), qn = (ccn + 1) / 2;
        // the chunk's records are one contiguous block [q][x] of the row's [cp][wp] records
        uint32_t *dblk = dst + (int64_t(rr) * cp + c0 / 2) * wp * 3;
        if (unsigned(ih) >= unsigned(h)) {  // a padding row (uniform over the workgroup)
            for (int i = threadIdx.x; i < qn * wp * 3; i += 256) dblk[i] = 0u;
            continue;
        }
        const float *srow = src + (int64_t(b) * h + ih) * w * c;
        {
            __syncthreads();  // the previous item's stores have read the tile
            if (d.vec) {  // groups of four channels (uniform)
                const int g4 = ccn / 4, cnt = w * g4;
                const float inv_g4 = 1.0f / float(g4);
                for (int e0 = threadIdx.x; e0 < cnt; e0 += 256 * 4) {
                    u32x4 v[4];
                    int x[4], ch[4];
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const int e = e0 + 256 * k;
                        x[k] = div_small(e, g4, inv_g4, true);
                        ch[k] = 4 * (e - x[k] * g4);
                        v[k] = e < cnt ? *reinterpret_cast<const u32x4 *>(srow + x[k] * c + c0 + ch[k])
                                       : u32x4{0u, 0u, 0u, 0u};
                    }
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        if (e0 + 256 * k >= cnt) break;
#pragma unroll
                        for (int t = 0; t < 4; ++t) {
                            st.add(v[k][t]);
                            tile[(ch[k] + t) * ws + x[k]] = amsim_decode_fmt(v[k][t], f);
                        }
                    }
                }
            } else {
                const int cnt = w * ccn;
                const float inv_ccn = 1.0f / float(ccn);
                for (int e0 = threadIdx.x; e0 < cnt; e0 += 256 * 8) {
                    uint32_t v[8];
                    int x[8], ch[8];
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        const int e = e0 + 256 * k;
                        x[k] = div_small(e, ccn, inv_ccn, true);
                        ch[k] = e - x[k] * ccn;
                        v[k] = e < cnt ? __float_as_uint(srow[x[k] * c + c0 + ch[k]]) : 0u;
                    }
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        if (e0 + 256 * k >= cnt) break;
                        st.add(v[k]);
                        tile[ch[k] * ws + x[k]] = amsim_decode_fmt(v[k], f);
                    }
                }
            }
            __syncthreads();
            // consecutive threads write consecutive records
            const float inv_wp = 1.0f / float(wp);
            const bool small = qn * wp < (1 << 24);
            for (int rec = threadIdx.x; rec < qn * wp; rec += 256) {
                const int q = div_small(rec, wp, inv_wp, small), x = rec - q * wp, ix = x - left;
                uint32_t w0 = 0u, w1 = 0u;
                if (unsigned(ix) < unsigned(w)) {
                    w0 = tile[(2 * q) * ws + ix];
                    w1 = 2 * q + 1 < ccn ? tile[(2 * q + 1) * ws + ix] : 0u;
                }
                store_record(dblk + int64_t(rec) * 3, w0, w1, f.raw);
            }
        }
    }
    store_stats(st, stats, bid);
}

// Forward pass with few input channels: x unfolded along w into the step-pair records of a
// virtual input x'[n][y][ow][kw * c + ci] = x[n][y - top][ow * sw + kw - left][ci] (zero outside
// x), laid out [n][hp][cp'][ow_n] (cp' = ceil(kw_n * c / 2)) like the DecNhcw decode's
// records; an odd kw_n * c leaves a padding channel, written as -0.  The forward pass of a
// kh x kw kernel over x is then a sum over (kh, kw * c) steps whose records lie at one stride
// (the host's unfolded_shape).  A workgroup takes one padded image row at a time and stages the
// decoded source row (w * c <= kNhcwTile words) in LDS.
struct DecUnfold {
    const float *src;
    int n, h, w, c, top, left, hp, kw_n, sw, ow_n;
    uint32_t *dst;
};

__device__ __forceinline__ void decode_a_body(const DecUnfold &d, DecFmt f, uint32_t *__restrict__ stats, int bid,
                                              int nblk)
{
    extern __shared__ uint32_t tile[];  // w * c words (the launch sizes it)
    const float *__restrict__ src = d.src;
    uint32_t *__restrict__ dst = d.dst;
    const int n = d.n, h = d.h, w = d.w, c = d.c, top = d.top, left = d.left, hp = d.hp, kw_n = d.kw_n, sw = d.sw,
              ow_n = d.ow_n;
    const int cu = kw_n * c, cp = (cu + 1) / 2;
    ExpStats st;
    for (int rr = bid; rr < n * hp; rr += nblk) {
        const int b = rr / hp, y = rr - b * hp, ih = y - top;
        uint32_t *dimg = dst + int64_t(rr) * cp * ow_n * 3;
        if (unsigned(ih) >= unsigned(h)) {  // a padding row (uniform over the workgroup): +0, and the
            // padding channel's -0 in the last channel pair
            for (int rec = threadIdx.x; rec < cp * ow_n; rec += 256)
                store_record(dimg + int64_t(rec) * 3, 0u, (cu & 1) && rec >= (cp - 1) * ow_n ? 0x80000000u : 0u, f.raw);
            continue;
        }
        const float *srow = src + (int64_t(b) * h + ih) * w * c;
        __syncthreads();  // the previous row's record stores have read the tile
        for (int e = threadIdx.x; e < w * c; e += 256) {
            const uint32_t v = __float_as_uint(srow[e]);
            st.add(v);
            tile[e] = amsim_decode_fmt(v, f);
        }
        __syncthreads();
        const float inv_own = 1.0f / float(ow_n);
        const bool small = cp * ow_n < (1 << 24);
        for (int rec = threadIdx.x; rec < cp * ow_n; rec += 256) {  // record (q, xo), consecutive per thread
            const int q = div_small(rec, ow_n, inv_own, small), xo = rec - q * ow_n;
            uint32_t wd[2] = {0u, 0u};
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const int j = 2 * q + t;  // = kw * c + ci
                const int k = j / c, ix = xo * sw + k - left;
                if (j >= cu)
                    wd[t] = 0x80000000u;  // the padding channel: a decoded -0
                else if (unsigned(ix) < unsigned(w))
                    wd[t] = tile[ix * c + (j - k * c)];
            }
            store_record(dimg + int64_t(rec) * 3, wd[0], wd[1], f.raw);
        }
    }
    store_stats(st, stats, bid);
}

// Backward data: the products of the padded, dilated error (Algorithm 4) that the stride-phase
// decomposition does not evaluate.  Every tap (kh, kw) of the kernel window contributes to every
// output; a tap outside the output's stride phase reads a dilation or padding zero, so it adds
// amul(+0, w[kh][kw][ci][co]) for every co: NaN when the weight, as the call's format casts it,
// is Inf or NaN (Inf x 0), else a zero whose sign is the weight's (so a +0 unless the sign bit
// is set).  Such products leave every sum but an exactly zero one (-0 turns into +0 when one
// of them is +0) and make it NaN when one of them is.  One word per (stride phase, ci) over the
// taps outside the phase and per (kw, ci) over all kh (for the w-unfolded pass's fold): bit 0 a
// NaN product, bit 1 a +0 product.  w is [KH][KW][CI][CO]; `hi` the largest finite exponent field of
// the format (values above it are Inf unless `sat`).
constexpr uint32_t kZeroNan = 1u, kZeroPos = 2u;

__device__ __forceinline__ uint32_t zero_product_class(uint32_t u, int hi, int sat)
{
    const int e = int((u >> 23) & 0xFFu);
    if (e == 0xFF || (!sat && e > hi)) return kZeroNan;
    return (u >> 31) ? 0u : kZeroPos;
}

// One workgroup per flag: its threads read the flag's weights (co innermost, contiguous) and OR
// their classes.
struct ZeroTapFlags {
    const float *w;
    int KH, KW, CI, CO, sh, sw, pt, pl, hi, sat;
    uint32_t *phase_flags, *kw_flags;
    int total() const { return (phase_flags ? sh * sw * CI : 0) + (kw_flags ? KW * CI : 0); }
};

__device__ __forceinline__ void zero_tap_flags_body(const ZeroTapFlags &z, int bid, int nblk)
{
    __shared__ uint32_t s_or[4];
    const int KH = z.KH, KW = z.KW, CI = z.CI, CO = z.CO, sh = z.sh, sw = z.sw, pt = z.pt, pl = z.pl;
    uint32_t *__restrict__ phase_flags = z.phase_flags;
    uint32_t *__restrict__ kw_flags = z.kw_flags;
    const int nphase = phase_flags ? sh * sw * CI : 0, total = nphase + (kw_flags ? KW * CI : 0);
    const uint32_t *wu = reinterpret_cast<const uint32_t *>(z.w);
    for (int t = bid; t < total; t += nblk) {
        uint32_t f = 0u;
        if (t < nphase) {  // every (kh, kw, co) outside the phase's taps
            const int ci = t % CI, phase = t / CI, ph = phase / sw, pw = phase % sw;
            for (int j = threadIdx.x; j < KH * KW * CO; j += 256) {
                const int co = j % CO, kk = j / CO, kh = kk / KW, kw = kk % KW;
                if ((kh - ph - pt) % sh == 0 && (kw - pw - pl) % sw == 0) continue;  // a tap of the phase
                f |= zero_product_class(wu[(int64_t(kk) * CI + ci) * CO + co], z.hi, z.sat);
            }
        } else {  // every (kh, co) of the kernel column
            const int ci = (t - nphase) % CI, kw = (t - nphase) / CI;
            for (int j = threadIdx.x; j < KH * CO; j += 256) {
                const int co = j % CO, kh = j / CO;
                f |= zero_product_class(wu[(int64_t(kh * KW + kw) * CI + ci) * CO + co], z.hi, z.sat);
            }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) f |= uint32_t(__shfl_xor(int(f), o));
        if ((threadIdx.x & 63) == 0) s_or[threadIdx.x >> 6] = f;
        __syncthreads();
        if (threadIdx.x == 0) {
            const uint32_t r = s_or[0] | s_or[1] | s_or[2] | s_or[3];
            if (t < nphase)
                phase_flags[t] = r;
            else
                kw_flags[t - nphase] = r;
        }
        __syncthreads();  // s_or is reused by the next flag
    }
}

// Adds the products outside each output's stride phase (see zero_tap_flags_body) to dx
// [n][H][W][CI]: NaN where one is NaN, +0 for an exactly -0 sum where one is +0.
// (total < 2^31: the convolution limits keep tensors below 2^29 elements)
__global__ __launch_bounds__(256) void dilation_fixup_kernel(float *__restrict__ dx, int total, int H, int Wd, int CI,
                                                             int sh, int sw, const uint32_t *__restrict__ phase_flags)
{
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        const int ci = i % CI, t = i / CI;
        const int x = t % Wd, y = (t / Wd) % H;
        const uint32_t f = phase_flags[((y % sh) * sw + x % sw) * CI + ci];
        if (f == 0u) continue;
        const uint32_t u = __float_as_uint(dx[i]);
        if (f & kZeroNan)
            dx[i] = __uint_as_float(0x7FC00000u);
        else if (u == 0x80000000u)
            dx[i] = 0.0f;
    }
}

// Backward-data pass with few input channels, second half: the gradient of the w-unfolded input
// (see the DecUnfold decode), dxu[n][ih][ow][kw * c + ci], folded back onto x's pixels:
// dx[n][ih][iw][ci] = the sum, in ascending kw, of dxu[n][ih][ow][kw * c + ci] over the (kw, ow)
// with ow * sw + kw - left = iw, 0 <= ow < ow_n; -0 (the empty sum) where there is none.  A kw with
// no such ow reads zeros of the dilated, padded error at every kh: its products are those of
// kw_flags (see zero_tap_flags_body).  phase_flags (stride sh > 1): the virtual pass's flags per
// row phase ih mod sh and unfolded channel, applied to each term as dilation_fixup_kernel would
// apply them to dxu.  (n * h * w * c and the unfolded gradient stay below 2^31 elements.)
__global__ __launch_bounds__(256) void fold_w_kernel(const float *__restrict__ dxu, int n, int h, int w, int c,
                                                     int kw_n, int sw, int left, int ow_n,
                                                     const uint32_t *__restrict__ kw_flags,
                                                     const uint32_t *__restrict__ phase_flags, int sh,
                                                     float *__restrict__ dx)
{
    const int total = n * h * w * c;
    const int cu = kw_n * c;
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        const int ci = i % c, t = i / c;
        const int iw = t % w, row = t / w;  // row = n * h + ih
        const uint32_t *pf = phase_flags ? phase_flags + (row % h % sh) * cu : nullptr;
        float acc = -0.0f;
        uint32_t zf = 0u;
        for (int k = 0; k < kw_n; ++k) {
            const int num = iw + left - k;
            const int ow = num >= 0 ? num / sw : -1;
            if (num < 0 || ow * sw != num || ow >= ow_n) {
                zf |= kw_flags[k * c + ci];
                continue;
            }
            float term = dxu[(row * ow_n + ow) * cu + k * c + ci];
            if (pf) {
                const uint32_t f = pf[k * c + ci];
                if (f & kZeroNan)
                    term = __uint_as_float(0x7FC00000u);
                else if ((f & kZeroPos) && __float_as_uint(term) == 0x80000000u)
                    term = 0.0f;
            }
            acc += term;
        }
        if (zf & kZeroNan)
            acc = __uint_as_float(0x7FC00000u);
        else if ((zf & kZeroPos) && __float_as_uint(acc) == 0x80000000u)
            acc = 0.0f;
        dx[i] = acc;
    }
}

// Tiled transpose-decode for the GEMM first operand: src is `rows x cols` with strides
// (sr, sc); dst[c * dld + r] = decode(src(r, c)), rows padded to dld with decoded +0.
// Pair records (records != null): records[(c / 2) * dld + r] = {index field of (r, c), head of
// (r, c) | head of (r, c + 1) << 16 as bf16, index field of (r, c + 1)}, a column past the end
// being a decoded +0.  The grid strides over 64 x 64 tiles in both directions.
// The workgroups form a gx x (nblk / gx) grid over the tiles, workgroup bid at (bid % gx, bid / gx).
struct DecT {
    const float *src;
    int64_t sr, sc;
    int rows, cols;
    uint32_t *dst;
    int dld;
    uint32_t *records;
    int gx;
};

__device__ __forceinline__ void decode_a_body(const DecT &d, DecFmt f, uint32_t *__restrict__ stats, int bid, int nblk)
{
    __shared__ uint32_t tile[64][65];
    const float *__restrict__ src = d.src;
    uint32_t *__restrict__ dst = d.dst;
    uint32_t *__restrict__ records = d.records;
    const int64_t sr = d.sr, sc = d.sc;
    const int rows = d.rows, cols = d.cols, dld = d.dld;
    const int gx = d.gx, gy = nblk / d.gx, bx = bid % gx, by = bid / gx;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    ExpStats st;
    for (int r0 = bx * 64; r0 < dld; r0 += gx * 64) {
        for (int c0 = by * 64; c0 < cols; c0 += gy * 64) {
            // two halves of 8 loads: the registers of the second-operand decode it shares a launch with
#pragma unroll 1
            for (int hf = 0; hf < 16; hf += 8) {
                uint32_t u[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const int r = r0 + ty + 4 * (hf + i), c = c0 + tx;
                    u[i] = (r < rows && c < cols) ? __float_as_uint(src[int64_t(r) * sr + int64_t(c) * sc]) : 0u;
                }
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    st.add(u[i]);
                    tile[ty + 4 * (hf + i)][tx] = amsim_decode_fmt(u[i], f);
                }
            }
            __syncthreads();
            if (records == nullptr) {
                for (int i = ty; i < 64; i += 4) {
                    const int c = c0 + i, r = r0 + tx;
                    if (c < cols && r < dld) dst[int64_t(c) * dld + r] = tile[tx][i];
                }
            } else {
                for (int i = ty; i < 32; i += 4) {  // c0 is even: pair (c, c + 1) lies in the tile
                    const int c = c0 + 2 * i, r = r0 + tx;
                    if (c < cols && r < dld) {
                        store_record(records + (int64_t(c >> 1) * dld + r) * 3, tile[tx][2 * i], tile[tx][2 * i + 1],
                                     f.raw);
                    }
                }
            }
            __syncthreads();
        }
    }
    store_stats(st, stats, bid);
}

// Direct evaluation, the comparison the paper draws for AMSim (Sec. "AMSim", its figure of GEMM
// run time for AMSim, direct simulation and the native multiply): the same GEMM with no table.
//   DIRECT_NATIVE    every product the native FP32 multiply, then an FP32 add.
//   DIRECT_MITCHELL  every product Mitchell's multiplier computed from the operands' bits.  With
//                    ka, kb the top-M mantissa fields, its mantissa product on the truncated
//                    fractions x = ka / 2^M, y = kb / 2^M is 1 + x + y below 2 and 2 (x + y) from
//                    2 on -- in FP32 bits 0x3F800000 + (ka + kb) << (23 - M) in both cases (a sum
//                    that reaches 2^M carries into the exponent field) -- then times pa * pb as
//                    on the table path, with the same zero, overflow, Inf and NaN rules.
// 64 x 64 outputs per workgroup of 256 threads, 4 x 4 per thread; 16-step tiles of both operands
// go through LDS step-major, so each thread reads its 4 rows and 4 columns with 16-byte loads.
enum { DIRECT_NATIVE = 0, DIRECT_MITCHELL = 1 };
constexpr int kDirTile = 64, kDirK = 16;

template <int MODE>
__global__ __launch_bounds__(256) void direct_gemm_kernel(const float *__restrict__ A, int64_t lda,
                                                          const float *__restrict__ B, int64_t ldb,
                                                          float *__restrict__ C, int64_t ldc, int m, int n, int k,
                                                          int mb)
{
    // [0]: raw operand (native) or head; [1]: Mitchell's shifted field (B's with the bias added)
    __shared__ __attribute__((aligned(16))) uint32_t sa[2][kDirK][kDirTile];
    __shared__ __attribute__((aligned(16))) uint32_t sb[2][kDirK][kDirTile];
    const int tx = int(threadIdx.x) % 16, ty = int(threadIdx.x) / 16;
    const int row0 = int(blockIdx.x) * kDirTile, col0 = int(blockIdx.y) * kDirTile;
    const int sh = 23 - mb;
    float acc[4][4];
    init_acc(acc);
    for (int k0 = 0; k0 < k; k0 += kDirK) {
        for (int i = threadIdx.x; i < kDirTile * kDirK; i += 256) {
            const int r = i / kDirK, kk = i % kDirK;  // A: consecutive threads along k
            const int gr = row0 + r, gk = k0 + kk;
            const uint32_t u = (gr < m && gk < k) ? __float_as_uint(A[int64_t(gr) * lda + gk]) : 0u;
            if constexpr (MODE == DIRECT_NATIVE) {
                sa[0][kk][r] = u;
            } else {
                const uint32_t w = amsim_decode(u, mb, 0);
                sa[0][kk][r] = w & kHeadMask;
                sa[1][kk][r] = (w & ((1u << mb) - 1u)) << sh;
            }
        }
        for (int i = threadIdx.x; i < kDirTile * kDirK; i += 256) {
            const int kk = i / kDirTile, c = i % kDirTile;  // B: consecutive threads along columns
            const int gc = col0 + c, gk = k0 + kk;
            const uint32_t u = (gc < n && gk < k) ? __float_as_uint(B[int64_t(gk) * ldb + gc]) : 0u;
            if constexpr (MODE == DIRECT_NATIVE) {
                sb[0][kk][c] = u;
            } else {
                const uint32_t w = amsim_decode(u, mb, 0);
                sb[0][kk][c] = w & kHeadMask;
                sb[1][kk][c] = ((w & ((1u << mb) - 1u)) << sh) + 0x3F800000u;
            }
        }
        __syncthreads();
        const int kn = min(kDirK, k - k0);
        for (int kk = 0; kk < kn; ++kk) {
            const u32x4 a0 = *reinterpret_cast<const u32x4 *>(&sa[0][kk][4 * ty]);
            const u32x4 b0 = *reinterpret_cast<const u32x4 *>(&sb[0][kk][4 * tx]);
            if constexpr (MODE == DIRECT_NATIVE) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const float p = __uint_as_float(a0[i]) * __uint_as_float(b0[j]);
                        acc[i][j] = acc[i][j] + p;
                    }
            } else {
                const u32x4 a1 = *reinterpret_cast<const u32x4 *>(&sa[1][kk][4 * ty]);
                const u32x4 b1 = *reinterpret_cast<const u32x4 *>(&sb[1][kk][4 * tx]);
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        // the product rounded on its own before the add: it may overflow to Inf
                        // (exponent 254 plus a carry), which an fma with the sum would not see
                        const float v = __uint_as_float(a1[i] + b1[j]);
                        const float c = v * (__uint_as_float(a0[i]) * __uint_as_float(b0[j]));
                        acc[i][j] = acc[i][j] + c;
                    }
            }
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = row0 + 4 * ty + i;
        if (r >= m) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int c = col0 + 4 * tx + j;
            if (c < n) C[int64_t(r) * ldc + c] = acc[i][j];
        }
    }
}

// C[r][c] = sum over z of part[z][r][c] in a fixed order (deterministic): the splits are cut into
// G consecutive groups, summed in z order within a group (eight loads in flight) and the group
// sums then added in group order.  G > 1 gives outputs with many splits more threads.  Workgroups
// of 256 threads: thread (g, o) for g < G, o < 256 / G.
__global__ __launch_bounds__(256) void reduce_splits_kernel(const float *__restrict__ part, int splits, int rows,
                                                            int cols, float *__restrict__ C, int64_t ldc, int G)
{
    __shared__ float s_part[256];
    const int64_t total = int64_t(rows) * cols;
    const int opb = 256 / G;  // outputs per workgroup and pass
    const int g = int(threadIdx.x) / opb, ol = int(threadIdx.x) % opb;
    const int per = (splits + G - 1) / G, z0 = min(splits, g * per), z1 = min(splits, z0 + per);
    for (int64_t base = int64_t(blockIdx.x) * opb; base < total; base += int64_t(gridDim.x) * opb) {
        const int64_t i = base + ol;
        float s = -0.0f;
        if (i < total) {
            int z = z0;
            for (; z + 8 <= z1; z += 8) {
                float v[8];
#pragma unroll
                for (int k = 0; k < 8; ++k) v[k] = part[int64_t(z + k) * total + i];
#pragma unroll
                for (int k = 0; k < 8; ++k) s += v[k];
            }
            for (; z < z1; ++z) s += part[int64_t(z) * total + i];
        }
        if (G > 1) {
            __syncthreads();  // the previous pass has read s_part
            s_part[threadIdx.x] = s;
            __syncthreads();
            if (g == 0) {
                for (int k = 1; k < G; ++k) s += s_part[k * opb + ol];
            }
        }
        if (g == 0 && i < total) {
            const int64_t r = i / cols, c = i % cols;
            C[r * ldc + c] = s;
        }
    }
}

__global__ void fill_kernel(float *__restrict__ C, int rows, int cols, int64_t ldc, float v)
{
    const int64_t total = int64_t(rows) * cols;
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < total;
         i += int64_t(gridDim.x) * blockDim.x)
        C[(i / cols) * ldc + (i % cols)] = v;
}

// Element-wise products through the same decode/combine path as the GEMM kernels, with the
// table read from global memory in its canonical layout (index = ka * 2^M + kb).  fa, fb: the
// operands' decode (fa's index field ka << M, fb's kb); vadd, su, sd: the exact path's format
// scaling (see tab_body).
__global__ void mul_ew_kernel(int64_t n, const float *__restrict__ a, const float *__restrict__ b,
                              float *__restrict__ c, const uint32_t *__restrict__ lut, DecFmt fa, DecFmt fb,
                              uint32_t vadd, float su, float sd)
{
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x) {
        const uint32_t wa = amsim_decode_fmt(__float_as_uint(a[i]), fa);
        const uint32_t wb = amsim_decode_fmt(__float_as_uint(b[i]), fb);
        const float v = __uint_as_float(((lut[(wa & kIdxMask) + (wb & kIdxMask)] & 0x00FFFFFFu) + 0x3F800000u) + vadd);
        c[i] = ((v * (head_value(wa) * head_value(wb))) * su) * sd;
    }
}

// ------------------------------------------------------------------ vector GEMMs --------
// One product a * b of the table's multiplier from the operands' bits (fa's index field ka << M,
// fb's kb; the table in its canonical layout in global memory); NARROW: a format with fewer
// exponent bits, scaled as the exact path scales it.
template <bool NARROW>
__device__ __forceinline__ float vec_product(uint32_t ua, uint32_t ub, const uint32_t *__restrict__ lut,
                                             const DecFmt &fa, const DecFmt &fb, uint32_t vadd, float su, float sd)
{
    const uint32_t wa = amsim_decode_fmt(ua, fa), wb = amsim_decode_fmt(ub, fb);
    const float v = __uint_as_float(((lut[(wa & kIdxMask) + (wb & kIdxMask)] & 0x00FFFFFFu) + 0x3F800000u) + vadd);
    const float c = v * (head_value(wa) * head_value(wb));
    return NARROW ? (c * su) * sd : c;
}

// GEMM with a vector operand (m == 1: op(A) is a row, the outputs are C's columns; n == 1:
// op(B) is a column, the outputs are C's rows) -- a dense layer at batch 1.  The matrix element of
// output o and step kk is mat[o * so + kk * sk], the vector's vec[kk * vs].  Every operand is
// decoded where it is read, so the call is one of the two kernels below (and, when k is split,
// the fixed-order reduction) only; split y of the grid covers steps [y * kchunk, (y + 1) * kchunk)
// and writes its sums to part[y][o] when the grid splits k, else to out[o * os].  VEC_FIRST: the
// vector is the first operand (the table's high index).  A product past the end of a run is
// skipped, not added as a zero (a +0 product would turn a sum of -0 products into +0).
//
// MODE: GV_TAB_LDS (FP32 operands, M <= 7: each workgroup first stages the whole table into LDS
// as the factors v = 2^carry * 1.mantissa, so a product is one LDS gather and two multiplies),
// GV_TAB (FP32 operands, the table read from global memory), GV_NARROW (a (1, e, m) format, the
// generic decode) or GV_NATIVE (the native FP32 multiply, one fma per product).
enum { GV_NATIVE = 0, GV_TAB = 1, GV_TAB_LDS = 2, GV_NARROW = 3 };

// An FP32 operand's head without branches: sign | exponent, with the quiet bit set for NaN (zeros
// and denormals give +-0, Inf +-Inf: Algorithm 2's operand classes, as amsim_decode reads them).
__device__ __forceinline__ float fp32_head(uint32_t u)
{
    return __uint_as_float((u & 0xFF800000u) | ((u & 0x7FFFFFFFu) > 0x7F800000u ? 0x00400000u : 0u));
}

struct GvCtx {
    const uint32_t *lut;  // the table, canonical layout
    const float *tab;     // GV_TAB_LDS: the staged factors
    int m, shift;         // M, 23 - M
    DecFmt fa, fb;        // GV_NARROW
    uint32_t vadd;
    float su, sd;
};

// One operand as the products use it: its bits, head and index field (ka << M for the first
// operand, kb for the second).
struct GvOp {
    uint32_t u;
    float p;
    uint32_t i;
};

template <int MODE>
__device__ __forceinline__ GvOp gv_operand(uint32_t u, bool first, const GvCtx &cx)
{
    GvOp o{u, 0.0f, 0u};
    if constexpr (MODE == GV_TAB || MODE == GV_TAB_LDS) {
        o.p = fp32_head(u);
        o.i = ((u >> cx.shift) & ((1u << cx.m) - 1u)) << (first ? cx.m : 0);
    }
    return o;
}

template <int MODE>
__device__ __forceinline__ float gv_mac(float acc, const GvOp &a, const GvOp &b, const GvCtx &cx)
{
    if constexpr (MODE == GV_NATIVE) {
        return __builtin_fmaf(__uint_as_float(a.u), __uint_as_float(b.u), acc);
    } else if constexpr (MODE == GV_NARROW) {
        return acc + vec_product<true>(a.u, b.u, cx.lut, cx.fa, cx.fb, cx.vadd, cx.su, cx.sd);
    } else {
        const uint32_t idx = a.i | b.i;
        const float v = MODE == GV_TAB_LDS ? cx.tab[idx]
                                           : __uint_as_float((cx.lut[idx] & 0x00FFFFFFu) + 0x3F800000u);
        return acc + v * (a.p * b.p);
    }
}

template <bool VEC_FIRST, int MODE>
__device__ __forceinline__ float gv_step(float acc, const GvOp &vop, uint32_t um, const GvCtx &cx)
{
    const GvOp mop = gv_operand<MODE>(um, !VEC_FIRST, cx);
    return VEC_FIRST ? gv_mac<MODE>(acc, vop, mop, cx) : gv_mac<MODE>(acc, mop, vop, cx);
}

// GV_TAB_LDS without NaN operands: a product's factor v sits at LDS byte offset
// (ka << (M + 2)) | (kb << 2), taken from each operand's bits with one shift and one mask, and its
// head is the operand's sign and exponent bits alone (zeros and denormals +-0, Inf +-Inf); a
// batch with a NaN operand takes the generic form instead (gv_step).
struct GvFast {
    int sh_m;        // matrix element: shift and mask of its index bits, already at their byte offset
    uint32_t mk_m;
    int sh_v;        // vector element: likewise
    uint32_t mk_v;
};

template <bool VEC_FIRST>
__device__ __forceinline__ GvFast gv_fast(const GvCtx &cx)
{
    const uint32_t mask = (1u << cx.m) - 1u;
    const int hi = 21 - 2 * cx.m, lo = 21 - cx.m;  // shifts that leave ka at bit M + 2, kb at bit 2
    return VEC_FIRST ? GvFast{lo, mask << 2, hi, mask << (cx.m + 2)} : GvFast{hi, mask << (cx.m + 2), lo, mask << 2};
}

__device__ __forceinline__ bool is_nan_bits(uint32_t u) { return (u & 0x7FFFFFFFu) > 0x7F800000u; }

// The products of a batch of NV steps and NC outputs, added to acc[c] in step order: step i's
// vector element uv[i] with the matrix element mat_at(i, c).  GV_TAB_LDS batches without a NaN
// operand (checked over the wave) gather all their factors first, then multiply.
template <bool VEC_FIRST, int MODE, int NV, int NC, class MatAt>
__device__ __forceinline__ void gv_batch(float (&acc)[NC], const uint32_t (&uv)[NV], MatAt mat_at, const GvCtx &cx)
{
    if constexpr (MODE == GV_TAB_LDS) {
        bool nan = false;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            nan |= is_nan_bits(uv[i]);
#pragma unroll
            for (int c = 0; c < NC; ++c) nan |= is_nan_bits(mat_at(i, c));
        }
        if (__builtin_amdgcn_ballot_w64(nan) == 0) {
            const GvFast f = gv_fast<VEC_FIRST>(cx);
            const unsigned char *tb = reinterpret_cast<const unsigned char *>(cx.tab);
            float v[NV][NC];
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const uint32_t voff = (uv[i] >> f.sh_v) & f.mk_v;
#pragma unroll
                for (int c = 0; c < NC; ++c)
                    v[i][c] = *reinterpret_cast<const float *>(tb + (((mat_at(i, c) >> f.sh_m) & f.mk_m) | voff));
            }
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const float pv = __uint_as_float(uv[i] & 0xFF800000u);
#pragma unroll
                for (int c = 0; c < NC; ++c) acc[c] += v[i][c] * (pv * __uint_as_float(mat_at(i, c) & 0xFF800000u));
            }
            return;
        }
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const GvOp vop = gv_operand<MODE>(uv[i], VEC_FIRST, cx);
#pragma unroll
        for (int c = 0; c < NC; ++c) acc[c] = gv_step<VEC_FIRST, MODE>(acc[c], vop, mat_at(i, c), cx);
    }
}

// The table's factors into LDS (GV_TAB_LDS): 2^(2M) floats at the start of the dynamic LDS.
template <int MODE>
__device__ __forceinline__ const float *gv_stage(const GvCtx &cx, float *lds)
{
    if constexpr (MODE == GV_TAB_LDS) {
        const int entries = 1 << (2 * cx.m);
        for (int i = threadIdx.x; i < entries; i += blockDim.x)
            lds[i] = __uint_as_float((cx.lut[i] & 0x00FFFFFFu) + 0x3F800000u);
        __syncthreads();
    }
    return lds;
}

constexpr int kGemvUnroll = 8;  // steps whose loads a lane has in flight (column kernel)

// Outputs contiguous in the matrix (so == 1): each lane owns kGemvCols consecutive outputs and
// reads them with one 16-byte load per step (v4: mat 16-byte aligned and sk a multiple of 4;
// otherwise, and for a last partial group, one load per element).  The vector's element of a
// step is the same for the whole wave.  The waves of a workgroup (gv_waves) sum consecutive
// parts of the split's steps for the same outputs, in step order, and their sums are added in
// wave order.
constexpr int gv_waves(int mode) { return mode == GV_TAB_LDS ? kGemvWavesLds : kGemvWavesGlobal; }

template <bool VEC_FIRST, int MODE>
__global__ __launch_bounds__(64 * gv_waves(MODE)) void gemv_cols_kernel(int64_t nout, int64_t k,
                                                                    const float *__restrict__ vec, int64_t vs,
                                                                    const float *__restrict__ mat, int64_t sk, int v4,
                                                                    float *__restrict__ out, int64_t os,
                                                                    float *__restrict__ part, int64_t kchunk, GvCtx cx)
{
    constexpr int WAVES = gv_waves(MODE);
    extern __shared__ float gv_lds[];  // [table factors (GV_TAB_LDS)][WAVES][kGemvCols][64] sums
    cx.tab = gv_stage<MODE>(cx, gv_lds);
    float(*sums)[kGemvCols][64] =
        reinterpret_cast<float(*)[kGemvCols][64]>(gv_lds + (MODE == GV_TAB_LDS ? (1 << (2 * cx.m)) : 0));
    const int lane = threadIdx.x & 63, wave = wave_id();
    const int64_t o0 = (int64_t(blockIdx.x) * 64 + lane) * kGemvCols;
    const int64_t k0 = int64_t(blockIdx.y) * kchunk, k1 = min(k, k0 + kchunk);
    const int64_t q = (k1 - k0 + WAVES - 1) / WAVES;
    const int64_t s0 = min(k1, k0 + wave * q), s1 = min(k1, s0 + q);
    float acc[kGemvCols];
#pragma unroll
    for (int c = 0; c < kGemvCols; ++c) acc[c] = -0.0f;
    // every lane of the block owns kGemvCols outputs that 16-byte loads can read (uniform)
    const bool block_full = v4 && (int64_t(blockIdx.x) + 1) * 64 * kGemvCols <= nout;
    if (block_full) {
        auto load = [&](int64_t k_at, uint32_t (&uv)[kGemvUnroll], u32x4 (&um)[kGemvUnroll]) {
#pragma unroll
            for (int i = 0; i < kGemvUnroll; ++i) {
                uv[i] = __float_as_uint(vec[(k_at + i) * vs]);
                um[i] = *reinterpret_cast<const u32x4 *>(mat + (k_at + i) * sk + o0);
            }
        };
        // software pipeline over two register buffers: the next batch's loads are in flight while
        // this batch's products run
        uint32_t uv0[kGemvUnroll], uv1[kGemvUnroll];
        u32x4 um0[kGemvUnroll], um1[kGemvUnroll];
        auto run = [&](const uint32_t(&uv)[kGemvUnroll], const u32x4(&um)[kGemvUnroll]) {
            gv_batch<VEC_FIRST, MODE, kGemvUnroll, kGemvCols>(acc, uv, [&](int i, int c) { return um[i][c]; }, cx);
        };
        int64_t kk = s0;
        if (kk + kGemvUnroll <= s1) load(kk, uv0, um0);
        while (kk + kGemvUnroll <= s1) {
            const bool more = kk + 2 * kGemvUnroll <= s1;
            if (more) load(kk + kGemvUnroll, uv1, um1);
            run(uv0, um0);
            kk += kGemvUnroll;
            if (!more) break;
            if (kk + 2 * kGemvUnroll <= s1) load(kk + kGemvUnroll, uv0, um0);
            run(uv1, um1);
            kk += kGemvUnroll;
            if (!(kk + kGemvUnroll <= s1)) break;
        }
        for (; kk < s1; ++kk) {
            const GvOp vop = gv_operand<MODE>(__float_as_uint(vec[kk * vs]), VEC_FIRST, cx);
            const u32x4 um1 = *reinterpret_cast<const u32x4 *>(mat + kk * sk + o0);
#pragma unroll
            for (int c = 0; c < kGemvCols; ++c) acc[c] = gv_step<VEC_FIRST, MODE>(acc[c], vop, um1[c], cx);
        }
    } else if (o0 < nout) {  // the last block, or a matrix 16-byte loads cannot read: one load per element
        const int nc = int(min<int64_t>(kGemvCols, nout - o0));
        for (int64_t kk = s0; kk < s1; ++kk) {
            const GvOp vop = gv_operand<MODE>(__float_as_uint(vec[kk * vs]), VEC_FIRST, cx);
            const float *src = mat + kk * sk + o0;
#pragma unroll
            for (int c = 0; c < kGemvCols; ++c)
                if (c < nc) acc[c] = gv_step<VEC_FIRST, MODE>(acc[c], vop, __float_as_uint(src[c]), cx);
        }
    }
#pragma unroll
    for (int c = 0; c < kGemvCols; ++c) sums[wave][c][lane] = acc[c];
    __syncthreads();
    if (wave != 0 || o0 >= nout) return;
#pragma unroll
    for (int c = 0; c < kGemvCols; ++c) {
        const int64_t o = o0 + c;
        if (o >= nout) break;
        float r = sums[0][c][lane];
#pragma unroll
        for (int w = 1; w < WAVES; ++w) r += sums[w][c][lane];
        if (part != nullptr)
            part[int64_t(blockIdx.y) * nout + o] = r;
        else
            out[o * os] = r;
    }
}

// Steps contiguous in the matrix (sk == 1): each wave owns kGemvRows outputs; its lanes take four
// consecutive steps each (one 16-byte load per output when v4: mat 16-byte aligned and so a
// multiple of 4), 256 steps per pass, and every lane sums its steps in order; a fixed butterfly
// over the 64 lanes then adds the lanes' sums, and lane 0 stores them.  kchunk is a multiple of
// 256, so the lanes' steps stay 4-aligned.
template <bool VEC_FIRST, int MODE>
__global__ __launch_bounds__(64 * gv_waves(MODE)) void gemv_rows_kernel(int64_t nout, int64_t k,
                                                                    const float *__restrict__ vec, int64_t vs,
                                                                    const float *__restrict__ mat, int64_t so, int v4,
                                                                    float *__restrict__ out, int64_t os,
                                                                    float *__restrict__ part, int64_t kchunk, GvCtx cx)
{
    constexpr int WAVES = gv_waves(MODE);
    extern __shared__ float gv_lds[];  // table factors (GV_TAB_LDS)
    cx.tab = gv_stage<MODE>(cx, gv_lds);
    const int lane = threadIdx.x & 63, wave = wave_id();
    const int64_t ob = (int64_t(blockIdx.x) * WAVES + wave) * kGemvRows;  // the wave's first output
    if (ob >= nout) return;  // uniform over the wave (after the workgroup's staging)
    const int64_t k0 = int64_t(blockIdx.y) * kchunk, k1 = min(k, k0 + kchunk);
    const int nr = int(min<int64_t>(kGemvRows, nout - ob));
    float acc[kGemvRows];
#pragma unroll
    for (int r = 0; r < kGemvRows; ++r) acc[r] = -0.0f;
    // whole passes of 256 steps over kGemvRows outputs that 16-byte loads can read (uniform)
    const bool fast = v4 && nr == kGemvRows;
    const int64_t k_fast = fast ? k0 + (k1 - k0) / 256 * 256 : k0;
    if (fast) {
        auto load = [&](int64_t kb, uint32_t (&uv)[4], u32x4 (&um)[kGemvRows]) {
            const int64_t kk = kb + 4 * lane;
#pragma unroll
            for (int i = 0; i < 4; ++i) uv[i] = __float_as_uint(vec[(kk + i) * vs]);
#pragma unroll
            for (int r = 0; r < kGemvRows; ++r) um[r] = *reinterpret_cast<const u32x4 *>(mat + (ob + r) * so + kk);
        };
        // software pipeline over two register buffers: the next pass's loads are in flight while
        // this pass's products run
        uint32_t uv0[4], uv1[4];
        u32x4 um0[kGemvRows], um1[kGemvRows];
        auto run = [&](const uint32_t(&uv)[4], const u32x4(&um)[kGemvRows]) {
            gv_batch<VEC_FIRST, MODE, 4, kGemvRows>(acc, uv, [&](int i, int r) { return um[r][i]; }, cx);
        };
        int64_t kb = k0;
        if (kb < k_fast) load(kb, uv0, um0);
        while (kb < k_fast) {
            const bool more = kb + 256 < k_fast;
            if (more) load(kb + 256, uv1, um1);
            run(uv0, um0);
            kb += 256;
            if (!more) break;
            if (kb + 256 < k_fast) load(kb + 256, uv0, um0);
            run(uv1, um1);
            kb += 256;
        }
    }
    // the rest (a last partial pass, fewer rows, or a matrix 16-byte loads cannot read): one load
    // per element
    for (int64_t kb = k_fast; kb < k1; kb += 256) {
        const int64_t kk = kb + 4 * lane;
        const int ns = int(max<int64_t>(0, min<int64_t>(4, k1 - kk)));
        for (int i = 0; i < ns; ++i) {
            const GvOp vop = gv_operand<MODE>(__float_as_uint(vec[(kk + i) * vs]), VEC_FIRST, cx);
#pragma unroll
            for (int r = 0; r < kGemvRows; ++r)
                if (r < nr)
                    acc[r] = gv_step<VEC_FIRST, MODE>(acc[r], vop, __float_as_uint(mat[(ob + r) * so + kk + i]), cx);
        }
    }
#pragma unroll
    for (int r = 0; r < kGemvRows; ++r)
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) acc[r] += __shfl_xor(acc[r], off);
    if (lane != 0) return;
    for (int r = 0; r < nr; ++r) {
        const int64_t o = ob + r;
        if (part != nullptr)
            part[int64_t(blockIdx.y) * nout + o] = acc[r];
        else
            out[o * os] = acc[r];
    }
}

// GEMM with k == 1 (an outer product -- the weight gradient of a dense layer at batch 1): every
// output is one product, C[i][j] = a_i * b_j (a sum of one product from -0.0 is that product).
template <bool NATIVE, bool NARROW>
__global__ __launch_bounds__(256) void outer_kernel(int64_t m, int64_t n, const float *__restrict__ a, int64_t as,
                                                   const float *__restrict__ b, int64_t bs, float *__restrict__ C,
                                                   int64_t ldc, const uint32_t *__restrict__ lut, DecFmt fa, DecFmt fb,
                                                   uint32_t vadd, float su, float sd)
{
    for (int64_t t = int64_t(blockIdx.x) * 256 + threadIdx.x; t < m * n; t += int64_t(gridDim.x) * 256) {
        const int64_t i = t / n, j = t - i * n;
        const uint32_t ua = __float_as_uint(a[i * as]), ub = __float_as_uint(b[j * bs]);
        C[i * ldc + j] = NATIVE ? __builtin_fmaf(__uint_as_float(ua), __uint_as_float(ub), -0.0f)
                                : vec_product<NARROW>(ua, ub, lut, fa, fb, vadd, su, sd);
    }
}

// The exponent cast on its own: y[i] = x[i] cast to the (1, e, m) format's range (see DecFmt),
// as an FP32 value -- in range unchanged, below it a signed zero, above it a signed Inf or the
// largest finite value (2 - 2^-m) * 2^beta; NaN and Inf as they are, denormals a signed zero.
__global__ void cast_kernel(int64_t n, const float *__restrict__ x, float *__restrict__ y, DecFmt f)
{
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x) {
        const uint32_t u = __float_as_uint(x[i]);
        const uint32_t e = (u >> 23) & 0xFFu, sign = u & 0x80000000u;
        uint32_t r = u;
        if (e == 0u || (e != 0xFFu && int(e) < f.lo))
            r = sign;
        else if (e != 0xFFu && int(e) > f.hi)
            r = f.sat ? (sign | (uint32_t(f.hi) << 23) | (((1u << f.m) - 1u) << (23 - f.m))) : (sign | 0x7F800000u);
        y[i] = __uint_as_float(r);
    }
}

// ------------------------------------------------------------------ table preparation

// The table's transposed, width-reduced rows (M <= 7), one job of the pre-pass.  The entry width
// eb is the fewest bytes that hold every entry's mantissa field: 1 when the low 16 bits of every
// entry are zero, 2 when the low 8 are, else 4.  Row kb (kTabRowEntries * eb bytes) holds entry
// (ka, kb) at byte ka * eb; with 1-byte entries dot_rows holds the same bytes in the order the
// bf16 path stages them (byte 4 * (ka % 32) + ka / 32 of row kb), with 2-byte entries hl_rows the
// entries split into bf16 halves for the hi/lo path.  Every workgroup ORs the whole table for eb
// (a few tens of KiB, read from L2 after the first) and writes the rows kb of its share;
// workgroup 0 also writes flags[0] = eb and the zero rows.
struct TablePrep {
    const uint32_t *lut;
    int m;
    int vec;               // lut 16-byte aligned
    unsigned char *rows, *dot_rows;
    uint32_t *hl_rows;
    int *flags;
    uint32_t *part;        // wide tables: one low-bits word per workgroup of the job
};

// Workgroups of the table job for M <= 7: rows of 8 entries kb each.
inline int table_jobs(int m) { return std::max(1, std::min(16, (1 << m) / 8)); }

__device__ __forceinline__ uint32_t block_or(uint32_t v, uint32_t *s4)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v |= uint32_t(__shfl_xor(int(v), o));
    if ((threadIdx.x & 63) == 0) s4[threadIdx.x >> 6] = v;
    __syncthreads();
    return s4[0] | s4[1] | s4[2] | s4[3];
}

__device__ __forceinline__ void prep_table_body(const TablePrep &t, int bid, int nblk)
{
    __shared__ uint32_t s_low[4];
    const uint32_t *__restrict__ lut = t.lut;
    const int n = 1 << t.m, total = n * n;
    uint32_t low = 0u;
    if (t.vec) {
#pragma unroll 4
        for (int i = threadIdx.x; i < total / 4; i += 256) {
            const u32x4 q = reinterpret_cast<const u32x4 *>(lut)[i];
            low |= q[0] | q[1] | q[2] | q[3];
        }
        for (int i = (total / 4) * 4 + threadIdx.x; i < total; i += 256) low |= lut[i];
    } else {
#pragma unroll 4
        for (int i = threadIdx.x; i < total; i += 256) low |= lut[i];
    }
    const uint32_t lb = block_or(low & 0xFFFFu, s_low);
    const int eb = lb == 0u ? 1 : ((lb & 0xFFu) == 0u ? 2 : 4);
    const bool lead = bid == 0;
    if (lead && threadIdx.x == 0) t.flags[0] = eb;
    const int per = (n + nblk - 1) / nblk, kb0 = bid * per, nk = max(0, min(n, kb0 + per) - kb0);
    unsigned char *__restrict__ dst = t.rows;
    // rows: thread -> (kb, group of 4 entries), consecutive threads along kb
    for (int i = threadIdx.x; i < nk * ((n + 3) / 4); i += 256) {
        const int kb = kb0 + i % nk, k4 = (i / nk) * 4;
        if (eb == 1) {
            uint32_t word = 0u;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (k4 + j < n) word |= ((lut[(k4 + j) * n + kb] >> 16) & 0xFFu) << (8 * j);
            if (k4 + 4 <= n)
                *reinterpret_cast<uint32_t *>(dst + size_t(kb) * kTabRowEntries + k4) = word;
            else
                for (int j = 0; k4 + j < n; ++j) dst[size_t(kb) * kTabRowEntries + k4 + j] = (word >> (8 * j)) & 0xFFu;
        } else {
            for (int j = 0; j < 4 && k4 + j < n; ++j) {
                const uint32_t e = lut[(k4 + j) * n + kb] & 0x00FFFFFFu;
                unsigned char *row = dst + size_t(kb) * kTabRowEntries * eb;
                if (eb == 2)
                    reinterpret_cast<uint16_t *>(row)[k4 + j] = static_cast<uint16_t>(e >> 8);
                else
                    reinterpret_cast<uint32_t *>(row)[k4 + j] = e + 0x3F800000u;
            }
        }
    }
    // the zero row
    if (lead) {
        for (int i = threadIdx.x; i < kTabRowEntries * eb / 4; i += 256)
            reinterpret_cast<uint32_t *>(dst + size_t(kZeroRow) * kTabRowEntries * eb)[i] = 0u;
        if (eb == 1 && threadIdx.x < kTabRowEntries / 4)
            reinterpret_cast<uint32_t *>(t.dot_rows + size_t(kZeroRow) * kTabRowEntries)[threadIdx.x] = 0u;
    }
    // hi/lo rows (2-byte entries): words 2 g + i of row kb hold entry ka = g + 64 i as
    // (v_hi - 0x3F80) | (v_lo - 0x3F80) << 16 in bf16 bits; v_lo is never zero (see tab_body_hl).
    // Workgroup 0 also writes the zero row's (kb = n).
    if (eb == 2) {
        const int nr = nk + (lead ? 1 : 0);
        for (int i = threadIdx.x; i < nr * 64; i += 256) {
            const int r = i / 64, g = i % 64;
            const int kb = r < nk ? kb0 + r : n;
            uint32_t word[2] = {0u, 0u};
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int ka = g + 64 * j;
                if (kb < n && ka < n) {
                    const float v = __uint_as_float((lut[ka * n + kb] & 0x00FFFFFFu) + 0x3F800000u);
                    float hi = __uint_as_float(__float_as_uint(v) & 0xFFFF0000u);
                    float lo = v - hi;  // exact: the low 8 of v's 16 significant bits
                    if (lo == 0.0f) {   // one bf16 unit of v moves to the low half
                        lo = __uint_as_float((__float_as_uint(v) & 0x7F800000u) - (7u << 23));
                        hi = v - lo;
                    }
                    word[j] = ((__float_as_uint(hi) >> 16) - 0x3F80u) & 0xFFFFu;
                    word[j] |= (((__float_as_uint(lo) >> 16) - 0x3F80u) & 0xFFFFu) << 16;
                }
            }
            const int row = kb < n ? kb : kZeroRow;
            t.hl_rows[(row * 64 + g) * 2 + 0] = word[0];
            t.hl_rows[(row * 64 + g) * 2 + 1] = word[1];
        }
    }
    // bf16-path rows: word g of row kb holds the bytes of entries g, g + 32, g + 64, g + 96.
    if (eb == 1) {
        for (int i = threadIdx.x; i < nk * 32; i += 256) {
            const int kb = kb0 + i % nk, g = i / nk;
            uint32_t word = 0u;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int ka = g + 32 * j;
                if (ka < n) word |= ((lut[ka * n + kb] >> 16) & 0xFFu) << (8 * j);
            }
            *reinterpret_cast<uint32_t *>(t.dot_rows + size_t(kb) * kTabRowEntries + 4 * g) = word;
        }
    }
}

// Wide tables (M = 8..11, rows of 2^M entries, no bf16 path).  The pre-pass job, one word per
// workgroup: the OR of the entries' low 16 mantissa bits, and bit 31 set when an entry (ka, kb)
// differs from the entry of the same index sum s = ka + kb in row min(s, 2^M - 1) -- i.e. when the
// table is not sum-indexed (T[ka][kb] = g(ka + kb)).
__device__ __forceinline__ void lut_low_bits_body(const TablePrep &t, int bid, int nblk)
{
    __shared__ uint32_t s_low[4];
    const int n = 1 << t.m, total = n * n;
    uint32_t low = 0u;
    for (int i = bid * 256 + int(threadIdx.x); i < total; i += nblk * 256) {
        const uint32_t e = t.lut[i];
        const int s = (i >> t.m) + (i & (n - 1)), ka = min(s, n - 1);
        low |= e & 0xFFFFu;
        if (((e ^ t.lut[(ka << t.m) + (s - ka)]) & 0x00FFFFFFu) != 0u) low |= 0x80000000u;
    }
    const uint32_t r = block_or(low, s_low);
    if (threadIdx.x == 0) t.part[bid] = r;
}

// Second launch for wide tables: the entry width from the nparts partial words, then the
// transposed rows -- row kb (2^m entries of eb bytes) holds entry (ka, kb) at byte ka * eb --
// through 64 x 64 LDS tiles (loads along kb, stores along ka).  Workgroup 0 writes flags[0] = eb,
// flags[1] = 0 (no bf16 path for wide rows), flags[2], the exact path's product form, from
// the decode statistics (n_a and n_b words; null for the native multiply), and flags[3] = 1 when
// the table is sum-indexed.
__global__ __launch_bounds__(256) void prep_rows_wide_kernel(const uint32_t *__restrict__ lut, int m,
                                                             const uint32_t *__restrict__ part, int nparts,
                                                             const uint32_t *__restrict__ stats_a, int n_a,
                                                             const uint32_t *__restrict__ stats_b, int n_b,
                                                             int narrow, unsigned char *__restrict__ dst,
                                                             int *__restrict__ flags)
{
    __shared__ uint32_t tile[64][65];
    __shared__ uint32_t s_low[4], s_ahs[4], s_bhs[4];
    uint32_t low = 0u;
    for (int i = threadIdx.x; i < nparts; i += 256) low |= part[i];
    const uint32_t lb = block_or(low, s_low);
    const int eb = (lb & 0xFFFFu) == 0u ? 1 : ((lb & 0xFFu) == 0u ? 2 : 4);
    if (blockIdx.x == 0) {  // uniform
        uint32_t alo = 255u, ahs = 0u, blo = 255u, bhs = 0u;
        const bool have = stats_a != nullptr;
        if (have) {
            stats_fold<256>(stats_a, n_a, alo, ahs);
            stats_fold<256>(stats_b, n_b, blo, bhs);
        }
        ahs = wave_max(ahs);
        bhs = wave_max(bhs);
        if ((threadIdx.x & 63) == 0) {
            s_ahs[threadIdx.x >> 6] = ahs;
            s_bhs[threadIdx.x >> 6] = bhs;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            const uint32_t a_hs = max(max(s_ahs[0], s_ahs[1]), max(s_ahs[2], s_ahs[3]));
            const uint32_t b_hs = max(max(s_bhs[0], s_bhs[1]), max(s_bhs[2], s_bhs[3]));
            int path, rounded;
            decide_paths(eb, 0u, a_hs, 0u, b_hs, have, narrow, path, rounded);
            flags[0] = eb;
            flags[1] = 0;
            flags[2] = rounded;
            flags[3] = (lb >> 31) == 0u ? 1 : 0;
        }
    }
    const int n = 1 << m, tiles_1d = n / 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int t = blockIdx.x; t < tiles_1d * tiles_1d; t += gridDim.x) {
        const int ka0 = (t / tiles_1d) * 64, kb0 = (t % tiles_1d) * 64;
        for (int i = ty; i < 64; i += 4) tile[i][tx] = lut[size_t(ka0 + i) * n + kb0 + tx];  // [ka][kb]
        __syncthreads();
        for (int i = ty; i < 64; i += 4) {
            const uint32_t e = tile[tx][i] & 0x00FFFFFFu;  // entry (ka0 + tx, kb0 + i)
            unsigned char *row = dst + size_t(kb0 + i) * n * eb;
            if (eb == 1)
                row[ka0 + tx] = static_cast<unsigned char>(e >> 16);
            else if (eb == 2)
                reinterpret_cast<uint16_t *>(row)[ka0 + tx] = static_cast<uint16_t>(e >> 8);
            else
                reinterpret_cast<uint32_t *>(row)[ka0 + tx] = e + 0x3F800000u;
        }
        __syncthreads();
    }
}

// The path flags of a call on rows of 128 entries whose table kernel reads them (kTabApprox):
// flags[1] and flags[2] (decide_paths) from the decode statistics, once the pre-pass has written
// the entry width flags[0].  One workgroup.
__global__ __launch_bounds__(1024) void path_flags_kernel(const uint32_t *__restrict__ stats_a, int n_a,
                                                          const uint32_t *__restrict__ stats_b, int n_b, int narrow,
                                                          int *__restrict__ flags)
{
    __shared__ uint32_t red[16][4];
    uint32_t alo = 255u, ahs = 0u, blo = 255u, bhs = 0u;
    stats_fold<1024>(stats_a, n_a, alo, ahs);
    stats_fold<1024>(stats_b, n_b, blo, bhs);
    alo = wave_min(alo);
    ahs = wave_max(ahs);
    blo = wave_min(blo);
    bhs = wave_max(bhs);
    const int wave = int(threadIdx.x) >> 6;
    if ((threadIdx.x & 63) == 0) {
        red[wave][0] = alo;
        red[wave][1] = ahs;
        red[wave][2] = blo;
        red[wave][3] = bhs;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t a_lo = 255u, a_hs = 0u, b_lo = 255u, b_hs = 0u;
        for (int w = 0; w < 16; ++w) {
            a_lo = min(a_lo, red[w][0]);
            a_hs = max(a_hs, red[w][1]);
            b_lo = min(b_lo, red[w][2]);
            b_hs = max(b_hs, red[w][3]);
        }
        int path, rounded;
        decide_paths(flags[0], a_lo, a_hs, b_lo, b_hs, true, narrow, path, rounded);
        flags[1] = path;
        flags[2] = rounded;
    }
}

// ------------------------------------------------------------------ the pre-pass --------
// One launch before each table kernel prepares everything it reads.  Its workgroups are dealt
// out to four independent jobs, in this order: the table (prep_table_body, or the low-bits pass
// of a wide table), the backward-data pass's zero-tap flags, the first operand's decode (one of
// the decode_a_body layouts) and the second operand's (decode_rows_body).  The jobs write
// disjoint parts of the workspace.  The decode jobs' exponent statistics, which decide the table
// kernel's path, are reduced by that kernel's own workgroups in a small call (tab_paths: nothing
// runs between the two launches), else by path_flags_kernel or prep_rows_wide_kernel.
struct PrepJobs {
    int n_tab, n_flag, n_a, n_b;  // workgroups of each job
    int wide;                     // the table job is a wide table's low-bits pass
    TablePrep t;
    ZeroTapFlags z;
    DecFmt fa, fb;
    uint32_t *stats_a, *stats_b;  // decode statistics, or null (native multiply)
    DecRows b;
};

template <class A>
__global__ __launch_bounds__(256) void prepass_kernel(PrepJobs j, A a)
{
    int bid = int(blockIdx.x);
    if (bid < j.n_tab) {
        if (j.wide)
            lut_low_bits_body(j.t, bid, j.n_tab);
        else
            prep_table_body(j.t, bid, j.n_tab);
        return;
    }
    bid -= j.n_tab;
    if (bid < j.n_flag) {
        zero_tap_flags_body(j.z, bid, j.n_flag);
        return;
    }
    bid -= j.n_flag;
    if (bid < j.n_a) {
        decode_a_body(a, j.fa, j.stats_a, bid, j.n_a);
        return;
    }
    bid -= j.n_a;
    decode_rows_body(j.b, j.fb, j.stats_b, uint32_t(bid), uint32_t(j.n_b));
}

// ------------------------------------------------------------------ host dispatch -------

std::once_flag g_attr_once;
hipError_t g_attr_err = hipSuccess;

hipError_t gemv_attributes();

void set_attributes()
{
    for (hipError_t e : {tab_attributes<OP_GEMM>(), tab_attributes<OP_FWD>(), tab_attributes<OP_BWD_DATA>(),
                         tab_attributes<OP_BWD_WEIGHT>(), gemv_attributes()})
        if (e != hipSuccess && g_attr_err == hipSuccess) g_attr_err = e;
}

int ensure_attributes()
{
    std::call_once(g_attr_once, set_attributes);
    return g_attr_err == hipSuccess ? AMSIM_OK : AMSIM_ERR_HIP;
}

// Split reduction of `splits` partial results of rows x cols into C (leading dimension ldc).
void launch_reduce(const float *part, int splits, int rows, int cols, float *C, int64_t ldc, hipStream_t st)
{
    const int64_t outputs = int64_t(rows) * cols;
    int G = 1;
    while (G < 32 && outputs * G < 65536 && splits >= 16 * G) G *= 2;
    const int64_t blocks = std::min<int64_t>(ceil_div(outputs, 256 / G), 65536);
    hipLaunchKernelGGL(reduce_splits_kernel, dim3(unsigned(blocks)), dim3(256), 0, st, part, splits, rows, cols, C, ldc,
                       G);
}

int launch_status()
{
    return hipGetLastError() == hipSuccess ? AMSIM_OK : AMSIM_ERR_HIP;
}

inline int grid_for(int64_t total, int block = 256)
{
    return int(std::max<int64_t>(1, std::min<int64_t>(ceil_div(total, block), 8192)));
}

// Workgroups of a decode_rows_body job for `words` output words (8 per thread and iteration).
inline int decode_grid(int64_t words) { return grid_for(ceil_div(words, 8)); }

// decode_rows_body's 16-byte load path: unit column stride and 16-byte aligned rows.
inline int decode_vec(const float *src, int64_t sb, int64_t sr, int64_t sc)
{
    return sc == 1 && reinterpret_cast<uintptr_t>(src) % 16 == 0 && sr % 4 == 0 && sb % 4 == 0 ? 1 : 0;
}


// How the products of a call are formed (amsim_options): the table's approximate product or the
// native FP32 multiply, on operands cast to a (1, e, m) format (e = 8: FP32's own exponent).
struct Mode {
    int native = 0;
    int e_bits = 8;
    int sat = 0;
};

int mode_of(const amsim_options *o, Mode &md)
{
    md = Mode{};
    if (!o) return AMSIM_OK;
    if (o->multiply != AMSIM_MULTIPLY_TABLE && o->multiply != AMSIM_MULTIPLY_NATIVE) return AMSIM_ERR_INVALID_ARG;
    if (o->exp_cast != AMSIM_CAST_INF && o->exp_cast != AMSIM_CAST_SATURATE) return AMSIM_ERR_INVALID_ARG;
    if (o->e_bits < 2 || o->e_bits > 8) return AMSIM_ERR_UNSUPPORTED;
    md.native = o->multiply == AMSIM_MULTIPLY_NATIVE ? 1 : 0;
    md.e_bits = o->e_bits;
    md.sat = o->exp_cast == AMSIM_CAST_SATURATE ? 1 : 0;
    if (md.native && md.e_bits != 8) return AMSIM_ERR_UNSUPPORTED;  // the native multiply is FP32's
    return AMSIM_OK;
}

// The format's bias beta = 2^(e-1) - 1 and the decode's exponent offset delta = (127 - beta) / 2.
inline int fmt_beta(const Mode &md) { return (1 << (md.e_bits - 1)) - 1; }
inline int fmt_delta(const Mode &md) { return (127 - fmt_beta(md)) / 2; }
// The largest finite FP32 exponent field the format keeps (beyond it the cast gives Inf or saturates).
inline int fmt_hi(const Mode &md) { return md.native || md.e_bits == 8 ? 254 : 127 + fmt_beta(md); }

// Decoded-index fields: the first operand's mantissa times 16 (the bf16 path's entry size; the
// exact path extracts it), the second's times the row length (its row offset in entries); zeros
// of the second operand on the zero row where rows have 128 entries (any row serves on the exact
// path, the zero head making the product a signed zero).
inline int shift_first(int) { return 4; }
inline int shift_second(int m_bits) { return row_log(m_bits); }
inline uint32_t zidx_second(const Plan &p) { return p.rl == 7 ? kZeroRowWord : 0u; }

DecFmt dec_fmt(const Mode &md, int m_bits, int shift, uint32_t zidx)
{
    DecFmt f = fp32_fmt(m_bits, shift, zidx);
    if (md.native) {
        f.raw = 1;
        f.zidx = 0u;
    } else if (md.e_bits < 8) {
        const int beta = fmt_beta(md);
        f.lo = 128 - beta;
        f.hi = 127 + beta;
        f.delta = fmt_delta(md);
        f.sat = md.sat;
    }
    return f;
}
inline DecFmt fmt_first(const Mode &md, int m_bits) { return dec_fmt(md, m_bits, shift_first(m_bits), 0u); }
inline DecFmt fmt_second(const Mode &md, const Plan &p, int m_bits)
{
    return dec_fmt(md, m_bits, shift_second(m_bits), zidx_second(p));
}

// Decode statistics (the bf16 path's exponent window and the exact path's product form):
// kStatSlots words per operand.
inline uint32_t *stats_a(char *ws, const Plan &p) { return reinterpret_cast<uint32_t *>(ws + p.off_stats); }
inline uint32_t *stats_b(char *ws, const Plan &p) { return reinterpret_cast<uint32_t *>(ws + p.off_stats) + kStatSlots; }

// A call's pre-pass jobs without the decodes' geometry: the table job (none for the native
// multiply; M <= 7 writes the rows itself, a wide table's low-bits pass is followed by
// prep_rows_wide_kernel), the statistics and the operand formats.
PrepJobs prep_jobs(const Mode &md, const uint32_t *lut, int mb, char *ws, const Plan &p)
{
    PrepJobs j{};
    j.fa = fmt_first(md, mb);
    j.fb = fmt_second(md, p, mb);
    if (md.native) return j;
    j.stats_a = stats_a(ws, p);
    j.stats_b = stats_b(ws, p);
    j.t.lut = lut;
    j.t.m = mb;
    j.t.vec = reinterpret_cast<uintptr_t>(lut) % 16 == 0 ? 1 : 0;
    j.t.rows = reinterpret_cast<unsigned char *>(ws + p.off_rows);
    j.t.dot_rows = reinterpret_cast<unsigned char *>(ws + p.off_dot_rows);
    j.t.hl_rows = reinterpret_cast<uint32_t *>(ws + p.off_hl_rows);
    j.t.flags = reinterpret_cast<int *>(ws + p.off_eb);
    if (p.rl == 7) {
        j.n_tab = table_jobs(mb);
    } else {
        j.wide = 1;
        j.t.part = reinterpret_cast<uint32_t *>(ws + p.off_wpart);
        j.n_tab = int(std::min<int64_t>(ceil_div(int64_t(1) << (2 * mb), 256 * 16), kWidePartWords));
    }
    return j;
}

// The table kernel variant of a call of `macs` products: the native multiply's; for a small call
// (small_call) the variant that decides its path itself (one launch fewer, for calls whose
// launches take about as long as their work); else the one that reads the path flags.
inline int tab_variant(const Mode &md, const Plan &p, double macs)
{
    if (md.native) return kTabNative;
    return small_call(macs, p.rl) ? kTabApproxSelf : kTabApprox;
}

// Launches the pre-pass (first-operand decode a, lds its dynamic LDS bytes), then what the table
// kernel variant `var` still needs: for a wide table the second table launch (which also writes
// the path flags), for kTabApprox on rows of 128 entries the path flags.
template <class A>
int run_prepass(const PrepJobs &j, const A &a, size_t lds, int var, int narrow, hipStream_t st)
{
    const int blocks = j.n_tab + j.n_flag + j.n_a + j.n_b;
    hipLaunchKernelGGL((prepass_kernel<A>), dim3(unsigned(blocks)), dim3(256), lds, st, j, a);
    if (j.wide) {
        const int tiles = (1 << (j.t.m - 6)) * (1 << (j.t.m - 6));
        hipLaunchKernelGGL(prep_rows_wide_kernel, dim3(std::min(tiles, 2048)), dim3(256), 0, st, j.t.lut, j.t.m,
                           j.t.part, j.n_tab, j.stats_a, j.n_a, j.stats_b, j.n_b, narrow, j.t.rows, j.t.flags);
    } else if (var == kTabApprox) {
        hipLaunchKernelGGL(path_flags_kernel, dim3(1), dim3(1024), 0, st, j.stats_a, j.n_a, j.stats_b, j.n_b, narrow,
                           j.t.flags);
    }
    return launch_status();
}

// The pointers of a launch's arguments (the rest is the plan's geometry, g).
TabArgs tab_args(TabArgs g, const Plan &p, char *ws, const uint32_t *A, const uint32_t *Bd, float *out)
{
    TabArgs a = g;
    a.A = A;
    a.Bd = Bd;
    a.out = out;
    a.rows = reinterpret_cast<const unsigned char *>(ws + p.off_rows);
    a.dot_rows = reinterpret_cast<const unsigned char *>(ws + p.off_dot_rows);
    a.hl_rows = reinterpret_cast<const unsigned char *>(ws + p.off_hl_rows);
    a.eb = reinterpret_cast<const int *>(ws + p.off_eb);
    return a;
}

// Operands cast to fewer exponent bits than FP32's (no bf16 path; products scaled before the add).
inline int narrow_of(const Mode &md) { return !md.native && md.e_bits < 8 ? 1 : 0; }

// The table kernel's view of the decode statistics (kTabApproxSelf decides its path from them).
void set_stats(TabArgs &a, const PrepJobs &j, const Mode &md)
{
    a.stats_a = j.stats_a;
    a.stats_b = j.stats_b;
    a.n_a = j.n_a;
    a.n_b = j.n_b;
    a.narrow = narrow_of(md);
}

// Products of a convolution pass (the same for the three passes).
inline double conv_macs(const ConvShape &s) { return double(s.n) * s.oh * s.ow * s.co * s.kh * s.kw * s.ci; }

inline dim3 dim3_of(const TabGrid &g) { return dim3(g.x, g.y, g.z); }

// The exact path's scaling for a format with fewer exponent bits (see tab_body).
void set_format_scales(TabArgs &a, const Mode &md)
{
    if (md.native || md.e_bits == 8) return;
    const int d2 = 2 * fmt_delta(md);  // 127 - beta, at most 126
    a.vadd = uint32_t(d2) << 23;
    a.su = std::ldexp(1.0f, d2);
    a.sd = std::ldexp(1.0f, -d2);
}

// ------------------------------------------------------------------ kernel timer --------

constexpr int kKernelKinds = 8;  // AMSIM_KERNEL_*

struct KernelTimer {
    std::mutex mu;
    bool active = false;
    unsigned kinds = 0u;  // bit k set: kernel kind k is timed
    std::vector<hipEvent_t> begin, end;
    std::vector<int> kind;
    size_t used = 0;
    int launches[kKernelKinds] = {};
    double total_ms[kKernelKinds] = {};
};

KernelTimer &timer()
{
    static KernelTimer t;
    return t;
}

// Brackets one main-kernel launch with events on its stream while profiling is active.
class TimedLaunch {
  public:
    TimedLaunch(int kind, hipStream_t st) : st_(st)
    {
        KernelTimer &t = timer();
        std::lock_guard<std::mutex> g(t.mu);
        if (t.active && ((t.kinds >> kind) & 1u) && t.used < t.begin.size()) {
            slot_ = long(t.used++);
            t.kind[size_t(slot_)] = kind;
            (void)hipEventRecord(t.begin[size_t(slot_)], st_);
        }
    }
    ~TimedLaunch()
    {
        if (slot_ < 0) return;
        KernelTimer &t = timer();
        std::lock_guard<std::mutex> g(t.mu);
        (void)hipEventRecord(t.end[size_t(slot_)], st_);
    }

  private:
    hipStream_t st_;
    long slot_ = -1;
};

void destroy_events(KernelTimer &t)
{
    for (hipEvent_t e : t.begin) (void)hipEventDestroy(e);
    for (hipEvent_t e : t.end) (void)hipEventDestroy(e);
    t.begin.clear();
    t.end.clear();
    t.kind.clear();
}

}  // namespace

// ==================================================================== C entry points =====

namespace {

// The table's row length for a call: the native multiply reads no table (its plan is M = 7's).
inline int plan_m(const Mode &md, int m_bits) { return md.native ? 7 : m_bits; }

// The column kernel's sums, per wave of its workgroup.
inline size_t gemv_sum_bytes(int mode) { return size_t(gv_waves(mode)) * kGemvCols * 64 * 4; }

inline size_t gemv_table_bytes(int mode, int m) { return mode == GV_TAB_LDS ? size_t(4) << (2 * m) : 0; }

template <bool VEC_FIRST, int MODE>
void launch_gemv(const VecPlan &vp, int64_t k, const float *vec, int64_t vs, const float *mat, int64_t so,
                 int64_t sk, float *out, int64_t os, float *part, const GvCtx &cx, hipStream_t st)
{
    const bool aligned = reinterpret_cast<uintptr_t>(mat) % 16 == 0;
    const size_t tab = gemv_table_bytes(MODE, cx.m);
    const dim3 grid(unsigned(vp.blocks), unsigned(vp.splits));
    if (!vp.rows) {  // so == 1
        const int v4 = aligned && sk % 4 == 0 ? 1 : 0;
        hipLaunchKernelGGL((gemv_cols_kernel<VEC_FIRST, MODE>), grid, dim3(64 * gv_waves(MODE)), tab + gemv_sum_bytes(MODE), st,
                           vp.nout, k, vec, vs, mat, sk, v4, out, os, part, vp.kchunk, cx);
    } else {  // sk == 1
        const int v4 = aligned && so % 4 == 0 ? 1 : 0;
        hipLaunchKernelGGL((gemv_rows_kernel<VEC_FIRST, MODE>), grid, dim3(64 * gv_waves(MODE)), tab, st, vp.nout, k,
                           vec, vs, mat, so, v4, out, os, part, vp.kchunk, cx);
    }
}

// m == 1: the vector op(A)(0, kk) = A[kk * a_sc], outputs C's columns; n == 1: the vector
// op(B)(kk, 0) = B[kk * b_sr], outputs C's rows.
template <int MODE>
void launch_gemv_mode(const VecPlan &vp, int64_t m, int64_t k, const float *A, int64_t a_sr, int64_t a_sc,
                      const float *B, int64_t b_sr, int64_t b_sc, float *C, int64_t ldc, float *part, const GvCtx &cx,
                      hipStream_t st)
{
    if (m == 1)
        launch_gemv<true, MODE>(vp, k, A, a_sc, B, b_sc, b_sr, C, 1, part, cx, st);
    else
        launch_gemv<false, MODE>(vp, k, B, b_sr, A, a_sr, a_sc, C, ldc, part, cx, st);
}

// Dynamic LDS beyond the default for the kernels that stage the table (called once).
hipError_t gemv_attributes()
{
    const int cols = int(gemv_table_bytes(GV_TAB_LDS, 7) + gemv_sum_bytes(GV_TAB_LDS));
    const int rows = int(gemv_table_bytes(GV_TAB_LDS, 7));
    hipError_t e = hipSuccess;
    for (hipError_t r :
         {hipFuncSetAttribute(reinterpret_cast<const void *>(gemv_cols_kernel<true, GV_TAB_LDS>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, cols),
          hipFuncSetAttribute(reinterpret_cast<const void *>(gemv_cols_kernel<false, GV_TAB_LDS>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, cols),
          hipFuncSetAttribute(reinterpret_cast<const void *>(gemv_rows_kernel<true, GV_TAB_LDS>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, rows),
          hipFuncSetAttribute(reinterpret_cast<const void *>(gemv_rows_kernel<false, GV_TAB_LDS>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, rows)})
        if (r != hipSuccess && e == hipSuccess) e = r;
    return e;
}

// Whether the vector kernels stage the table in LDS for a call (GV_TAB_LDS).
inline bool gemv_lds(const Mode &md, int m_bits) { return !md.native && md.e_bits == 8 && m_bits <= 7; }

// The GEMM with a vector operand or k == 1 (plan_vec): one kernel, plus the fixed-order
// reduction when the vector kernel splits k.
int vec_run(const Mode &md, const VecPlan &vp, int trans_a, int trans_b, int64_t m, int64_t n, int64_t k,
            const float *A, int64_t lda, const float *B, int64_t ldb, float *C, int64_t ldc, const uint32_t *lut,
            int m_bits, void *workspace, size_t workspace_bytes, hipStream_t st, int timer_kind)
{
    if (vp.total > 0 && (!workspace || workspace_bytes < vp.total)) return AMSIM_ERR_WORKSPACE;
    if (ensure_attributes() != AMSIM_OK) return AMSIM_ERR_HIP;
    // op(A)(i, kk) = A[i * a_sr + kk * a_sc], op(B)(kk, j) = B[kk * b_sr + j * b_sc]
    const int64_t a_sr = trans_a ? 1 : lda, a_sc = trans_a ? lda : 1;
    const int64_t b_sr = trans_b ? 1 : ldb, b_sc = trans_b ? ldb : 1;
    const int mb = plan_m(md, m_bits);
    TabArgs sc{};
    sc.vadd = 0u;
    sc.su = sc.sd = 1.0f;
    set_format_scales(sc, md);
    GvCtx cx{};
    cx.lut = lut;
    cx.tab = nullptr;
    cx.m = mb;
    cx.shift = 23 - mb;
    cx.fa = dec_fmt(md, mb, mb, 0u);  // index fields ka << M ...
    cx.fb = dec_fmt(md, mb, 0, 0u);   // ... and kb
    cx.vadd = sc.vadd;
    cx.su = sc.su;
    cx.sd = sc.sd;
    const bool narrow = !md.native && md.e_bits < 8;
    float *part = vp.kind == VEC_GEMV && vp.splits > 1 ? static_cast<float *>(workspace) : nullptr;
    {
        TimedLaunch tl(timer_kind, st);
        if (vp.kind == VEC_OUTER) {  // a_i = op(A)(i, 0), b_j = op(B)(0, j)
            const dim3 g(unsigned(grid_for(m * n)));
            if (md.native)
                hipLaunchKernelGGL((outer_kernel<true, false>), g, dim3(256), 0, st, m, n, A, a_sr, B, b_sc, C, ldc,
                                   lut, cx.fa, cx.fb, cx.vadd, cx.su, cx.sd);
            else if (narrow)
                hipLaunchKernelGGL((outer_kernel<false, true>), g, dim3(256), 0, st, m, n, A, a_sr, B, b_sc, C, ldc,
                                   lut, cx.fa, cx.fb, cx.vadd, cx.su, cx.sd);
            else
                hipLaunchKernelGGL((outer_kernel<false, false>), g, dim3(256), 0, st, m, n, A, a_sr, B, b_sc, C, ldc,
                                   lut, cx.fa, cx.fb, cx.vadd, cx.su, cx.sd);
        } else if (md.native) {
            launch_gemv_mode<GV_NATIVE>(vp, m, k, A, a_sr, a_sc, B, b_sr, b_sc, C, ldc, part, cx, st);
        } else if (narrow) {
            launch_gemv_mode<GV_NARROW>(vp, m, k, A, a_sr, a_sc, B, b_sr, b_sc, C, ldc, part, cx, st);
        } else if (mb <= 7) {
            launch_gemv_mode<GV_TAB_LDS>(vp, m, k, A, a_sr, a_sc, B, b_sr, b_sc, C, ldc, part, cx, st);
        } else {
            launch_gemv_mode<GV_TAB>(vp, m, k, A, a_sr, a_sc, B, b_sr, b_sc, C, ldc, part, cx, st);
        }
    }
    if (launch_status() != AMSIM_OK) return AMSIM_ERR_HIP;
    if (part != nullptr) {
        launch_reduce(part, vp.splits, m == 1 ? 1 : int(m), m == 1 ? int(n) : 1, C, ldc, st);
        return launch_status();
    }
    return AMSIM_OK;
}

// timer_kind: the kernel timer's kind for the main kernel (-1: the GEMM's).
int gemm_run(const Mode &md, int trans_a, int trans_b, int64_t m, int64_t n, int64_t k, const float *A, int64_t lda,
             const float *B, int64_t ldb, float *C, int64_t ldc, const uint32_t *lut, int m_bits, void *workspace,
             size_t workspace_bytes, hipStream_t st, int timer_kind = -1)
{
    if (timer_kind < 0) timer_kind = md.native ? AMSIM_KERNEL_GEMM_NATIVE : AMSIM_KERNEL_GEMM;
    if (!md.native && !valid_m(m_bits)) return AMSIM_ERR_UNSUPPORTED;
    if (m < 0 || n < 0 || k < 0) return AMSIM_ERR_INVALID_ARG;
    if (m == 0 || n == 0) return AMSIM_OK;
    if (!C || ldc < n) return AMSIM_ERR_INVALID_ARG;
    const int64_t lim = int64_t(1) << 31;
    if (m >= lim || n >= lim || k >= lim) return AMSIM_ERR_UNSUPPORTED;
    if (k == 0) {
        hipLaunchKernelGGL(fill_kernel, dim3(grid_for(m * n)), dim3(256), 0, st, C, int(m), int(n), ldc, -0.0f);
        return launch_status();
    }
    if (!A || !B || (!lut && !md.native)) return AMSIM_ERR_INVALID_ARG;
    if (lda < (trans_a ? m : k) || ldb < (trans_b ? k : n)) return AMSIM_ERR_INVALID_ARG;
    const VecPlan vp = plan_vec(m, n, k, trans_a, trans_b, gemv_lds(md, m_bits));
    if (vp.kind != VEC_NONE)
        return vec_run(md, vp, trans_a, trans_b, m, n, k, A, lda, B, ldb, C, ldc, lut, m_bits, workspace,
                       workspace_bytes, st, timer_kind);
    const int mb = plan_m(md, m_bits);
    const Plan p = plan_gemm(m, n, k, mb);
    if (!gemm_fits(p, m, n, k)) return AMSIM_ERR_UNSUPPORTED;
    if (p.total > 0 && (!workspace || workspace_bytes < p.total)) return AMSIM_ERR_WORKSPACE;
    if (ensure_attributes() != AMSIM_OK) return AMSIM_ERR_HIP;
    char *ws = static_cast<char *>(workspace);
    uint32_t *Ad = reinterpret_cast<uint32_t *>(ws + p.off_a);
    uint32_t *Bd = reinterpret_cast<uint32_t *>(ws + p.off_b);
    float *out = p.splits > 1 ? reinterpret_cast<float *>(ws + p.off_part) : C;
    // op(A)(i, kk): row stride / column stride in A's storage
    const int64_t a_sr = trans_a ? 1 : lda, a_sc = trans_a ? lda : 1;
    const int64_t b_sr = trans_b ? 1 : ldb, b_sc = trans_b ? ldb : 1;
    PrepJobs j = prep_jobs(md, lut, mb, ws, p);
    const int gx = int(std::min<int64_t>(ceil_div(p.a_ld, 64), 128)), gy = int(std::min<int64_t>(ceil_div(k, 64), 64));
    const DecT da{A, a_sr, a_sc, int(m), int(k), nullptr, int(p.a_ld), Ad, gx};
    j.n_a = gx * gy;  // <= kStatSlots
    j.b = DecRows{B, 0, b_sr, b_sc, 1, int(k), int(k), int(n), Bd, int(p.b_ld), decode_vec(B, 0, b_sr, b_sc)};
    j.n_b = decode_grid(k * p.b_ld);
    const int var = tab_variant(md, p, double(m) * double(n) * double(k));
    if (run_prepass(j, da, 0, var, narrow_of(md), st) != AMSIM_OK) return AMSIM_ERR_HIP;
    int rc;
    {
        TabArgs a = tab_args(gemm_geom(p, m, n, k, ldc), p, ws, Ad, Bd, out);
        set_stats(a, j, md);
        set_format_scales(a, md);
        const dim3 grid = dim3_of(gemm_grid(p));
        TimedLaunch tl(timer_kind, st);
        rc = tab_launch<OP_GEMM>(p.tile, p.rl, var, a, grid, st) == hipSuccess
                 ? AMSIM_OK
                 : AMSIM_ERR_HIP;
    }
    if (rc != AMSIM_OK) return AMSIM_ERR_HIP;
    if (p.splits > 1) {
        launch_reduce(reinterpret_cast<const float *>(ws + p.off_part), p.splits, int(m), int(n), C, ldc, st);
        if (launch_status() != AMSIM_OK) return AMSIM_ERR_HIP;
    }
    return AMSIM_OK;
}

// A convolution pass that runs as its GEMM (conv_runs_as_gemm): validated as a convolution, run as
// the GEMM, timed as the pass.  in0 / in1: the pass's first and second operands, as for the
// convolution.
int conv_gemm_run(const Mode &md, const amsim_conv2d *desc, int pass, const float *in0, const float *in1, float *out,
                  const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes, hipStream_t st)
{
    if (!md.native && !valid_m(m_bits)) return AMSIM_ERR_UNSUPPORTED;
    const int rc = check_conv(desc, pass);
    if (rc != AMSIM_OK) return rc;
    if (!in0 || !in1 || !out || (!lut && !md.native)) return AMSIM_ERR_INVALID_ARG;
    static const int kinds[3][2] = {{AMSIM_KERNEL_CONV_FWD, AMSIM_KERNEL_CONV_FWD_NATIVE},
                                    {AMSIM_KERNEL_CONV_BWD_DATA, AMSIM_KERNEL_CONV_BWD_DATA_NATIVE},
                                    {AMSIM_KERNEL_CONV_BWD_WEIGHT, AMSIM_KERNEL_CONV_BWD_WEIGHT_NATIVE}};
    const ConvGemm g = conv_gemm(desc, pass);
    // backward data: the second operand w[ci][co] read transposed
    return gemm_run(md, g.trans_a, g.trans_b, g.m, g.n, g.k, in0, g.lda, in1, g.ldb, out, g.ldc, lut, m_bits, workspace,
                    workspace_bytes, st, kinds[pass][md.native ? 1 : 0]);
}

// Whether a call's pass runs as its GEMM: a valid pass that conv_runs_as_gemm accepts (the same
// decision as the workspace query's; the native multiply's m_bits, which it ignores, counts as 7).
inline bool pass_as_gemm(const amsim_conv2d *desc, int pass, int m_bits)
{
    return desc && check_conv(desc, pass) == AMSIM_OK && conv_runs_as_gemm(desc, pass, valid_m(m_bits) ? m_bits : 7);
}

int conv_common(const Mode &md, const amsim_conv2d *desc, int pass, const void *in0, const void *in1, void *out,
                const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes, Plan *p)
{
    if (!md.native && !valid_m(m_bits)) return AMSIM_ERR_UNSUPPORTED;
    const int rc = check_conv(desc, pass);
    if (rc != AMSIM_OK) return rc;
    if (!in0 || !in1 || !out || (!lut && !md.native)) return AMSIM_ERR_INVALID_ARG;
    *p = plan_conv(desc, pass, plan_m(md, m_bits));
    if (p->total > 0 && (!workspace || workspace_bytes < p->total)) return AMSIM_ERR_WORKSPACE;
    if (ensure_attributes() != AMSIM_OK) return AMSIM_ERR_HIP;
    return AMSIM_OK;
}

// The first operand as step-pair records [n][hp][cp][wp] of an NHWC tensor inside its zero border
// (decode_a_body for DecNhcw): the channels per LDS chunk and the workgroups (one (padded row,
// chunk) item at a time); rec_c: channels of a record row (cp = ceil(rec_c / 2) records).
DecNhcw nhcw_job(const float *src, int n, int h, int w, int c, int top, int left, int hp, int wp, uint32_t *dst,
                 int rec_c, int *blocks, size_t *lds)
{
    int cc = std::max(2, std::min(c, kNhcwTile / (w | 1)));  // channels per LDS tile
    // few rows: narrower chunks, so that about 2048 (row, chunk) items keep the copy parallel
    const int64_t rows = int64_t(n) * hp;
    if (rows < 2048) cc = std::max(2, std::min(cc, int(ceil_div(c, ceil_div(2048, rows)))));
    if (cc < c) cc = std::max(2, cc & ~1);  // chunks hold whole channel pairs
    if (c % 4 == 0 && cc < c && cc >= 4) cc &= ~3;  // four-channel loads where every chunk allows them
    const int vec = c % 4 == 0 && cc % 4 == 0 && reinterpret_cast<uintptr_t>(src) % 16 == 0 ? 1 : 0;
    const int64_t items = rows * ceil_div(c, cc);
    *blocks = int(std::min<int64_t>(items, kStatSlots));
    *lds = size_t(cc) * (w | 1) * 4;
    return DecNhcw{src, n, h, w, c, top, left, hp, wp, dst, cc, (rec_c + 1) / 2, vec};
}

// The forward pass of desc.  flip_w: w is a backward-data pass's [kh][kw][c_out][c_in] weights (of
// the caller's convolution, whose c_in / c_out are desc's c_out / c_in), read flipped in both
// kernel axes and transposed (bwd_data_runs_as_fwd); timer_kind: the kernel timer's slot.
int fwd_core(const Mode &md, const amsim_conv2d *desc, const float *x, const float *w, bool flip_w, float *y,
             const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes, hipStream_t st, int timer_kind)
{
    Plan p;
    int rc = conv_common(md, desc, AMSIM_CONV_FWD, x, w, y, lut, m_bits, workspace, workspace_bytes, &p);
    if (rc != AMSIM_OK) return rc;
    const int mb = plan_m(md, m_bits);
    const ConvShape s = shape_of(desc);
    char *ws = static_cast<char *>(workspace);
    uint32_t *Xd = reinterpret_cast<uint32_t *>(ws + p.off_a);
    uint32_t *Wd = reinterpret_cast<uint32_t *>(ws + p.off_b);
    const int64_t rows = int64_t(s.n) * s.oh * s.ow;
    float *out = p.splits > 1 ? reinterpret_cast<float *>(ws + p.off_part) : y;
    PrepJobs j = prep_jobs(md, lut, mb, ws, p);
    // w [kh][kw * ci][co] as batches kh of kw * ci rows (unfolded: padded to cu rows with +0)
    const int kwc = s.kw * s.ci, wrows = p.unfold_w ? unfolded_channels(s) : kwc;
    if (flip_w)  // batches (kh, kw) of ci rows [kh][kw][ci][co] = w[KH-1-kh][KW-1-kw][co][ci]: the last
                 // kernel position first, rows ci at unit stride, columns co at stride ci
        j.b = DecRows{w + (int64_t(s.kh) * s.kw - 1) * s.ci * s.co, -int64_t(s.ci) * s.co, 1, int64_t(s.ci),
                      s.kh * s.kw, s.ci, s.ci, s.co, Wd, int(p.b_ld), 0};
    else
        j.b = DecRows{w, int64_t(kwc) * s.co, int64_t(s.co), 1, s.kh, wrows, kwc, s.co, Wd, int(p.b_ld),
                      decode_vec(w, int64_t(kwc) * s.co, s.co, 1)};
    j.n_b = decode_grid(int64_t(s.kh) * wrows * p.b_ld);
    const int var = tab_variant(md, p, conv_macs(s));
    if (p.unfold_w) {
        j.n_a = int(std::min<int64_t>(int64_t(s.n) * p.Hp, kStatSlots));  // one padded image row at a time
        const DecUnfold da{x, s.n, s.h, s.w, s.ci, s.pt, s.pl, p.Hp, s.kw, s.sw, s.ow, Xd};
        rc = run_prepass(j, da, size_t(s.w) * s.ci * 4, var, narrow_of(md), st);
    } else {
        size_t lds;
        const DecNhcw da = nhcw_job(x, s.n, s.h, s.w, s.ci, s.pt, s.pl, p.Hp, p.Wp, Xd, p.rec_c, &j.n_a, &lds);
        rc = run_prepass(j, da, lds, var, narrow_of(md), st);
    }
    if (rc != AMSIM_OK) return AMSIM_ERR_HIP;
    TabArgs a = tab_args(fwd_geom(p, s), p, ws, Xd, Wd, out);
    set_stats(a, j, md);
    set_format_scales(a, md);
    const dim3 grid = dim3_of(fwd_grid(p, s));
    {
        TimedLaunch tl(timer_kind, st);
        rc = tab_launch<OP_FWD>(p.tile, p.rl, var, a, grid, st) == hipSuccess
                 ? AMSIM_OK
                 : AMSIM_ERR_HIP;
    }
    if (rc != AMSIM_OK || p.splits == 1) return rc;
    launch_reduce(reinterpret_cast<const float *>(ws + p.off_part), p.splits, int(rows), s.co, y, int64_t(s.co), st);
    return launch_status();
}

int conv_fwd_run(const Mode &md, const amsim_conv2d *desc, const float *x, const float *w, float *y,
                 const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes, hipStream_t st)
{
    if (pass_as_gemm(desc, AMSIM_CONV_FWD, m_bits))
        return conv_gemm_run(md, desc, AMSIM_CONV_FWD, x, w, y, lut, m_bits, workspace, workspace_bytes, st);
    return fwd_core(md, desc, x, w, false, y, lut, m_bits, workspace, workspace_bytes, st,
                    md.native ? AMSIM_KERNEL_CONV_FWD_NATIVE : AMSIM_KERNEL_CONV_FWD);
}

// The backward-data pass of `desc` (the caller's, or the virtual unfolded one) under plan p, into dx.
// fixup: apply the dilation taps' products to dx here (the unfolded pass leaves them to the fold).
// zf: the zero-tap flags the pre-pass computes (none when zf.total() == 0).
int bwd_data_run(const Mode &md, const amsim_conv2d *desc, const Plan &p, const float *dy, const float *w, float *dx,
                 const uint32_t *lut, int m_bits, void *workspace, hipStream_t st, bool fixup, const ZeroTapFlags &zf)
{
    int rc;
    const int mb = plan_m(md, m_bits);
    const ConvShape s = shape_of(desc);
    char *ws = static_cast<char *>(workspace);
    uint32_t *Dyd = reinterpret_cast<uint32_t *>(ws + p.off_a);
    uint32_t *Wtd = reinterpret_cast<uint32_t *>(ws + p.off_b);
    float *out = p.splits > 1 ? reinterpret_cast<float *>(ws + p.off_part) : dx;
    PrepJobs j = prep_jobs(md, lut, mb, ws, p);
    j.z = zf;
    j.n_flag = std::min(zf.total(), 65535);
    size_t lds;
    const DecNhcw da =
        nhcw_job(dy, s.n, s.oh, s.ow, s.co, p.pad_oh, p.pad_ow, p.OHp, p.OWp, Dyd, p.rec_c, &j.n_a, &lds);
    // w[kh][kw][ci][co] -> Wt[kh][kw][co][ci]: batches (kh,kw), rows co, cols ci
    j.b = DecRows{w, int64_t(s.ci) * s.co, 1, int64_t(s.co), s.kh * s.kw, s.co, s.co, s.ci, Wtd, int(p.b_ld), 0};
    j.n_b = decode_grid(int64_t(s.kh) * s.kw * s.co * p.b_ld);
    const int var = tab_variant(md, p, conv_macs(s));
    if (run_prepass(j, da, lds, var, narrow_of(md), st) != AMSIM_OK) return AMSIM_ERR_HIP;
    TabArgs a = tab_args(bwd_data_geom(p, s), p, ws, Dyd, Wtd, out);
    set_stats(a, j, md);
    set_format_scales(a, md);
    const dim3 grid = dim3_of(bwd_data_grid(p, s));
    {
        TimedLaunch tl(md.native ? AMSIM_KERNEL_CONV_BWD_DATA_NATIVE : AMSIM_KERNEL_CONV_BWD_DATA, st);
        rc = tab_launch<OP_BWD_DATA>(p.tile, p.rl, var, a, grid, st) == hipSuccess
                 ? AMSIM_OK
                 : AMSIM_ERR_HIP;
    }
    if (rc != AMSIM_OK) return rc;
    if (p.splits > 1) {
        launch_reduce(reinterpret_cast<const float *>(ws + p.off_part), p.splits, s.n * s.h * s.w, s.ci, dx,
                      int64_t(s.ci), st);
        if (launch_status() != AMSIM_OK) return AMSIM_ERR_HIP;
    }
    if (fixup && s.sh * s.sw > 1) {  // the taps outside each output's stride phase (dilation zeros)
        const int total = s.n * s.h * s.w * s.ci;
        hipLaunchKernelGGL(dilation_fixup_kernel, dim3(grid_for(total)), dim3(256), 0, st, dx, total, s.h, s.w, s.ci,
                           s.sh, s.sw, zf.phase_flags);
    }
    return launch_status();
}

int conv_bwd_data_run(const Mode &md, const amsim_conv2d *desc, const float *dy, const float *w, float *dx,
                      const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes, hipStream_t st)
{
    if (pass_as_gemm(desc, AMSIM_CONV_BWD_DATA, m_bits))
        return conv_gemm_run(md, desc, AMSIM_CONV_BWD_DATA, dy, w, dx, lut, m_bits, workspace, workspace_bytes, st);
    if (desc && check_conv(desc, AMSIM_CONV_BWD_DATA) == AMSIM_OK && bwd_data_runs_as_fwd(desc)) {
        const amsim_conv2d f = bwd_data_fwd_desc(desc);
        return fwd_core(md, &f, dy, w, true, dx, lut, m_bits, workspace, workspace_bytes, st,
                        md.native ? AMSIM_KERNEL_CONV_BWD_DATA_NATIVE : AMSIM_KERNEL_CONV_BWD_DATA);
    }
    Plan p;
    int rc = conv_common(md, desc, AMSIM_CONV_BWD_DATA, dy, w, dx, lut, m_bits, workspace, workspace_bytes, &p);
    if (rc != AMSIM_OK) return rc;
    uint32_t *pf = reinterpret_cast<uint32_t *>(static_cast<char *>(workspace) + p.off_bflags);
    if (!p.unfold_w) {
        ZeroTapFlags zf{};
        if (desc->stride_h * desc->stride_w > 1)  // the taps outside each output's stride phase
            zf = ZeroTapFlags{w,  desc->kh, desc->kw, desc->c_in, desc->c_out, desc->stride_h, desc->stride_w,
                              desc->pad_top, desc->pad_left, fmt_hi(md), md.sat, pf, nullptr};
        return bwd_data_run(md, desc, p, dy, w, dx, lut, m_bits, workspace, st, true, zf);
    }
    // the unfolded input's gradient, then folded back onto x's pixels.  The pre-pass computes the
    // flags over the virtual pass's weights [kh][kw * c][co] (the caller's [kh][kw][c][co]): the
    // virtual pass's row-phase flags (stride_h > 1), then, per unfolded channel kw * c + ci, the
    // flags of the kw taps that reach no output column (see fold_w_kernel).  The fold applies both.
    const amsim_conv2d v = unfolded_desc(desc);
    float *dxu = reinterpret_cast<float *>(static_cast<char *>(workspace) + p.off_unf);
    const int phases = v.stride_h;  // the virtual pass's stride along w is 1
    uint32_t *kf = pf + size_t(phases) * v.c_in;
    const ZeroTapFlags zf{w, v.kh, 1, v.c_in, v.c_out, v.stride_h, 1, v.pad_top, 0, fmt_hi(md), md.sat,
                          phases > 1 ? pf : nullptr, kf};
    rc = bwd_data_run(md, &v, p, dy, w, dxu, lut, m_bits, workspace, st, false, zf);
    if (rc != AMSIM_OK) return rc;
    const int total = desc->n * desc->h * desc->w * desc->c_in;
    hipLaunchKernelGGL(fold_w_kernel, dim3(grid_for(total)), dim3(256), 0, st, dxu, desc->n, desc->h, desc->w,
                       desc->c_in, desc->kw, desc->stride_w, desc->pad_left, v.w, kf, phases > 1 ? pf : nullptr,
                       phases, dx);
    return launch_status();
}

int conv_bwd_weight_run(const Mode &md, const amsim_conv2d *desc, const float *x, const float *dy, float *dw,
                        const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes, hipStream_t st)
{
    if (pass_as_gemm(desc, AMSIM_CONV_BWD_WEIGHT, m_bits))
        return conv_gemm_run(md, desc, AMSIM_CONV_BWD_WEIGHT, x, dy, dw, lut, m_bits, workspace, workspace_bytes, st);
    Plan p;
    int rc = conv_common(md, desc, AMSIM_CONV_BWD_WEIGHT, x, dy, dw, lut, m_bits, workspace, workspace_bytes, &p);
    if (rc != AMSIM_OK) return rc;
    const int mb = plan_m(md, m_bits);
    const ConvShape s = shape_of(desc);
    char *ws = static_cast<char *>(workspace);
    uint32_t *Xd = reinterpret_cast<uint32_t *>(ws + p.off_a);
    uint32_t *Dyd = reinterpret_cast<uint32_t *>(ws + p.off_b);
    PrepJobs j = prep_jobs(md, lut, mb, ws, p);
    // x as step-pair records inside its zero border, one padded image row per workgroup at a time
    const int64_t wc = int64_t(s.w) * s.ci;
    const int row_lds = wc <= kPairsRowWords ? 1 : 0;
    const int vec = wc % 4 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0 ? 1 : 0;
    const DecPairs da{x, s.n, s.h, s.w, s.ci, s.pt, s.pl, p.Hp, p.Wp, s.sw, Xd, row_lds, vec};
    j.n_a = int(std::min<int64_t>(int64_t(s.n) * p.Hp, kStatSlots));
    const int64_t npo = int64_t(s.n) * s.oh * s.ow;
    j.b = DecRows{dy, 0, int64_t(s.co), 1, 1, int(npo), int(npo), s.co, Dyd, int(p.b_ld), decode_vec(dy, 0, s.co, 1)};
    j.n_b = decode_grid(npo * p.b_ld);
    const int var = tab_variant(md, p, conv_macs(s));
    if (run_prepass(j, da, row_lds ? size_t(wc) * 4 : 0, var, narrow_of(md), st) != AMSIM_OK) return AMSIM_ERR_HIP;
    const int R = s.kh * s.kw * s.ci;
    float *out = p.splits > 1 ? reinterpret_cast<float *>(ws + p.off_part) : dw;
    {
        TimedLaunch tl(md.native ? AMSIM_KERNEL_CONV_BWD_WEIGHT_NATIVE : AMSIM_KERNEL_CONV_BWD_WEIGHT, st);
        TabArgs a = tab_args(bwd_weight_geom(p, s), p, ws, Xd, Dyd, out);
        set_stats(a, j, md);
        set_format_scales(a, md);
        const dim3 grid = dim3_of(bwd_weight_grid(p, s));
        rc = tab_launch<OP_BWD_WEIGHT>(p.tile, p.rl, var, a, grid, st) == hipSuccess
                 ? AMSIM_OK
                 : AMSIM_ERR_HIP;
    }
    if (rc != AMSIM_OK) return AMSIM_ERR_HIP;
    if (p.splits > 1) {
        launch_reduce(reinterpret_cast<const float *>(ws + p.off_part), p.splits, R, s.co, dw, int64_t(s.co), st);
        return launch_status();
    }
    return AMSIM_OK;
}

// ------------------------------------------------------------------ fixed scratch -------
// The workspace of approx_gemm_noalloc: one array per GPU, held from the library's load until the
// process ends.  Host code never names it directly (its host-side name is a stand-in, not a
// device address): scratch_address gets each device's address once, with that device current.
constexpr size_t kScratchBytes = size_t(AMSIM_NOALLOC_SCRATCH_BYTES);
static_assert(kScratchBytes % kAlign == 0, "the plans' offsets assume an aligned base");
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxScratchDevices] = {};

// The current device's copy of `scratch` (looked up on the first call per device).
int scratch_address(void **ptr)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return AMSIM_ERR_HIP;
    if (dev < 0 || dev >= kMaxScratchDevices) return AMSIM_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return AMSIM_ERR_HIP;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return AMSIM_OK;
}

}  // namespace

extern "C" {

int approx_gemm_noalloc(int trans_a, int trans_b, int64_t m, int64_t n, int64_t k, const float *A, int64_t lda,
                        const float *B, int64_t ldb, float *C, int64_t ldc, const uint32_t *lut, int m_bits,
                        void *stream)
{
    // the same argument checks as approx_gemm, then the plan's size against the fixed buffer
    if (!valid_m(m_bits)) return AMSIM_ERR_UNSUPPORTED;
    if (m < 0 || n < 0 || k < 0) return AMSIM_ERR_INVALID_ARG;
    size_t need = 0;
    if (m > 0 && n > 0 && k > 0) {
        const int64_t lim = int64_t(1) << 31;
        if (m >= lim || n >= lim || k >= lim) return AMSIM_ERR_UNSUPPORTED;
        const VecPlan vp = plan_vec(m, n, k, trans_a, trans_b, gemv_lds(Mode{}, m_bits));
        need = vp.kind != VEC_NONE ? vp.total : plan_gemm(m, n, k, m_bits).total;
    }
    if (need > kScratchBytes) return AMSIM_ERR_SCRATCH;
    void *ws = nullptr;
    if (need > 0) {
        const int rc = scratch_address(&ws);
        if (rc != AMSIM_OK) return rc;
    }
    return gemm_run(Mode{}, trans_a, trans_b, m, n, k, A, lda, B, ldb, C, ldc, lut, m_bits, ws, kScratchBytes,
                    static_cast<hipStream_t>(stream));
}

int amsim_gemm_workspace_size(int trans_a, int trans_b, int64_t m, int64_t n, int64_t k, int m_bits, size_t *bytes)
{
    if (!bytes) return AMSIM_ERR_INVALID_ARG;
    if (!valid_m(m_bits)) return AMSIM_ERR_UNSUPPORTED;
    if (m < 0 || n < 0 || k < 0) return AMSIM_ERR_INVALID_ARG;
    *bytes = gemm_workspace_bytes(trans_a, trans_b, m, n, k, m_bits);
    return AMSIM_OK;
}

int approx_gemm(int trans_a, int trans_b, int64_t m, int64_t n, int64_t k, const float *A, int64_t lda,
                const float *B, int64_t ldb, float *C, int64_t ldc, const uint32_t *lut, int m_bits, void *workspace,
                size_t workspace_bytes, void *stream)
{
    return gemm_run(Mode{}, trans_a, trans_b, m, n, k, A, lda, B, ldb, C, ldc, lut, m_bits, workspace,
                    workspace_bytes, static_cast<hipStream_t>(stream));
}

int approx_gemm_ex(const amsim_options *opt, int trans_a, int trans_b, int64_t m, int64_t n, int64_t k,
                   const float *A, int64_t lda, const float *B, int64_t ldb, float *C, int64_t ldc, const uint32_t *lut,
                   int m_bits, void *workspace, size_t workspace_bytes, void *stream)
{
    Mode md;
    const int rc = mode_of(opt, md);
    if (rc != AMSIM_OK) return rc;
    return gemm_run(md, trans_a, trans_b, m, n, k, A, lda, B, ldb, C, ldc, lut, m_bits, workspace, workspace_bytes,
                    static_cast<hipStream_t>(stream));
}

int amsim_conv2d_workspace_size(const amsim_conv2d *desc, int pass, int m_bits, size_t *bytes)
{
    if (!bytes) return AMSIM_ERR_INVALID_ARG;
    if (!valid_m(m_bits)) return AMSIM_ERR_UNSUPPORTED;
    if (pass < AMSIM_CONV_FWD || pass > AMSIM_CONV_BWD_WEIGHT) return AMSIM_ERR_INVALID_ARG;
    const int rc = check_conv(desc, pass);
    if (rc != AMSIM_OK) return rc;
    if (conv_runs_as_gemm(desc, pass, m_bits)) {
        const ConvGemm g = conv_gemm(desc, pass);
        *bytes = gemm_workspace_bytes(g.trans_a, g.trans_b, g.m, g.n, g.k, m_bits);
        return AMSIM_OK;
    }
    if (pass == AMSIM_CONV_BWD_DATA && bwd_data_runs_as_fwd(desc)) {
        const amsim_conv2d f = bwd_data_fwd_desc(desc);
        *bytes = std::max(plan_conv(&f, AMSIM_CONV_FWD, m_bits).total, plan_conv(&f, AMSIM_CONV_FWD, 7).total);
        return AMSIM_OK;
    }
    *bytes = std::max(plan_conv(desc, pass, m_bits).total, plan_conv(desc, pass, 7).total);
    return AMSIM_OK;
}

int approx_conv2d_fwd(const amsim_conv2d *desc, const float *x, const float *w, float *y, const uint32_t *lut,
                      int m_bits, void *workspace, size_t workspace_bytes, void *stream)
{
    return conv_fwd_run(Mode{}, desc, x, w, y, lut, m_bits, workspace, workspace_bytes,
                        static_cast<hipStream_t>(stream));
}

int approx_conv2d_bwd_data(const amsim_conv2d *desc, const float *dy, const float *w, float *dx,
                           const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes, void *stream)
{
    return conv_bwd_data_run(Mode{}, desc, dy, w, dx, lut, m_bits, workspace, workspace_bytes,
                             static_cast<hipStream_t>(stream));
}

int approx_conv2d_bwd_weight(const amsim_conv2d *desc, const float *x, const float *dy, float *dw,
                             const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes, void *stream)
{
    return conv_bwd_weight_run(Mode{}, desc, x, dy, dw, lut, m_bits, workspace, workspace_bytes,
                               static_cast<hipStream_t>(stream));
}

int approx_conv2d_fwd_ex(const amsim_options *opt, const amsim_conv2d *desc, const float *x, const float *w, float *y,
                         const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes, void *stream)
{
    Mode md;
    const int rc = mode_of(opt, md);
    if (rc != AMSIM_OK) return rc;
    return conv_fwd_run(md, desc, x, w, y, lut, m_bits, workspace, workspace_bytes, static_cast<hipStream_t>(stream));
}

int approx_conv2d_bwd_data_ex(const amsim_options *opt, const amsim_conv2d *desc, const float *dy, const float *w,
                              float *dx, const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes,
                              void *stream)
{
    Mode md;
    const int rc = mode_of(opt, md);
    if (rc != AMSIM_OK) return rc;
    return conv_bwd_data_run(md, desc, dy, w, dx, lut, m_bits, workspace, workspace_bytes,
                             static_cast<hipStream_t>(stream));
}

int approx_conv2d_bwd_weight_ex(const amsim_options *opt, const amsim_conv2d *desc, const float *x, const float *dy,
                                float *dw, const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes,
                                void *stream)
{
    Mode md;
    const int rc = mode_of(opt, md);
    if (rc != AMSIM_OK) return rc;
    return conv_bwd_weight_run(md, desc, x, dy, dw, lut, m_bits, workspace, workspace_bytes,
                               static_cast<hipStream_t>(stream));
}

int approx_gemm_direct(int mode, int m_bits, int64_t m, int64_t n, int64_t k, const float *A, int64_t lda,
                       const float *B, int64_t ldb, float *C, int64_t ldc, void *stream)
{
    if (mode != AMSIM_DIRECT_NATIVE && mode != AMSIM_DIRECT_MITCHELL) return AMSIM_ERR_INVALID_ARG;
    if (mode == AMSIM_DIRECT_MITCHELL && !valid_m(m_bits)) return AMSIM_ERR_UNSUPPORTED;
    if (m < 0 || n < 0 || k < 0) return AMSIM_ERR_INVALID_ARG;
    if (m == 0 || n == 0) return AMSIM_OK;
    if (!C || ldc < n) return AMSIM_ERR_INVALID_ARG;
    const int64_t lim = int64_t(1) << 31;
    if (m >= lim || n >= lim || k >= lim || ceil_div(n, kDirTile) > 65535) return AMSIM_ERR_UNSUPPORTED;
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (k == 0) {
        hipLaunchKernelGGL(fill_kernel, dim3(grid_for(m * n)), dim3(256), 0, st, C, int(m), int(n), ldc, -0.0f);
        return launch_status();
    }
    if (!A || !B || lda < k || ldb < n) return AMSIM_ERR_INVALID_ARG;
    const dim3 grid(unsigned(ceil_div(m, kDirTile)), unsigned(ceil_div(n, kDirTile)));
    if (mode == AMSIM_DIRECT_NATIVE)
        hipLaunchKernelGGL(direct_gemm_kernel<DIRECT_NATIVE>, grid, dim3(256), 0, st, A, lda, B, ldb, C, ldc, int(m),
                           int(n), int(k), 0);
    else
        hipLaunchKernelGGL(direct_gemm_kernel<DIRECT_MITCHELL>, grid, dim3(256), 0, st, A, lda, B, ldb, C, ldc,
                           int(m), int(n), int(k), m_bits);
    return launch_status();
}

int approx_mul_ew(int64_t n, const float *a, const float *b, float *c, const uint32_t *lut, int m_bits, void *stream)
{
    return approx_mul_ew_ex(nullptr, n, a, b, c, lut, m_bits, stream);
}

int approx_mul_ew_ex(const amsim_options *opt, int64_t n, const float *a, const float *b, float *c,
                     const uint32_t *lut, int m_bits, void *stream)
{
    Mode md;
    const int rc = mode_of(opt, md);
    if (rc != AMSIM_OK) return rc;
    if (md.native) return AMSIM_ERR_UNSUPPORTED;  // element-wise products are the table's
    if (!valid_m(m_bits)) return AMSIM_ERR_UNSUPPORTED;
    if (n < 0) return AMSIM_ERR_INVALID_ARG;
    if (n == 0) return AMSIM_OK;
    if (!a || !b || !c || !lut) return AMSIM_ERR_INVALID_ARG;
    hipStream_t st = static_cast<hipStream_t>(stream);
    TabArgs sc{};
    sc.vadd = 0u;
    sc.su = sc.sd = 1.0f;
    set_format_scales(sc, md);
    hipLaunchKernelGGL(mul_ew_kernel, dim3(grid_for(n)), dim3(256), 0, st, n, a, b, c, lut,
                       dec_fmt(md, m_bits, m_bits, 0u), dec_fmt(md, m_bits, 0, 0u), sc.vadd, sc.su, sc.sd);
    return launch_status();
}

int amsim_cast_exponent(int e_bits, int exp_cast, int m_bits, int64_t n, const float *x, float *y, void *stream)
{
    const amsim_options o{AMSIM_MULTIPLY_TABLE, e_bits, exp_cast};
    Mode md;
    const int rc = mode_of(&o, md);
    if (rc != AMSIM_OK) return rc;
    if (!valid_m(m_bits)) return AMSIM_ERR_UNSUPPORTED;
    if (n < 0) return AMSIM_ERR_INVALID_ARG;
    if (n == 0) return AMSIM_OK;
    if (!x || !y) return AMSIM_ERR_INVALID_ARG;
    DecFmt f = dec_fmt(md, m_bits, 0, 0u);
    hipLaunchKernelGGL(cast_kernel, dim3(grid_for(n)), dim3(256), 0, static_cast<hipStream_t>(stream), n, x, y, f);
    return launch_status();
}

int amsim_profile_start(int max_launches) { return amsim_profile_start_kinds(max_launches, (1u << kKernelKinds) - 1u); }

int amsim_profile_start_kinds(int max_launches, unsigned kinds)
{
    if (max_launches < 1 || kinds == 0u || (kinds >> kKernelKinds) != 0u) return AMSIM_ERR_INVALID_ARG;
    KernelTimer &t = timer();
    std::lock_guard<std::mutex> g(t.mu);
    t.active = false;
    t.kinds = kinds;
    destroy_events(t);
    t.used = 0;
    for (int k = 0; k < kKernelKinds; ++k) {
        t.launches[k] = 0;
        t.total_ms[k] = 0.0;
    }
    t.begin.resize(size_t(max_launches));
    t.end.resize(size_t(max_launches));
    t.kind.assign(size_t(max_launches), 0);
    for (int i = 0; i < max_launches; ++i) {
        // Timing-only events: no system-scope fence when they complete.  That fence writes back and
        // invalidates the caches; measured on MI355X, it left ~5.6 us idle on each side of a table
        // kernel (where the step's launches otherwise follow one another with no gap).
        hipEvent_t b = nullptr, e = nullptr;
        if (hipEventCreateWithFlags(&b, hipEventDisableSystemFence) != hipSuccess ||
            hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) {
            if (b != nullptr) (void)hipEventDestroy(b);
            t.begin.resize(size_t(i));
            t.end.resize(size_t(i));
            destroy_events(t);
            return AMSIM_ERR_HIP;
        }
        t.begin[size_t(i)] = b;
        t.end[size_t(i)] = e;
    }
    t.active = true;
    return AMSIM_OK;
}

int amsim_profile_stop(void)
{
    KernelTimer &t = timer();
    std::lock_guard<std::mutex> g(t.mu);
    t.active = false;
    int rc = AMSIM_OK;
    for (size_t i = 0; i < t.used; ++i) {
        float ms = 0.f;
        if (hipEventSynchronize(t.end[i]) != hipSuccess || hipEventElapsedTime(&ms, t.begin[i], t.end[i]) != hipSuccess) {
            rc = AMSIM_ERR_HIP;
            continue;
        }
        t.launches[t.kind[i]] += 1;
        t.total_ms[t.kind[i]] += double(ms);
    }
    t.used = 0;
    return rc;
}

int amsim_profile_read(int kind, int *launches, double *total_ms)
{
    if (kind < 0 || kind >= kKernelKinds || !launches || !total_ms) return AMSIM_ERR_INVALID_ARG;
    KernelTimer &t = timer();
    std::lock_guard<std::mutex> g(t.mu);
    *launches = t.launches[kind];
    *total_ms = t.total_ms[kind];
    return AMSIM_OK;
}

}  // extern "C"
