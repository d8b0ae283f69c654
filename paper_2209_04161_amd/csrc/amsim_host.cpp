// amsim_host.cpp -- host side of the library: built-in functional multiplier models, the
// table generator (Algorithm 1 of ApproxTrain, arXiv 2209.04161), table files and status
// strings.  No HIP calls live here.
#include <cstdint>
#include <cstdio>
#include <cstring>

#include "amsim.h"

namespace {

inline uint32_t f2u(float f)
{
    uint32_t u;
    std::memcpy(&u, &f, 4);
    return u;
}

inline float u2f(uint32_t u)
{
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

inline int model_bits(void *ctx)
{
    return ctx ? *static_cast<const int *>(ctx) : 7;
}

}  // namespace

extern "C" {

const char *amsim_status_string(int status)
{
    switch (status) {
    case AMSIM_OK: return "ok";
    case AMSIM_ERR_INVALID_ARG: return "invalid argument";
    case AMSIM_ERR_UNSUPPORTED: return "unsupported (mantissa bits outside [1,11] or shape beyond limits)";
    case AMSIM_ERR_MODEL: return "model cannot be represented by a mantissa table";
    case AMSIM_ERR_WORKSPACE: return "workspace missing or too small";
    case AMSIM_ERR_HIP: return "HIP runtime error";
    case AMSIM_ERR_IO: return "table file error";
    case AMSIM_ERR_SCRATCH: return "call needs more than the fixed scratch buffer (AMSIM_NOALLOC_SCRATCH_BYTES)";
    default: return "unknown status";
    }
}

int amsim_version(void) { return 10000; }

// Mitchell's logarithmic multiplier in integer form: with both fractions truncated to M bits
// and read as integers fa, fb in units of 2^-M, log2|a| + log2|b| ~= (Ea + Eb) + (fa + fb) 2^-M;
// the antilog puts the fractional part back as the mantissa and an integer overflow of
// fa + fb becomes an exponent increment.
float amsim_model_mitchell(float a, float b, void *ctx)
{
    const int m = model_bits(ctx);
    const uint32_t ua = f2u(a), ub = f2u(b);
    const uint32_t one = 1u << m;
    uint32_t s = ((ua >> (23 - m)) & (one - 1)) + ((ub >> (23 - m)) & (one - 1));
    int32_t e = int32_t((ua >> 23) & 0xFF) + int32_t((ub >> 23) & 0xFF) - 127;
    if (s >= one) {
        s -= one;
        e += 1;
    }
    const uint32_t sign = (ua ^ ub) & 0x80000000u;
    if (e <= 0) return u2f(sign);
    if (e >= 255) return u2f(sign | 0x7F800000u);
    return u2f(sign | (uint32_t(e) << 23) | (s << (23 - m)));
}

// Exact multiplier of operands truncated to M mantissa bits: drop the low 23-M mantissa bits
// of each operand and multiply in FP32.  The product of two (M+1)-bit significands has at most
// 2M+2 <= 24 significant bits, so the FP32 multiply is exact for in-range results.
float amsim_model_exact_trunc(float a, float b, void *ctx)
{
    const int m = model_bits(ctx);
    const uint32_t mask = 0xFFFFFFFFu << (23 - m);
    return u2f(f2u(a) & mask) * u2f(f2u(b) & mask);
}

// One Algorithm 1 entry for mantissa fields k, j with the given sign bits and biased
// exponents.  Returns false if the model's result cannot be encoded.
static bool lut_entry(int m, amsim_model_fn model, void *ctx, uint32_t k, uint32_t j, uint32_t sa, uint32_t sb,
                      uint32_t ea, uint32_t eb, uint32_t *entry)
{
    const float A = u2f((sa << 31) | (ea << 23) | (k << (23 - m)));
    const float B = u2f((sb << 31) | (eb << 23) | (j << (23 - m)));
    const uint32_t uc = f2u(model(A, B, ctx));
    const uint32_t exp_c = (uc >> 23) & 0xFF;
    const uint32_t un_normalized_exp = ea + eb - 127;
    if (exp_c == 0xFF) return false;                        // Inf / NaN
    if (((uc >> 31) & 1u) != (sa ^ sb)) return false;       // sign must be the XOR
    uint32_t carry;
    if (exp_c == un_normalized_exp) carry = 0;
    else if (exp_c == un_normalized_exp + 1) carry = 1;
    else return false;                                       // borrow or a two-step carry
    *entry = (carry << 23) | (uc & 0x7FFFFFu);
    return true;
}

int lut_build(int m_bits, amsim_model_fn model, void *ctx, uint32_t *out, size_t out_len)
{
    if (m_bits < 1 || m_bits > 11) return AMSIM_ERR_UNSUPPORTED;
    if (!model || !out) return AMSIM_ERR_INVALID_ARG;
    const uint32_t n = 1u << m_bits;
    if (out_len < size_t(n) * n) return AMSIM_ERR_INVALID_ARG;

    // Algorithm 1 with positive operands and exponent fields N = K = 127.
    for (uint32_t k = 0; k < n; ++k)
        for (uint32_t j = 0; j < n; ++j)
            if (!lut_entry(m_bits, model, ctx, k, j, 0, 0, 127, 127, &out[size_t(k) * n + j]))
                return AMSIM_ERR_MODEL;

    // The table is only valid if the mantissa product does not depend on signs or exponents:
    // rebuild a deterministic sample of entries at other legal (N, K) and every sign pair.
    static const uint32_t exps[][2] = {{100, 150}, {150, 100}, {1, 200}, {200, 1}, {64, 64}, {190, 190}};
    const size_t total = size_t(n) * n;
    const size_t stride = total > 4096 ? 61 : 1;
    int variant = 0;
    for (size_t idx = 0; idx < total; idx += stride, ++variant) {
        const uint32_t k = uint32_t(idx / n), j = uint32_t(idx % n);
        const uint32_t *e = exps[variant % 6];
        const uint32_t sa = (variant >> 1) & 1u, sb = (variant >> 2) & 1u;
        uint32_t entry;
        if (!lut_entry(m_bits, model, ctx, k, j, sa, sb, e[0], e[1], &entry) || entry != out[idx])
            return AMSIM_ERR_MODEL;
    }
    return AMSIM_OK;
}

int lut_save(const char *path, int m_bits, const uint32_t *lut, size_t len)
{
    if (!path || !lut) return AMSIM_ERR_INVALID_ARG;
    if (m_bits < 1 || m_bits > 11) return AMSIM_ERR_UNSUPPORTED;
    const size_t entries = size_t(1) << (2 * m_bits);
    if (len < entries) return AMSIM_ERR_INVALID_ARG;
    FILE *f = std::fopen(path, "wb");
    if (!f) return AMSIM_ERR_IO;
    const uint32_t hdr[4] = {0x544C4D41u /* "AMLT" */, 1u, uint32_t(m_bits), 0u};
    bool ok = std::fwrite(hdr, 4, 4, f) == 4;
    // entries little-endian (host order on x86-64)
    ok = ok && std::fwrite(lut, 4, entries, f) == entries;
    ok = (std::fclose(f) == 0) && ok;
    return ok ? AMSIM_OK : AMSIM_ERR_IO;
}

int lut_load(const char *path, int *m_bits, uint32_t *out, size_t out_len)
{
    if (!path || !m_bits) return AMSIM_ERR_INVALID_ARG;
    FILE *f = std::fopen(path, "rb");
    if (!f) return AMSIM_ERR_IO;
    uint32_t hdr[4];
    if (std::fread(hdr, 4, 4, f) != 4 || hdr[0] != 0x544C4D41u || hdr[1] != 1u || hdr[2] < 1 || hdr[2] > 11) {
        std::fclose(f);
        return AMSIM_ERR_IO;
    }
    const int m = int(hdr[2]);
    const size_t entries = size_t(1) << (2 * m);
    int rc = AMSIM_OK;
    if (out) {
        if (out_len < entries) rc = AMSIM_ERR_INVALID_ARG;
        else if (std::fread(out, 4, entries, f) != entries) rc = AMSIM_ERR_IO;
    }
    std::fclose(f);
    if (rc == AMSIM_OK) *m_bits = m;
    return rc;
}

}  // extern "C"
