// Host-only bounds harness for the table kernels' planning and tap arithmetic (test
// infrastructure; built with the address and undefined-behaviour sanitizers by
// tests/test_plan_bounds.py, no GPU involved).
//
// For seeded random GEMM shapes and convolution descriptors within the library's limits
// (check_conv / gemm_fits), it plans every pass exactly as the library does (amsim_plan.h) and
// checks, with 64-bit arithmetic against the kernels' own 32-bit forms:
//   * the workspace layout: every region aligned, inside `total`, regions in order;
//   * the grid: tiles cover the rows and padded columns, y and z within the hardware limits,
//     every reduction split non-empty;
//   * every first-operand byte offset a tap can form (lane row's record offset + the tap's step
//     offset + one 12-byte record) inside a_bytes, for sampled rows, taps and steps including
//     the extremes, with no wrap of the 32-bit forms;
//   * second-operand element offsets inside the decoded operand, result offsets inside the
//     result (or the split partial sums).
// Signed overflow anywhere in that arithmetic is reported by the undefined-behaviour sanitizer.
// Usage: plan_bounds_harness <gemm cases> <conv cases> <seed>.  Prints "OK ..." and exits 0, or
// prints the first failing case and exits 1.
#include <cinttypes>
#include <cstdio>
#include <cstdlib>

#include "amsim_plan.h"

using namespace amsim_detail;

namespace {

struct Rng {
    uint64_t s;
    uint64_t next()
    {
        s ^= s << 13;
        s ^= s >> 7;
        s ^= s << 17;
        return s;
    }
    int64_t uniform(int64_t lo, int64_t hi) { return lo + int64_t(next() % uint64_t(hi - lo + 1)); }
    // log-uniform in [lo, hi]
    int64_t logu(int64_t lo, int64_t hi)
    {
        const double a = std::log(double(lo)), b = std::log(double(hi) + 1.0);
        const double u = double(next() >> 11) / double(uint64_t(1) << 53);
        int64_t v = int64_t(std::exp(a + (b - a) * u));
        return std::min(hi, std::max(lo, v));
    }
};

char g_case[512];
long g_checks = 0;
int64_t g_max_a_bytes = 0;     // largest first-operand buffer planned
int64_t g_max_offset = 0;      // largest record end formed (row base + step offset + 12)
long g_bwd_as_fwd = 0;         // backward-data passes checked on the forward route

[[noreturn]] void fail(const char *what, int64_t v1, int64_t v2)
{
    std::printf("FAIL %s: %" PRId64 " vs %" PRId64 " in %s\n", what, v1, v2, g_case);
    std::fflush(stdout);
    std::exit(1);
}

void expect(bool ok, const char *what, int64_t v1 = 0, int64_t v2 = 0)
{
    ++g_checks;
    if (!ok) fail(what, v1, v2);
}

void check_region(const char *what, size_t off, size_t bytes, size_t end)
{
    expect(off % kAlign == 0, what, int64_t(off), int64_t(kAlign));
    expect(off + bytes <= end, what, int64_t(off + bytes), int64_t(end));
}

void check_table_area(const Plan &p)
{
    check_region("rows", p.off_rows, rows_bytes(p.rl), p.off_dot_rows);
    check_region("dot rows", p.off_dot_rows, kDotRowsBytes, p.off_hl_rows);
    check_region("hl rows", p.off_hl_rows, p.rl == 7 ? kHlRowsBytes : 0, p.off_eb);
    check_region("flags", p.off_eb, 3 * sizeof(int), p.off_stats);
    check_region("stats", p.off_stats, kStatsBytes, p.off_wpart);
    check_region("wide partials", p.off_wpart, p.rl == 7 ? 0 : size_t(kWidePartWords) * 4, p.off_a);
}

// A few indexes of [0, n): the first and last ones and some random ones (all when n is small).
template <class F>
void sample(Rng &rng, int64_t n, int k, F f)
{
    if (n <= 0) return;
    if (n <= 2 * k) {
        for (int64_t i = 0; i < n; ++i) f(i);
        return;
    }
    for (int64_t i = 0; i < 2; ++i) f(i);
    for (int64_t i = n - 2; i < n; ++i) f(i);
    for (int i = 0; i < k; ++i) f(rng.uniform(0, n - 1));
}

// The tile's reduction splits cover its chunks, and (one tap count per launch) none is empty.
template <int OP>
void check_splits(const TabArgs &a)
{
    const int cpt = (tab_count<OP>(a) + a.chunk - 1) / a.chunk;
    const int64_t q = int64_t(tab_taps<OP>(a)) * cpt;
    if (q == 0) return;  // a backward-data phase without taps
    expect(int64_t(a.splits) * a.chunks_per_split >= q, "splits cover the chunks", int64_t(a.splits) * a.chunks_per_split, q);
    // (a backward-data phase with fewer taps than the largest one may leave splits empty: they
    // write -0 partial sums, which the reduction adds as nothing)
    if (OP != OP_BWD_DATA)
        expect(int64_t(a.splits - 1) * a.chunks_per_split < q, "no empty split", int64_t(a.splits - 1) * a.chunks_per_split,
               q);
}

// Offsets of one operation's taps for the tile z (and its phase), sampled rows / taps / steps.
//   b_rows: rows of the decoded second operand (leading dimension a.Np); out_limit: elements of
//   the result or of one split's partial sums.
template <int OP>
void check_taps(Rng &rng, TabArgs a, const TabGrid &g, int64_t b_rows, int64_t out_limit, int64_t ldc)
{
    const int64_t R = tab_rows<OP>(a);
    const int taps = tab_taps<OP>(a), count = tab_count<OP>(a);
    if (taps == 0 || R == 0) return;
    expect(count > 0, "steps per tap", count, 0);
    check_splits<OP>(a);
    const int64_t cols = int64_t(g.y) * int64_t(a.Np / g.y);
    expect(cols == a.Np, "column blocks cover the padded columns", cols, a.Np);
    expect(a.N <= a.Np, "result columns inside the padded columns", a.N, a.Np);
    sample(rng, R + 1, 6, [&](int64_t row64) {
        const int row = int(row64);
        int rec = 0;  // rows past R read record 0's run (their results are never stored)
        if (row < R) {
            rec = tab_row_rec<OP>(a, row);
            expect(rec >= 0, "record offset >= 0", rec, 0);
            // result offsets of the row's first and last columns
            const int64_t ob = tab_row_out<OP>(a, row);
            if (OP == OP_GEMM) expect(ob == int64_t(row) * ldc, "GEMM result row", ob, int64_t(row) * ldc);
            expect(ob >= 0 && ob + (a.N - 1) < out_limit, "result offset", ob + (a.N - 1), out_limit);
        }
        const uint32_t voff = uint32_t(rec) * kPairRecordBytes;  // the kernels' 32-bit form
        const int64_t voff64 = int64_t(rec) * kPairRecordBytes;
        expect(int64_t(voff) == voff64, "row offset fits 32 bits", voff64, int64_t(voff));
        sample(rng, taps, 3, [&](int64_t tap) {
            const TabTap tp = tab_tap_raw<OP>(a, int(tap));
            expect(tp.count == count, "tap step count", tp.count, count);
            sample(rng, count, 2, [&](int64_t j) {
                const int64_t so64 = (int64_t(tp.pbase) + (j >> 1) * int64_t(tp.ustride)) * kPairRecordBytes;
                const uint32_t so = a_step_offset<OP>(tp, int(j));
                expect(so64 >= 0 && int64_t(so) == so64, "step offset fits 32 bits", so64, int64_t(so));
                g_max_offset = std::max(g_max_offset, voff64 + so64 + int64_t(kPairRecordBytes));
                expect(voff64 + so64 + int64_t(kPairRecordBytes) <= int64_t(a.a_bytes), "record inside a_bytes",
                       voff64 + so64 + int64_t(kPairRecordBytes), int64_t(a.a_bytes));
                const int64_t brow = int64_t(tp.bbase) + j;
                expect(tp.bbase >= 0 && brow < b_rows, "second-operand row", brow, b_rows);
            });
        });
    });
}

template <int OP>
void check_all_tiles(Rng &rng, const TabArgs &a0, const TabGrid &g, int64_t b_rows, int64_t out_limit, int64_t ldc)
{
    g_max_a_bytes = std::max(g_max_a_bytes, int64_t(a0.a_bytes));
    expect(g.x >= 1 && g.y >= 1 && g.z >= 1, "grid non-empty", g.x, g.y);
    expect(g.y <= 65535 && g.z <= 65535, "grid y / z limits", g.y, g.z);
    const int phases = int(g.z) / a0.splits;
    expect(phases * a0.splits == int(g.z), "grid z = phases x splits", g.z, a0.splits);
    for (int ph = 0; ph < phases; ++ph) {
        TabArgs a = a0;
        a.tz = ph * a0.splits;
        sample(rng, a0.splits, 1, [&](int64_t sp) {
            a.tz = ph * a0.splits + int(sp);
            check_taps<OP>(rng, a, g, b_rows, out_limit, ldc);
        });
    }
}

void check_gemm(Rng &rng, int64_t m, int64_t n, int64_t k, int mb)
{
    std::snprintf(g_case, sizeof g_case, "gemm m=%" PRId64 " n=%" PRId64 " k=%" PRId64 " M=%d", m, n, k, mb);
    const Plan p = plan_gemm(m, n, k, mb);
    if (!gemm_fits(p, m, n, k)) return;
    check_table_area(p);
    const int64_t rec_bytes = gemm_record_pairs(k) * p.a_ld * 12;
    check_region("gemm A records", p.off_a, size_t(rec_bytes), p.off_b);
    check_region("gemm B", p.off_b, size_t(k * p.b_ld * 4), p.off_part);
    check_region("gemm partials", p.off_part, p.splits > 1 ? size_t(p.splits) * size_t(m * n) * 4 : 0, p.total);
    expect(p.total == p.off_part + (p.splits > 1 ? align_up(size_t(p.splits) * size_t(m * n) * 4) : 0), "total");
    const TabArgs a = gemm_geom(p, m, n, k, n);
    expect(int64_t(a.a_bytes) == rec_bytes, "a_bytes fits 32 bits", rec_bytes, a.a_bytes);
    const TabGrid g = gemm_grid(p);
    expect(int64_t(g.x) * 64 * p.tile.wr * p.tile.tm == p.a_ld, "row tiles", g.x, p.a_ld);
    expect(p.a_ld >= m && p.b_ld >= n, "padded dims", p.a_ld, p.b_ld);
    check_all_tiles<OP_GEMM>(rng, a, g, k, p.splits > 1 ? m * n : (m - 1) * n + n, n);
}

// The vector GEMMs (m == 1, n == 1, k == 1): split coverage, grid limits, partial sums inside the
// workspace, and the 16-byte loads' alignment assumption for the row kernel's passes.
void check_vec(int64_t m, int64_t n, int64_t k, int ta, int tb, bool lds)
{
    std::snprintf(g_case, sizeof g_case, "vector gemm m=%" PRId64 " n=%" PRId64 " k=%" PRId64 " ta=%d tb=%d lds=%d", m, n,
                  k, ta, tb, int(lds));
    const VecPlan v = plan_vec(m, n, k, ta, tb, lds);
    if (k == 1) {
        expect(v.kind == VEC_OUTER, "k == 1 is an outer product");
        return;
    }
    if (m != 1 && n != 1) {
        expect(v.kind == VEC_NONE, "not a vector shape");
        return;
    }
    expect(v.kind == VEC_GEMV, "vector shape");
    expect(v.nout == (m == 1 ? n : m), "outputs", v.nout, m == 1 ? n : m);
    expect(v.splits >= 1 && v.splits <= 65535, "grid y", v.splits, 65535);
    expect(v.kchunk >= 1 && int64_t(v.splits) * v.kchunk >= k, "splits cover k", int64_t(v.splits) * v.kchunk, k);
    expect(int64_t(v.splits - 1) * v.kchunk < k, "no empty split", int64_t(v.splits - 1) * v.kchunk, k);
    const int64_t per_block = v.rows ? int64_t(gemv_waves(lds)) * kGemvRows : int64_t(64) * kGemvCols;
    expect(v.blocks >= 1 && v.blocks * per_block >= v.nout && (v.blocks - 1) * per_block < v.nout, "blocks cover outputs",
           v.blocks, v.nout);
    expect(v.blocks < (int64_t(1) << 31), "grid x", v.blocks, 0);
    if (v.rows) expect(v.kchunk % 256 == 0, "row kernel passes stay 4-aligned", v.kchunk, 256);
    const size_t part = v.splits > 1 ? size_t(v.splits) * size_t(v.nout) * 4 : 0;
    expect(part <= v.total && v.total % kAlign == 0, "partial sums inside the workspace", int64_t(part), int64_t(v.total));
    expect(int64_t(v.splits) * v.nout < (int64_t(1) << 31), "reduction indexes", int64_t(v.splits) * v.nout, 0);
}

void check_conv_pass(Rng &rng, const amsim_conv2d &d, int pass, int mb)
{
    std::snprintf(g_case, sizeof g_case,
                  "conv pass=%d M=%d n=%d h=%d w=%d ci=%d co=%d kh=%d kw=%d s=%dx%d pads=%d,%d,%d,%d", pass, mb, d.n,
                  d.h, d.w, d.c_in, d.c_out, d.kh, d.kw, d.stride_h, d.stride_w, d.pad_top, d.pad_bottom, d.pad_left,
                  d.pad_right);
    if (check_conv(&d, pass) != AMSIM_OK) return;
    if (conv_runs_as_gemm(&d, pass, mb)) {  // a 1 x 1, stride-1, unpadded pass runs as its GEMM
        const ConvGemm g = conv_gemm(&d, pass);
        char conv_case[sizeof g_case];
        std::snprintf(conv_case, sizeof conv_case, "%s", g_case);
        expect(g.m * g.n == (pass == AMSIM_CONV_BWD_WEIGHT ? int64_t(d.c_in) * d.c_out
                                                             : int64_t(d.n) * d.h * d.w * (pass ? d.c_in : d.c_out)),
               "the GEMM covers the pass's result", g.m * g.n, 0);
        const bool vec = plan_vec(g.m, g.n, g.k, g.trans_a, g.trans_b, false).kind != VEC_NONE;
        if (vec)
            check_vec(g.m, g.n, g.k, g.trans_a, g.trans_b, mb <= 7);
        else
            check_gemm(rng, g.m, g.n, g.k, mb);
        std::snprintf(g_case, sizeof g_case, "%s", conv_case);
        return;
    }
    if (pass == AMSIM_CONV_BWD_DATA && bwd_data_runs_as_fwd(&d)) {  // stride 1: the forward pass over dy
        const amsim_conv2d f = bwd_data_fwd_desc(&d);
        const ConvShape sf = shape_of(&f);
        expect(sf.oh == d.h && sf.ow == d.w && f.c_out == d.c_in && f.n == d.n, "the forward pass yields dx's shape",
               int64_t(sf.oh) * sf.ow, int64_t(d.h) * d.w);
        expect(f.c_in == sf.ci && !fwd_unfolds(sf, f.h + f.pad_top + f.pad_bottom), "dy's channels stay whole",
               f.c_in, 0);
        // the flipped, transposed weight reads: batch b of kh * kw (from the last kernel position), row
        // r of c_out, column c of c_in, at (kh * kw - 1 - b) * ci * co + c * co + r of the caller's w
        const int64_t nw = int64_t(d.kh) * d.kw * d.c_in * d.c_out, kk = int64_t(d.kh) * d.kw;
        const int64_t base = (kk - 1) * d.c_in * d.c_out, sb = -int64_t(d.c_in) * d.c_out;
        const int64_t lo = base + (kk - 1) * sb;                                       // last batch, row 0, column 0
        const int64_t hi = base + (d.c_out - 1) + int64_t(d.c_in - 1) * d.c_out;       // batch 0, last row and column
        expect(lo == 0 && hi == nw - 1, "flipped weight reads inside w", hi, nw);
        ++g_bwd_as_fwd;
        char bd_case[sizeof g_case];
        std::snprintf(bd_case, sizeof bd_case, "%s", g_case);
        check_conv_pass(rng, f, AMSIM_CONV_FWD, mb);
        std::snprintf(g_case, sizeof g_case, "%s", bd_case);
        return;
    }
    const Plan p = plan_conv(&d, pass, mb);
    check_table_area(p);
    const ConvShape s0 = shape_of(&d);
    if (pass == AMSIM_CONV_FWD) {
        const ConvShape v = p.unfold_w ? unfolded_shape(s0) : s0;
        check_region("fwd x records", p.off_a, size_t(p.a_elems) * 4, p.off_b);
        const int64_t b_rows = int64_t(v.kh) * v.kw * v.ci;
        check_region("fwd w", p.off_b, size_t(b_rows * p.b_ld * 4), p.off_part);
        check_region("fwd partials", p.off_part, p.splits > 1 ? size_t(p.splits) * p.out_elems * 4 : 0, p.total);
        const TabArgs a = fwd_geom(p, s0);
        expect(int64_t(a.a_bytes) == p.a_elems * 4, "a_bytes fits 32 bits", p.a_elems * 4, a.a_bytes);
        expect(v.ci % p.csplit == 0, "channel chunks divide ci", v.ci, p.csplit);
        const TabGrid g = fwd_grid(p, s0);
        expect(int64_t(g.x) * 64 * p.tile.wr * p.tile.tm >= int64_t(s0.n) * s0.oh * s0.ow, "row tiles", g.x, 0);
        check_all_tiles<OP_FWD>(rng, a, g, b_rows, p.out_elems, 0);
    } else if (pass == AMSIM_CONV_BWD_DATA) {
        const ConvShape s = p.unfold_w ? shape_of(&(const amsim_conv2d &)unfolded_desc(&d)) : s0;
        check_region("bwd_data dy records", p.off_a, size_t(p.a_elems) * 4, p.off_b);
        const int64_t b_rows = int64_t(s.kh) * s.kw * s.co;
        check_region("bwd_data w", p.off_b, size_t(b_rows * p.b_ld * 4), p.off_bflags);
        check_region("bwd_data flags", p.off_bflags, (size_t(s.sh) * s.sw * s.ci + size_t(s.kw) * s.ci) * 4,
                     p.off_part);
        const size_t part_end = p.off_part + (p.splits > 1 ? align_up(size_t(p.splits) * p.out_elems * 4) : 0);
        if (p.unfold_w) {
            expect(part_end <= p.off_unf, "unfolded gradient after the virtual plan", int64_t(part_end), int64_t(p.off_unf));
            // the unfolded input's gradient of the caller's shape, and its zero-tap flags
            check_region("unfolded dx", p.off_unf, size_t(s.n) * s.h * s.w * s.ci * 4, p.total);
            // the fold's kw flags follow the virtual pass's phase flags in the same region
            expect(size_t(s.sh) * s.sw * s.ci + size_t(d.kw) * d.c_in <= size_t(s.sh) * s.sw * s.ci + size_t(s.kw) * s.ci ||
                       p.off_bflags + (size_t(s.sh) * s.sw * s.ci + size_t(d.kw) * d.c_in) * 4 <= p.off_part,
                   "fold flags inside the flag region");
        } else {
            expect(part_end == p.total, "total", int64_t(part_end), int64_t(p.total));
        }
        const TabArgs a = bwd_data_geom(p, s);
        expect(int64_t(a.a_bytes) == p.a_elems * 4, "a_bytes fits 32 bits", p.a_elems * 4, a.a_bytes);
        expect(s.co % p.csplit == 0, "channel chunks divide co", s.co, p.csplit);
        const TabGrid g = bwd_data_grid(p, s);
        check_all_tiles<OP_BWD_DATA>(rng, a, g, b_rows, p.out_elems, 0);
    } else {
        check_region("bwd_weight x records", p.off_a, size_t(p.a_elems) * 4, p.off_b);
        const int64_t b_rows = int64_t(s0.n) * s0.oh * s0.ow;
        check_region("bwd_weight dy", p.off_b, size_t(b_rows * p.b_ld * 4), p.off_part);
        check_region("bwd_weight partials", p.off_part, p.splits > 1 ? size_t(p.splits) * p.out_elems * 4 : 0, p.total);
        const TabArgs a = bwd_weight_geom(p, s0);
        expect(int64_t(a.a_bytes) == p.a_elems * 4, "a_bytes fits 32 bits", p.a_elems * 4, a.a_bytes);
        const TabGrid g = bwd_weight_grid(p, s0);
        check_all_tiles<OP_BWD_WEIGHT>(rng, a, g, b_rows, p.out_elems, 0);
    }
}

amsim_conv2d random_desc(Rng &rng)
{
    amsim_conv2d d{};
    const int big = rng.uniform(0, 9) == 0;  // one case in ten near the size limits
    d.n = int(rng.logu(1, big ? 512 : 64));
    d.h = int(rng.logu(1, big ? 1024 : 96));
    d.w = int(rng.logu(1, big ? 4095 : 96));
    d.c_in = int(rng.logu(1, big ? 4096 : 512));
    d.c_out = int(rng.logu(1, big ? 4096 : 512));
    d.kh = int(rng.uniform(0, 7) == 0 ? rng.uniform(1, d.h + 4) : rng.uniform(1, 7));
    d.kw = int(rng.uniform(0, 7) == 0 ? rng.uniform(1, d.w + 4) : rng.uniform(1, 7));
    do {
        d.stride_h = int(rng.uniform(1, 6));
        d.stride_w = int(rng.uniform(1, 6));
    } while (d.stride_h * d.stride_w > 32);
    d.pad_top = int(rng.uniform(0, d.kh));
    d.pad_bottom = int(rng.uniform(0, d.kh));
    d.pad_left = int(rng.uniform(0, d.kw));
    d.pad_right = int(rng.uniform(0, d.kw));
    if (rng.uniform(0, 7) == 0) {  // one in eight pointwise: 1 x 1, stride 1, no padding (the GEMM route)
        d.kh = d.kw = d.stride_h = d.stride_w = 1;
        d.pad_top = d.pad_bottom = d.pad_left = d.pad_right = 0;
    } else if (rng.uniform(0, 7) == 0) {  // stride 1, pads within the kernel (backward data as a forward pass)
        d.stride_h = d.stride_w = 1;
        d.pad_top = std::min(d.pad_top, d.kh - 1);
        d.pad_bottom = std::min(d.pad_bottom, d.kh - 1);
        d.pad_left = std::min(d.pad_left, d.kw - 1);
        d.pad_right = std::min(d.pad_right, d.kw - 1);
    }
    return d;
}

}  // namespace

int main(int argc, char **argv)
{
    const long n_gemm = argc > 1 ? std::atol(argv[1]) : 10000;
    const long n_conv = argc > 2 ? std::atol(argv[2]) : 10000;
    Rng rng{argc > 3 ? uint64_t(std::atoll(argv[3])) * 0x9E3779B97F4A7C15ull + 1 : 0x1234567ull};
    long gemm_done = 0, conv_done = 0, conv_tried = 0;
    const int mbs[] = {7, 7, 7, 1, 4, 8, 9, 10, 11};
    while (gemm_done < n_gemm) {
        const bool big = rng.uniform(0, 9) == 0;
        const int64_t m = rng.logu(1, big ? (int64_t(1) << 22) : 8192);
        const int64_t n = rng.logu(1, big ? (int64_t(1) << 22) : 8192);
        const int64_t k = rng.logu(1, big ? (int64_t(1) << 22) : 8192);
        check_gemm(rng, m, n, k, mbs[rng.uniform(0, 8)]);
        // the same sizes as vector shapes
        const int ta = int(rng.uniform(0, 1)), tb = int(rng.uniform(0, 1));
        const bool lds = rng.uniform(0, 1) != 0;
        check_vec(1, n, k, ta, tb, lds);
        check_vec(m, 1, k, ta, tb, lds);
        check_vec(m, n, 1, ta, tb, lds);
        ++gemm_done;
    }
    while (conv_done < n_conv) {
        const amsim_conv2d d = random_desc(rng);
        ++conv_tried;
        bool any = false;
        for (int pass = 0; pass < 3; ++pass) {
            if (check_conv(&d, pass) != AMSIM_OK) continue;
            any = true;
            check_conv_pass(rng, d, pass, mbs[rng.uniform(0, 8)]);
        }
        if (any) ++conv_done;
        if (conv_tried > 50 * n_conv + 1000) {
            std::printf("FAIL too few valid convolution descriptors (%ld of %ld)\n", conv_done, conv_tried);
            return 1;
        }
    }
    std::printf("OK gemm_cases=%ld conv_cases=%ld conv_descriptors_drawn=%ld checks=%ld max_a_bytes=%" PRId64
                " max_record_end=%" PRId64 " bwd_data_as_fwd=%ld\n",
                gemm_done, conv_done, conv_tried, g_checks, g_max_a_bytes, g_max_offset, g_bwd_as_fwd);
    return 0;
}
