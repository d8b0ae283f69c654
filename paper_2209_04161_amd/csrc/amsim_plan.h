// amsim_plan.h -- host-side planning of the table kernels' launches: the tile chooser, the
// workspace layout, the convolution shape rules and limits, and the kernels' argument geometry
// (TabArgs without its pointers, and the grid).  Plain host C++ over the shared types, so that a
// host-only build checks the very code the library runs (the bounds harness under the address
// and undefined-behaviour sanitizers).
#pragma once

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <iterator>
#include <utility>

#include "amsim.h"
#include "amsim_tab.h"

namespace amsim_detail __attribute__((visibility("hidden"))) {

// Words of the LDS tile through which the NHCW decode moves one padded image row's channels:
// cc * (w | 1) <= kNhcwTile (the convolution limits keep w and OW below half of it).
constexpr int kNhcwTile = 8192;

constexpr size_t kAlign = 256;

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
inline int64_t ceil_div(int64_t x, int64_t m) { return (x + m - 1) / m; }

// log2 of the table row length: rows are padded to 128 entries for M <= 7.
inline int row_log(int m_bits) { return m_bits > 7 ? m_bits : 7; }

// Calls of fewer products than kSelfMacs on rows of 128 entries are "small": they run the
// table-kernel variant that decides its path itself (one launch fewer), and they are planned as
// launches whose slabs wait on their own fetches -- too few workgroups to hide the staging's
// dependent loads, ~2.9 us a slab measured on MI355X (LeNet-5 layers, 3 to 60 workgroups)
// against ~0.7 us when rounds of workgroups overlap -- so they split their reductions down to
// single chunks.
// (products as a double: m * n * k of the largest shapes overflows 64 bits)
constexpr double kSelfMacs = double(int64_t(1) << 27);
inline bool small_call(double macs, int rl) { return rl == 7 && macs < kSelfMacs; }

// Cost per product used to choose among the candidate tiles (kTabCands and the wide-row lists):
// the inner loop (~1.2 VALU ops on the bf16 pair path, which 8-column tiles with all waves on
// rows take for 1-byte tables; 3 on the exact path), per-step overhead (~2.5 per row, ~4 per
// lane), and the table staging, which is per workgroup and slab, so its share per product falls
// with the workgroup's rows (64 * TM * WR) and grows with the row length (weight fitted on
// MI355X: a 64 x 32 backward-weight tile ran 2.4x slower than a 256 x 8 one, a 768-row GEMM tile
// 15% slower than a 1024-row one).
//
// Tile and reduction split for `rows` x `cols` outputs (times `phases` independent grids) over q
// reduction chunks of 8 steps.  The products a tile computes (rows padded to whole waves) times
// an issue-cost estimate per product, spread over the workgroups; the workgroups per CU that LDS
// and registers allow (four waves per SIMD) give the slots of one round, and a partly empty last
// round costs a whole one.  Tiles whose workgroups have few waves with rows in them (a 3 x 64-row
// wave tile over 147 rows) leave the SIMDs idle, which scales their issue rate down (measured on
// MI355X: the ResNet-50 stem's backward-weight 6%, the LeNet-5 stack 11% and an M = 11 1024^3
// GEMM 17% faster than without the scaling).  Only a launch under one round is split (at least
// 4 chunks per split, 1 for a small call).
inline Tile choose_tab_tile(int64_t rows, int64_t cols, int64_t q, bool small, bool allow_split, int rl, int max_tm,
                            int64_t phases)
{
    const int64_t min_chunks = small ? 1 : 4;
    const double fetch_ns = small ? 2900.0 : 700.0;
    constexpr int kCUs = 256, kWavesPerCU = 16;
    constexpr size_t kLdsPerCU = 160 * 1024;
    Tile best{};
    double best_cost = 0.0;
    const TabCand *cands = rl == 7 ? kTabCands : (rl < 11 ? kWideCands : kWide11Cands);
    const size_t ncands = rl == 7 ? std::size(kTabCands) : (rl < 11 ? std::size(kWideCands) : std::size(kWide11Cands));
    for (size_t ci = 0; ci < ncands; ++ci) {
        const TabCand &c = cands[ci];
        if (c.tm > max_tm) continue;
        const int64_t wrows = int64_t(64) * c.tm;  // rows per wave
        const int64_t rtile = wrows * c.wr;
        const int64_t ctile = int64_t(c.tn) * (c.nw / c.wr);
        const int64_t col_tiles = ceil_div(cols, ctile);
        const int64_t base = ceil_div(rows, rtile) * col_tiles * phases;  // workgroups without splits
        // waves whose rows all lie past the end skip the work; the fullest workgroup's live rows
        // share its staging
        const int64_t live_rows = std::min(rtile, ceil_div(rows, wrows) * wrows);
        const int64_t wgs_per_cu =
            std::max<int64_t>(1, std::min<int64_t>(kWavesPerCU / c.nw, kLdsPerCU / tab_lds_bytes(c.tn, c.wr, c.nw, rl)));
        const double slots = double(kCUs * wgs_per_cu);
        // fewer than two waves with rows per SIMD cannot keep the vector ALU and LDS busy: the
        // issue rate scales down with the live waves per CU below 8
        const double live_waves = double(live_rows / wrows) * double(c.nw / c.wr) * double(wgs_per_cu);
        const double occ = std::min(1.0, live_waves / 8.0);

        const double work =
            double(ceil_div(rows, wrows) * wrows) * double(col_tiles * ctile) * double(phases) * double(q * 8);
        const bool pair = rl == 7 && dot_cols_ok(c.tn) && c.wr == c.nw;
        // staging bytes per product grow with the row length (2^rl entries; wide rows are priced
        // at 2-byte entries)
        const double per_product =
            (pair ? 1.2 : 3.0) + 2.5 / c.tn + 4.0 / (c.tm * c.tn) +
            512.0 * double(1 << (rl - 7)) / double(live_rows) * (pair ? 0.5 : (rl == 7 ? 1.0 : 2.0));
        const double outputs = double(rows) * double(cols) * double(phases);
        // split only a launch that cannot fill one round by itself
        const int64_t max_split = allow_split && double(base) < slots
                                      ? std::max<int64_t>(1, std::min<int64_t>(q / std::max<int64_t>(1, min_chunks), 4096))
                                      : 1;
        // steps per slab (the bf16 path's, else a 2-byte table's) and a slab's time for one wave:
        // the staging fetch (a dependent pair of loads, fetch_ns) plus its products at ~1.15 (bf16
        // path) or ~3.7 (exact path) VALU instructions each, 4 clocks per instruction at 2.4 GHz
        const double slab_steps = pair ? 2.0 * c.nw : double(tab_slab_steps(int(ctile), rl, 2));
        const double slab_ns = fetch_ns + double(c.tm * c.tn) * slab_steps * (pair ? 1.15 : 3.7) * 4.0 / 2.4;
        // In ns, per round of workgroups: a workgroup's products at its share of the chip
        // (~20 T products/s, 28 cost units per ps, over all slots), or the slabs it walks through
        // one after another, whichever is longer; splits add their partial sums' traffic, a
        // launch, and the reduction's dependent loads (up to 32 groups of 8 per output).
        auto cost_of = [&](int64_t s) {
            const int64_t cps = ceil_div(q, s);           // chunks per split
            const int64_t s_eff = ceil_div(q, cps);       // the splits that chunking leaves
            const double wgs = double(base * s_eff);
            const double rounds = std::ceil(wgs / slots);
            const double issue_ns = (work / wgs) * per_product * slots / 28000.0 / occ;
            const double latency_ns = std::ceil(double(cps) * 8.0 / slab_steps) * slab_ns;
            double cst = rounds * std::max(issue_ns, latency_ns);
            if (s_eff > 1)
                cst += outputs * double(s_eff) * 8.0 / 5000.0 + 5000.0 + std::ceil(double(s_eff) / 256.0) * 800.0;
            return std::make_pair(cst, s_eff);
        };
        // candidate splits: none, the most allowed, and those that fill k whole rounds of slots
        int64_t trial[18];
        int nt = 0;
        trial[nt++] = 1;
        trial[nt++] = max_split;
        for (int k = 1; k <= 8; ++k) {
            const int64_t s0 = int64_t(std::floor(k * slots / double(base)));
            if (s0 >= 2 && s0 <= max_split) trial[nt++] = s0;
            if (s0 + 1 >= 2 && s0 + 1 <= max_split) trial[nt++] = s0 + 1;
        }
        for (int ti = 0; ti < nt; ++ti) {
            const auto cs = cost_of(trial[ti]);
            if (best_cost == 0.0 || cs.first < best_cost * 0.999) {
                best_cost = cs.first;
                best.tm = c.tm;
                best.tn = c.tn;
                best.wr = c.wr;
                best.nw = c.nw;
                best.split = int(cs.second);
            }
        }
    }
    return best;
}

// Columns of a table-kernel workgroup.
inline int64_t tab_cols(const Tile &t) { return int64_t(t.tn) * (t.nw / t.wr); }

// Workspace layout shared by the size queries and the launches:
//   [transposed rows][bf16-path rows][hi/lo rows][flags][statistics][wide-table partials]
//   [first operand][second operand][partials]
struct Plan {
    Tile tile;
    int rl;  // log2 of the table row length
    size_t off_rows, off_dot_rows, off_hl_rows, off_eb, off_stats, off_wpart, off_a, off_b, off_part, total;
    int64_t a_ld, b_ld;   // GEMM: padded leading dims of the decoded operands; conv: b_ld only
    int64_t a_elems;      // conv: elements of the decoded first operand
    int splits;           // reduction splits
    int chunks_per_split;   // 8-step reduction chunks per split
    int64_t out_elems;      // elements of the result (partial sums hold splits of them)
    int Hp, Wp, OHp, OWp, pad_oh, pad_ow;
    bool unfold_w;          // forward / backward-data pass over x unfolded along w
    int csplit;             // forward / backward data: channel chunks per kernel position (TabArgs::csplit)
    size_t off_unf;         // backward data, unfolded: the unfolded input's gradient
    int chunk;              // steps per reduction chunk (TabArgs::chunk)
    int rec_c;              // forward / backward data: channels of the first operand's record rows
    size_t off_bflags;      // backward data: zero-tap flags per (stride phase, ci), then per (kw, ci)
};

// Split of a reduction of `taps` taps of `count` steps, in chunks of p.chunk steps (the table
// kernels count chunks per tap as ceil(count / chunk)), into the tile's number of splits.
inline void plan_tab_split(Plan &p, int64_t taps, int64_t count)
{
    const int64_t q = taps * ceil_div(count, p.chunk);
    p.chunks_per_split = int(std::max<int64_t>(1, ceil_div(q, p.tile.split)));
    p.splits = int(std::max<int64_t>(1, ceil_div(q, p.chunks_per_split)));
}

inline bool valid_m(int m_bits) { return m_bits >= 1 && m_bits <= 11; }

// Transposed rows (the widest entry width, plus the zero row for 128-entry rows), bf16-path rows,
// hi/lo rows (128-entry rows only), flags, decode statistics (two operands), the wide-table
// preparation's partial words.
constexpr size_t kDotRowsBytes = size_t(kZeroRow + 1) * kTabRowEntries;
constexpr size_t kHlRowsBytes = size_t(kZeroRow + 1) * kHlRowBytes;  // 2-byte tables, hi/lo path
constexpr size_t kStatsBytes = size_t(2) * kStatSlots * 4;
constexpr int kWidePartWords = 1024;

inline size_t rows_bytes(int rl) { return (size_t(1) << rl) * ((size_t(1) << rl) + (rl == 7 ? 1 : 0)) * 4; }

// Step-pair records of the GEMM's first operand per row.
inline int64_t gemm_record_pairs(int64_t k) { return (k + 1) / 2; }

inline size_t table_area(Plan &p, size_t o)
{
    p.off_rows = o;
    p.off_dot_rows = p.off_rows + align_up(rows_bytes(p.rl));
    p.off_hl_rows = p.off_dot_rows + align_up(kDotRowsBytes);
    p.off_eb = p.off_hl_rows + (p.rl == 7 ? align_up(kHlRowsBytes) : 0);
    p.off_stats = p.off_eb + kAlign;
    p.off_wpart = p.off_stats + align_up(kStatsBytes);
    return p.off_wpart + (p.rl == 7 ? 0 : align_up(size_t(kWidePartWords) * 4));
}

inline Plan plan_gemm(int64_t m, int64_t n, int64_t k, int m_bits)
{
    Plan p{};
    p.rl = row_log(m_bits);
    p.tile = choose_tab_tile(m, n, ceil_div(k, 8), small_call(double(m) * double(n) * double(k), p.rl), true, p.rl, 8,
                             1);
    p.a_ld = round_up(m, int64_t(64) * p.tile.wr * p.tile.tm);
    p.chunk = 8;
    p.b_ld = round_up(n, tab_cols(p.tile));
    plan_tab_split(p, 1, k);
    size_t o = table_area(p, 0);
    p.off_a = o;  // step-pair records
    o += align_up(size_t(gemm_record_pairs(k)) * p.a_ld * 12);
    p.off_b = o;
    o += align_up(size_t(k) * p.b_ld * 4);
    p.out_elems = m * n;
    p.off_part = o;
    if (p.splits > 1) o += align_up(size_t(p.splits) * m * n * 4);
    p.total = o;
    return p;
}

inline ConvShape shape_of(const amsim_conv2d *d)
{
    ConvShape s;
    s.n = d->n; s.h = d->h; s.w = d->w; s.ci = d->c_in; s.co = d->c_out; s.kh = d->kh; s.kw = d->kw;
    s.sh = d->stride_h; s.sw = d->stride_w; s.pt = d->pad_top; s.pl = d->pad_left;
    s.oh = (d->h + d->pad_top + d->pad_bottom - d->kh) / d->stride_h + 1;
    s.ow = (d->w + d->pad_left + d->pad_right - d->kw) / d->stride_w + 1;
    return s;
}

inline int check_conv(const amsim_conv2d *d, int pass)
{
    if (!d) return AMSIM_ERR_INVALID_ARG;
    if (d->n < 1 || d->h < 1 || d->w < 1 || d->c_in < 1 || d->c_out < 1 || d->kh < 1 || d->kw < 1 ||
        d->stride_h < 1 || d->stride_w < 1 || d->pad_top < 0 || d->pad_bottom < 0 || d->pad_left < 0 ||
        d->pad_right < 0)
        return AMSIM_ERR_INVALID_ARG;
    const int64_t hp = int64_t(d->h) + d->pad_top + d->pad_bottom, wp = int64_t(d->w) + d->pad_left + d->pad_right;
    if (hp < d->kh || wp < d->kw) return AMSIM_ERR_INVALID_ARG;
    const int64_t oh = (hp - d->kh) / d->stride_h + 1, ow = (wp - d->kw) / d->stride_w + 1;
    // every index, padded tensor and byte offset must stay below 2^31
    const int64_t lim = int64_t(1) << 29;
    const int64_t xp = int64_t(d->n) * hp * wp * d->c_in;
    const int64_t yp = int64_t(d->n) * (oh + 2 * d->kh + 2) * (ow + 2 * d->kw + 2) * d->c_out;
    const int64_t w = int64_t(d->kh) * d->kw * (d->c_in + 16) * (d->c_out + 16);
    const int64_t y = int64_t(d->n) * oh * ow * (d->c_out + 16);
    // the step-pair records of zero-padded x and dy (12 bytes per pixel and channel pair) stay
    // below 2^31 bytes: the table kernels address them with 32-bit byte offsets
    const int64_t xr = int64_t(d->n) * hp * wp * ((d->c_in + 1) / 2) * 12;
    const int64_t yr = int64_t(d->n) * (oh + 2 * d->kh + 2) * (ow + 2 * d->kw + 2) * ((d->c_out + 1) / 2) * 12;
    // backward weight: one record per element of the zero-bordered x
    const int64_t xe = int64_t(d->n) * hp * wp * d->c_in * 12;
    if (xr >= (lim << 2) || yr >= (lim << 2) || (pass == AMSIM_CONV_BWD_WEIGHT && xe >= (lim << 2)))
        return AMSIM_ERR_UNSUPPORTED;
    if (xp >= lim || yp >= lim || w >= lim || y >= lim || d->pad_top >= 65536 || d->pad_bottom >= 65536 ||
        d->pad_left >= 65536 || d->pad_right >= 65536 || d->kh >= 65536 || d->kw >= 65536 ||
        int64_t(d->stride_h) * d->stride_w > 32 || d->c_in > 65535 * 16 || d->c_out > 65535 * 16 ||
        d->w >= kNhcwTile / 2 || ow >= kNhcwTile / 2)
        return AMSIM_ERR_UNSUPPORTED;
    return AMSIM_OK;
}

// Zero padding of dy for the backward-data table kernel: every phase row (hq, wq) plus every
// valid tap offset (dh, dw) must land inside the padded tensor.
inline void bwd_data_dy_pads(const ConvShape &s, int &top, int &bottom, int &left, int &right)
{
    top = bottom = left = right = 0;
    for (int ph = 0; ph < s.sh && ph < s.h; ++ph) {
        const int hq_n = (s.h - ph + s.sh - 1) / s.sh;
        for (int kh = (ph + s.pt) % s.sh; kh < s.kh; kh += s.sh) {
            const int dh = (ph + s.pt - kh) / s.sh;
            top = std::max(top, -dh);
            bottom = std::max(bottom, hq_n - 1 + dh - (s.oh - 1));
        }
    }
    for (int pw = 0; pw < s.sw && pw < s.w; ++pw) {
        const int wq_n = (s.w - pw + s.sw - 1) / s.sw;
        for (int kw = (pw + s.pl) % s.sw; kw < s.kw; kw += s.sw) {
            const int dw = (pw + s.pl - kw) / s.sw;
            left = std::max(left, -dw);
            right = std::max(right, wq_n - 1 + dw - (s.ow - 1));
        }
    }
}

inline int64_t bwd_data_rows(const ConvShape &s)
{
    return int64_t(s.n) * ceil_div(s.h, s.sh) * ceil_div(s.w, s.sw);  // largest phase
}

// The forward pass unfolds x along w (decode_unfold_w_kernel) when its taps are shorter than
// a slab of the widest tiles (c < 16 steps per (kh, kw) tap), the kernel is wider than one
// column, a source row fits the decode's LDS tile and the unfolded records stay below 2^31 bytes.
inline bool fwd_unfolds(const ConvShape &s, int hp)
{
    if (s.ci >= 16 || s.kw < 2 || int64_t(s.w) * s.ci > kNhcwTile) return false;
    const int64_t bytes = int64_t(s.n) * hp * s.ow * ((int64_t(s.kw) * s.ci + 1) / 2) * 12;
    return bytes < (int64_t(1) << 31);
}

// Channel chunks of the forward pass's taps (TabArgs::csplit): the taps run chunk-major, so that
// kernel positions one after another read the same chunk's input records.  With all channels in
// one tap, the records the rows in flight read per tap are the whole input (ResNet 3x3 64->64 at
// 32x32, batch 128: 57 MB, against 8 x 4 MB of L2), and each tap re-reads them from beyond L2.  Up
// to 4 chunks of a multiple of 16 channels (whole slabs; 8-step reduction chunks stay whole, so
// splits are unchanged); measured 2-3% faster on 3x3 layers.  Unfolded inputs have one tap.
inline int fwd_channel_chunks(const ConvShape &s, bool unfold)
{
    if (unfold) return 1;
    for (int c = 4; c > 1; c /= 2)
        if (s.ci % (16 * c) == 0) return c;
    return 1;
}

// Channel chunks of the backward-data pass's taps, over its output-gradient channels, for the same
// reason as the forward pass's: up to 8 chunks of a multiple of 16 channels (measured: ResNet 3x3
// 3.5% and ResNet-50 3x3 256->256 3% faster).
inline int bwd_data_channel_chunks(const ConvShape &s)
{
    for (int c = 8; c > 1; c /= 2)
        if (s.co % (16 * c) == 0) return c;
    return 1;
}

// Channels of the unfolded x, kw * c, rounded up to whole step pairs.
inline int unfolded_channels(const ConvShape &s) { return (s.kw * s.ci + 1) / 2 * 2; }

// The forward pass over the unfolded x as one tap: step kh * cu + j (cu = unfolded_channels) is
// channel j of image row oh * sh + kh, whose records follow those of row oh * sh + kh - 1 with the
// same stride (the rows' record blocks are cu / 2 records of ow apart), so the kernel sees a
// 1 x 1 "kernel" with kh * cu channels over a width-ow input; the table kernel's row records keep
// the real layout through TabArgs::rec_c = cu.  The output shape is unchanged.  A channel
// j >= kw * c of a row is padding: -0 in the records and +0 in the decoded weights, a -0 product
// that leaves every sum, and the sign of a zero sum, as it is.
inline ConvShape unfolded_shape(const ConvShape &s)
{
    ConvShape v = s;
    v.w = s.ow;
    v.ci = s.kh * unfolded_channels(s);
    v.kh = 1;
    v.kw = 1;
    v.sw = 1;
    v.pl = 0;
    return v;
}

// The backward-data pass unfolds along w in the same way when x has few channels (c < 8, which
// leaves most of an 8- or 4-column tile empty): it computes the gradient of the unfolded input,
// kw * c columns, as the backward-data pass of the virtual kh x 1 convolution below, then folds
// it back onto x (fold_w_kernel).  Not when the virtual pass or the unfolded gradient would
// exceed the limits.
inline amsim_conv2d unfolded_desc(const amsim_conv2d *d)
{
    amsim_conv2d v = *d;
    const int ow = (d->w + d->pad_left + d->pad_right - d->kw) / d->stride_w + 1;
    v.w = ow;
    v.c_in = d->kw * d->c_in;
    v.kw = 1;
    v.stride_w = 1;
    v.pad_left = v.pad_right = 0;
    return v;
}

inline bool bwd_data_unfolds(const amsim_conv2d *d)
{
    if (d->c_in >= 8 || d->kw < 2) return false;
    const amsim_conv2d v = unfolded_desc(d);
    return check_conv(&v, AMSIM_CONV_BWD_DATA) == AMSIM_OK && int64_t(v.n) * v.h * v.w * v.c_in < (int64_t(1) << 29);
}

inline Plan plan_conv(const amsim_conv2d *d, int pass, int m_bits)
{
    if (pass == AMSIM_CONV_BWD_DATA && bwd_data_unfolds(d)) {
        const amsim_conv2d v = unfolded_desc(d);
        Plan p = plan_conv(&v, pass, m_bits);  // the virtual pass (kw = 1: it does not unfold again)
        p.unfold_w = true;
        p.off_unf = align_up(p.total);  // the unfolded gradient [n][h][ow][kw * c]
        p.total = p.off_unf + align_up(size_t(v.n) * v.h * v.w * v.c_in * 4);
        return p;
    }
    const ConvShape s = shape_of(d);
    Plan p{};
    p.rl = row_log(m_bits);
    p.chunk = 8;
    size_t o = table_area(p, 0);
    const int64_t npix_in = int64_t(s.n) * s.h * s.w, npix_out = int64_t(s.n) * s.oh * s.ow;
    const bool small = small_call(double(npix_out) * s.co * s.kh * s.kw * s.ci, p.rl);
    p.Hp = d->h + d->pad_top + d->pad_bottom;
    p.Wp = d->w + d->pad_left + d->pad_right;
    if (pass == AMSIM_CONV_FWD) {
        p.unfold_w = fwd_unfolds(s, p.Hp);
        const ConvShape v = p.unfold_w ? unfolded_shape(s) : s;
        if (p.unfold_w) p.Wp = s.ow;  // the unfolded x has no w border
        const int64_t q = int64_t(v.kh) * v.kw * ceil_div(v.ci, 8);
        p.tile = choose_tab_tile(npix_out, s.co, q, small, true, p.rl, 8, 1);
        p.csplit = fwd_channel_chunks(s, p.unfold_w);
        plan_tab_split(p, int64_t(v.kh) * v.kw * p.csplit, v.ci / p.csplit);
        p.rec_c = p.unfold_w ? unfolded_channels(s) : s.ci;  // channels per record row block
        p.b_ld = round_up(s.co, tab_cols(p.tile));
        p.a_elems = int64_t(s.n) * p.Hp * p.Wp * ((p.rec_c + 1) / 2) * 3;  // zero-bordered x as step-pair records
        p.out_elems = npix_out * s.co;
        p.off_a = o;
        o += align_up(size_t(p.a_elems) * 4);
        p.off_b = o;  // decoded w [kh*kw*ci][COp] (unfolded: [kh][cu][COp])
        o += align_up(size_t(v.kh) * v.kw * v.ci * p.b_ld * 4);
    } else if (pass == AMSIM_CONV_BWD_DATA) {
        const int64_t rows = bwd_data_rows(s);
        const int64_t q = ceil_div(s.kh, s.sh) * ceil_div(s.kw, s.sw) * ceil_div(s.co, 8);  // largest phase
        p.tile = choose_tab_tile(rows, s.ci, q, small, true, p.rl, 4, int64_t(s.sh) * s.sw);  // 8-row tiles spill here
        int top, bottom, left, right;
        bwd_data_dy_pads(s, top, bottom, left, right);
        p.pad_oh = top;
        p.pad_ow = left;
        p.OHp = top + s.oh + bottom;
        p.OWp = left + s.ow + right;
        p.csplit = bwd_data_channel_chunks(s);
        plan_tab_split(p, ceil_div(s.kh, s.sh) * ceil_div(s.kw, s.sw) * p.csplit, s.co / p.csplit);
        p.rec_c = s.co;
        p.b_ld = round_up(s.ci, tab_cols(p.tile));
        p.a_elems = int64_t(s.n) * p.OHp * p.OWp * ((p.rec_c + 1) / 2) * 3;  // zero-padded dy as step-pair records
        p.out_elems = npix_in * s.ci;
        p.off_a = o;
        o += align_up(size_t(p.a_elems) * 4);
        p.off_b = o;  // decoded w^T [kh][kw][co][CIp]
        o += align_up(size_t(s.kh) * s.kw * s.co * p.b_ld * 4);
        p.off_bflags = o;
        o += align_up((size_t(s.sh) * s.sw * s.ci + size_t(s.kw) * s.ci) * 4);
    } else {
        const int64_t R = int64_t(s.kh) * s.kw * s.ci;
        const int64_t q = int64_t(s.n) * s.oh * ceil_div(s.ow, 8);
        p.tile = choose_tab_tile(R, s.co, q, small, true, p.rl, 8, 1);
        plan_tab_split(p, int64_t(s.n) * s.oh, s.ow);
        p.b_ld = round_up(s.co, tab_cols(p.tile));
        p.a_elems = int64_t(s.n) * p.Hp * p.Wp * s.ci * 3;
        p.out_elems = R * s.co;
        p.off_a = o;  // zero-bordered x as step-pair records, one per element
        o += align_up(size_t(p.a_elems) * 4);
        p.off_b = o;  // decoded dy [n*oh*ow][COp]
        o += align_up(size_t(npix_out) * p.b_ld * 4);
    }
    p.off_part = o;
    if (p.splits > 1) o += align_up(size_t(p.splits) * p.out_elems * 4);
    p.total = o;
    return p;
}

// The GEMM plans' limits (sizes below 2^31 given): the decoded first operand is addressed with
// 32-bit byte offsets, the second with 32-bit element offsets, partial sums with 32-bit indexes,
// and column blocks must fit a grid's y dimension.
inline bool gemm_fits(const Plan &p, int64_t m, int64_t n, int64_t k)
{
    const int64_t lim = int64_t(1) << 31;
    return k * p.a_ld < (int64_t(1) << 29) && k * p.b_ld < lim && int64_t(p.splits) * m * n < lim &&
           p.b_ld / tab_cols(p.tile) <= 65535;
}

// A 1 x 1 convolution with stride 1 and no padding: its im2col matrix is the input itself
// (Alg. 3), and there are no border or dilation zeros, so each pass is a plain GEMM over the
// pixels with the pass's first operand first -- forward y[pix][co] = x[pix][ci] . w[ci][co],
// backward data dx[pix][ci] = dy[pix][co] . w[ci][co]^T, backward weight
// dw[ci][co] = x[pix][ci]^T . dy[pix][co] -- and runs as one (the GEMM's planning, workspace
// and kernels).
inline bool conv_is_gemm(const amsim_conv2d *d)
{
    return d->kh == 1 && d->kw == 1 && d->stride_h == 1 && d->stride_w == 1 && d->pad_top == 0 &&
           d->pad_bottom == 0 && d->pad_left == 0 && d->pad_right == 0;
}

struct ConvGemm {
    int trans_a, trans_b;
    int64_t m, n, k, lda, ldb, ldc;
};

inline ConvGemm conv_gemm(const amsim_conv2d *d, int pass)
{
    const int64_t pix = int64_t(d->n) * d->h * d->w, ci = d->c_in, co = d->c_out;
    if (pass == AMSIM_CONV_FWD) return ConvGemm{0, 0, pix, co, ci, ci, co, co};
    if (pass == AMSIM_CONV_BWD_DATA) return ConvGemm{0, 1, pix, ci, co, co, co, ci};
    return ConvGemm{1, 0, ci, co, pix, ci, co, co};
}

// The vector GEMMs: m == 1 or n == 1 (one operand a vector: gemv_cols_kernel when the matrix's
// outputs are contiguous, gemv_rows_kernel when its steps are) and k == 1 (an outer product,
// outer_kernel).  k is split so that a launch holds about 2048 waves (8 per CU), each split at
// least 32 steps (one 256-step pass of a wave for the row kernel); the splits' partial sums
// [split][output] are the only workspace.
// Waves per workgroup: 16 when the workgroup stages the whole table in LDS (M <= 7, FP32
// operands: one 64 KiB copy then serves 16 waves), else 4.
constexpr int kGemvWavesLds = 16, kGemvWavesGlobal = 4;
inline int gemv_waves(bool lds) { return lds ? kGemvWavesLds : kGemvWavesGlobal; }
constexpr int kGemvCols = 4;   // outputs per lane, column kernel
constexpr int kGemvRows = 4;   // outputs per wave, row kernel

enum { VEC_NONE = 0, VEC_GEMV = 1, VEC_OUTER = 2 };

struct VecPlan {
    int kind;
    bool rows;       // the matrix's steps are contiguous (gemv_rows_kernel)
    int64_t nout;    // outputs (n when m == 1, else m)
    int64_t blocks;  // grid x
    int splits;      // grid y
    int64_t kchunk;  // steps per split
    size_t total;    // workspace bytes
};

// lds: the vector kernel stages the table in LDS (gemv_waves)
inline VecPlan plan_vec(int64_t m, int64_t n, int64_t k, int trans_a, int trans_b, bool lds)
{
    const int waves_wg = gemv_waves(lds);
    VecPlan v{};
    if (k == 1) {
        v.kind = VEC_OUTER;
        return v;
    }
    if (m != 1 && n != 1) return v;
    v.kind = VEC_GEMV;
    // m == 1: the matrix is B (steps contiguous when stored transposed); n == 1: A (steps
    // contiguous unless stored transposed)
    v.rows = m == 1 ? trans_b != 0 : trans_a == 0;
    v.nout = m == 1 ? n : m;
    int64_t waves, step_unit;
    if (v.rows) {
        v.blocks = ceil_div(v.nout, int64_t(waves_wg) * kGemvRows);
        waves = ceil_div(v.nout, int64_t(kGemvRows));
        step_unit = 256;
    } else {
        v.blocks = ceil_div(v.nout, int64_t(64) * kGemvCols);
        waves = v.blocks * waves_wg;
        step_unit = 32;
    }
    const int64_t want = std::max<int64_t>(1, ceil_div(2048, waves));
    const int64_t most = std::max<int64_t>(1, ceil_div(k, step_unit));
    v.kchunk = ceil_div(k, std::min(want, most));
    if (v.rows) v.kchunk = round_up(v.kchunk, 256);
    v.splits = int(ceil_div(k, v.kchunk));
    v.total = v.splits > 1 ? align_up(size_t(v.splits) * size_t(v.nout) * 4) : 0;
    return v;
}

// Workspace bytes of a GEMM call, enough for every option of it: the table's M or the native
// multiply's plan (M = 7), and the vector kernels with either workgroup size.
inline size_t gemm_workspace_bytes(int trans_a, int trans_b, int64_t m, int64_t n, int64_t k, int m_bits)
{
    if (m == 0 || n == 0 || k == 0) return 0;
    const VecPlan v0 = plan_vec(m, n, k, trans_a, trans_b, false), v1 = plan_vec(m, n, k, trans_a, trans_b, true);
    return v0.kind != VEC_NONE ? std::max(v0.total, v1.total)
                               : std::max(plan_gemm(m, n, k, m_bits).total, plan_gemm(m, n, k, 7).total);
}

// Whether a valid convolution pass runs as its GEMM (conv_is_gemm): when the GEMM's plans for the
// call's M and for the native multiply (M = 7) both fit the GEMM's limits; larger 1 x 1 passes keep
// the convolution path, whose limits are wider.
inline bool conv_runs_as_gemm(const amsim_conv2d *d, int pass, int m_bits)
{
    if (!conv_is_gemm(d)) return false;
    const ConvGemm g = conv_gemm(d, pass);
    if (plan_vec(g.m, g.n, g.k, g.trans_a, g.trans_b, false).kind != VEC_NONE) return true;
    return gemm_fits(plan_gemm(g.m, g.n, g.k, m_bits), g.m, g.n, g.k) && gemm_fits(plan_gemm(g.m, g.n, g.k, 7), g.m, g.n, g.k);
}

// Stride-1 backward data as a forward convolution.  With kh' = KH - 1 - kh and kw' = KW - 1 - kw,
// Algorithm 4's backward-data sum dx[n, h, w, ci] = sum over (kh, kw, co) of
// amul(dy[n, h + pt - kh, w + pl - kw, co], w[kh, kw, ci, co]), zeros of the padded dy included, is
// the forward pass over dy padded by (KH-1-pt, KH-1-pb, KW-1-pl, KW-1-pr) with the weights
// w'[kh'][kw'][co][ci] = w[KH-1-kh'][KW-1-kw'][ci][co]: the same products, dy first.  Taken where
// every pad is at most the kernel extent minus one and the forward pass keeps dy's channels whole
// (c_out >= 16, no unfolding): the forward kernel runs such shapes faster than the phase-decomposed
// backward-data kernel (ResNet 3x3 64->64: 0.255 against 0.274 ms on MI355X).
inline amsim_conv2d bwd_data_fwd_desc(const amsim_conv2d *d)
{
    amsim_conv2d f = *d;
    f.h = d->h + d->pad_top + d->pad_bottom - d->kh + 1;  // dy's height and width (stride 1)
    f.w = d->w + d->pad_left + d->pad_right - d->kw + 1;
    f.c_in = d->c_out;
    f.c_out = d->c_in;
    f.pad_top = d->kh - 1 - d->pad_top;
    f.pad_bottom = d->kh - 1 - d->pad_bottom;
    f.pad_left = d->kw - 1 - d->pad_left;
    f.pad_right = d->kw - 1 - d->pad_right;
    return f;
}

inline bool bwd_data_runs_as_fwd(const amsim_conv2d *d)
{
    if (d->stride_h != 1 || d->stride_w != 1 || d->c_out < 16 || conv_is_gemm(d)) return false;
    if (d->pad_top > d->kh - 1 || d->pad_bottom > d->kh - 1 || d->pad_left > d->kw - 1 || d->pad_right > d->kw - 1)
        return false;
    const amsim_conv2d f = bwd_data_fwd_desc(d);
    return check_conv(&f, AMSIM_CONV_FWD) == AMSIM_OK;
}

// ------------------------------------------------------------------ kernel geometry ------
// The table kernels' arguments apart from the pointers the launch fills in, and their grid.

struct TabGrid {
    unsigned x, y, z;
};

inline TabArgs tab_geom(const Plan &p, int64_t a_elems, int R, int N)
{
    TabArgs a{};
    a.a_bytes = uint32_t(a_elems * 4);
    a.Np = int(p.b_ld);
    a.R = R;
    a.N = N;
    a.Hp = p.Hp;
    a.Wp = p.Wp;
    a.OHp = p.OHp;
    a.OWp = p.OWp;
    a.pad_oh = p.pad_oh;
    a.pad_ow = p.pad_ow;
    a.splits = p.splits;
    a.chunk = p.chunk;
    a.chunks_per_split = p.chunks_per_split;
    a.out_elems = p.out_elems;
    a.csplit = 1;
    a.rec_c = p.rec_c;
    a.vadd = 0u;
    a.su = 1.0f;
    a.sd = 1.0f;
    return a;
}

// GEMM: m x n result with leading dimension ldc, reduction k.
inline TabArgs gemm_geom(const Plan &p, int64_t m, int64_t n, int64_t k, int64_t ldc)
{
    TabArgs a = tab_geom(p, 0, int(m), int(n));
    a.a_bytes = uint32_t(gemm_record_pairs(k) * p.a_ld * 12);
    a.ldc = p.splits > 1 ? n : ldc;  // partial sums are dense
    a.Mp = int(p.a_ld);
    a.K = int(k);
    return a;
}

inline TabGrid gemm_grid(const Plan &p)
{
    const Tile &t = p.tile;
    return TabGrid{unsigned(p.a_ld / (int64_t(64) * t.wr * t.tm)), unsigned(p.b_ld / tab_cols(t)),
                   unsigned(p.splits)};
}

// Forward pass of the convolution s (the caller's shape; unfolded here when the plan says so).
inline TabArgs fwd_geom(const Plan &p, const ConvShape &s)
{
    TabArgs a = tab_geom(p, p.a_elems, int(int64_t(s.n) * s.oh * s.ow), s.co);
    a.s = p.unfold_w ? unfolded_shape(s) : s;
    a.csplit = p.csplit;
    return a;
}

inline TabGrid fwd_grid(const Plan &p, const ConvShape &s)
{
    const Tile &t = p.tile;
    return TabGrid{unsigned(ceil_div(int64_t(s.n) * s.oh * s.ow, int64_t(64) * t.wr * t.tm)),
                   unsigned(p.b_ld / tab_cols(t)), unsigned(p.splits)};
}

// Backward-data pass of the convolution s (the virtual unfolded one when the plan unfolds).
inline TabArgs bwd_data_geom(const Plan &p, const ConvShape &s)
{
    TabArgs a = tab_geom(p, p.a_elems, int(bwd_data_rows(s)), s.ci);
    a.s = s;
    a.csplit = p.csplit;
    return a;
}

inline TabGrid bwd_data_grid(const Plan &p, const ConvShape &s)
{
    const Tile &t = p.tile;
    return TabGrid{unsigned(ceil_div(bwd_data_rows(s), int64_t(64) * t.wr * t.tm)), unsigned(p.b_ld / tab_cols(t)),
                   unsigned(s.sh * s.sw * p.splits)};
}

inline TabArgs bwd_weight_geom(const Plan &p, const ConvShape &s)
{
    TabArgs a = tab_geom(p, p.a_elems, s.kh * s.kw * s.ci, s.co);
    a.s = s;
    return a;
}

inline TabGrid bwd_weight_grid(const Plan &p, const ConvShape &s)
{
    const Tile &t = p.tile;
    return TabGrid{unsigned(ceil_div(int64_t(s.kh) * s.kw * s.ci, int64_t(64) * t.wr * t.tm)),
                   unsigned(p.b_ld / tab_cols(t)), unsigned(p.splits)};
}

}  // namespace amsim_detail
