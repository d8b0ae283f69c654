// amsim_tab.h -- the table kernels (Algorithms 2-4 on the vector ALU) as templates over the
// operation and the tile, the set of instantiated tiles, and the per-operation launch entry
// points that amsim_tab.hip instantiates (one translation unit per operation).
//
// Kernel shape: lanes of a wave own output rows (64*TM rows per wave), the wave's TN output
// columns are wave-uniform, waves of a workgroup lie along rows and/or columns.  Per slab of
// steps the workgroup stages into LDS, for each of its columns and steps, the table row that
// the column's second-operand mantissa selects (128 entries for M <= 7, 2^M for M = 8..11);
// lanes gather from it with their first-operand mantissas.  For 1-byte tables and operands
// whose exponents keep every product normal, the bf16 pair path folds the second operand into
// the staged entries and adds two steps' products with one dot instruction.  Products are
// never fed to MFMA: they are not IEEE.
#pragma once

#include <type_traits>

#include "amsim_common.h"

namespace amsim_detail __attribute__((visibility("hidden"))) {

// ------------------------------------------------------------------ per-column tables
// The exact path keeps, per step and output column j, the table row selected by that column's
// second-operand mantissa kb(k, j) -- LUT[. ][kb], indexed by the first operand's mantissa --
// at a fixed LDS address.  Lanes then gather with
//   ds_read  v, (lane's first-operand mantissa * entry bytes)  offset:(fixed row address)
// so no per-product address arithmetic is left: per product one LDS gather, one multiply
// (pa * pb) and one fma.  Rows are copied from a transposed copy of the table in global
// memory, slab by slab (KS steps), double-buffered with one barrier per slab.
//
// Rows are stored compressed when the table allows it without loss: 1 byte per entry when
// every entry's low 16 mantissa bits are zero (e.g. Mitchell at M <= 7), 2 bytes when the low 8
// are zero (e.g. the exact truncated product at M <= 7, Mitchell at M = 8..11), else the 4-byte
// rebiased float.  The entry width is decided on the device by the table-preparation kernels
// and read by the table kernel, which runs the matching specialisation.

// Which operation the table kernel evaluates.  Every one is a sum over "taps": runs of
// consecutive reduction steps j = 0 .. count-1 whose first operand sits in the step-pair record
//   A[lane row's record base + pbase + (j / 2) * ustride]
// and whose second-operand row is Bd[bbase + j].
//   GEMM         one tap of K steps: rows i, A = op(A) k-major, row base i
//   FWD          tap = (kh, kw): rows (n, oh, ow), A = zero-padded x stored [n][h][ci][w], j = ci
//   BWD_DATA     tap = valid (kh, kw) of the stride phase in tile z: rows (n, hq, wq),
//                A = zero-padded dy stored [n][h][co][w], j = co; weights read as [kh][kw][co][ci]
//   BWD_WEIGHT   tap = output row (n, oh): rows (kh, kw, ci), A = zero-padded x (NHWC), j = ow,
//                B = dy
// The channel-inside-row layouts put the lanes' consecutive output pixels on consecutive words,
// so each first-operand load of a wave touches a few cache lines instead of 64.
// The reduction is cut into chunks of 8 steps (a tap of `count` steps holds ceil(count / 8));
// split s (of tile z) sums chunks [s * chunks_per_split, (s + 1) * chunks_per_split) into its
// own partial result, laid out like the final one; a fixed-order pass adds the partials.
enum { OP_GEMM = 0, OP_FWD = 1, OP_BWD_DATA = 2, OP_BWD_WEIGHT = 3 };

struct TabArgs {
    const uint32_t *A;   // decoded first operand: words, or (pair records) 12-byte step-pair records
    uint32_t a_bytes;    // its size in bytes (buffer range: reads beyond return 0)
    const uint32_t *Bd;  // decoded second operand rows, leading dimension Np
    int Np;
    float *out;          // result, or split partial sums [z][R][N]
    int64_t ldc;         // GEMM result leading dimension
    const unsigned char *rows;      // transposed table rows (exact path)
    const unsigned char *dot_rows;  // the same 1-byte rows in bf16-path staging order
    const unsigned char *hl_rows;   // 2-byte tables: entries split into bf16 halves (hi/lo path)
    const int *eb;                  // [0] entry width, [1] 1 (2) when the bf16 (hi/lo) path may run,
                                    // [2] 1 when the exact path rounds each product before adding it,
                                    // [3] (rows of 256 entries or more) 1 when the table is sum-indexed
    const uint32_t *stats_a, *stats_b;  // kTabApproxSelf: the decode passes' exponent statistics
    int n_a, n_b;                       // (null: none), words of each operand, and whether the
    int narrow;                         // operands are cast to fewer exponent bits than FP32's
    uint32_t vadd;       // exact path, rounded form: table values scaled by 2^(vadd >> 23) ...
    float su, sd;        // ... and each product by su, then added times sd (1, 1, 1 for FP32 operands)
    int R, N;            // result rows and columns
    int splits;          // reduction splits: tile z = (phase *) splits + split
    int chunk;           // steps per reduction chunk (8)
    int chunks_per_split;  // reduction chunks per split
    int64_t out_elems;   // elements of one split's partial result (splits > 1)
    int Mp, K;           // GEMM
    ConvShape s;
    int Hp, Wp;          // zero-padded x (FWD, BWD_WEIGHT)
    int rec_c;           // FWD / BWD_DATA: channels of the record layout [n][hp][rec_c / 2][wp] of x / dy
                         // (s.ci / s.co, or the unfolded kw * ci rounded to even)
    int csplit;          // FWD / BWD_DATA: channel chunks; taps run chunk-major (csplit divides s.ci / s.co
                         // into multiples of 8)
    int OHp, OWp, pad_oh, pad_ow;  // zero-padded dy (BWD_DATA)
    int tx, ty, tz;      // this workgroup's tile (row block, column block, phase/split); set on entry
};

// Workgroups go to the 8 XCDs in turn (linear id mod 8), and each XCD has its own L2.  The table
// kernels give each XCD a contiguous range of tiles instead, in the order stride phase fastest
// (phases differ in work, so each XCD gets all of them), then column blocks, row blocks, splits --
// so that the workgroups an XCD runs together share first-operand rows and second-operand cache
// lines in its L2.  Grids whose size is not a multiple of 8 keep the hardware order.
__device__ __forceinline__ void tab_tile_id(int splits, int &tx, int &ty, int &tz)
{
    const uint32_t gx = gridDim.x, gy = gridDim.y, gz = gridDim.z, n = gx * gy * gz;
    const uint32_t id = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
    if (n % 8u != 0u) {
        tx = int(blockIdx.x);
        ty = int(blockIdx.y);
        tz = int(blockIdx.z);
        return;
    }
    const uint32_t lid = (id % 8u) * (n / 8u) + id / 8u;
    const uint32_t phases = gz / uint32_t(splits);
    const uint32_t ph = lid % phases, rest = lid / phases;
    ty = int(rest % gy);
    tx = int((rest / gy) % gx);
    tz = int(ph * uint32_t(splits) + rest / (gx * gy));
}

struct TabTap {
    int pbase;    // the tap's first record, relative to the lane row's record base
    int ustride;  // records between consecutive step pairs
    int bbase;    // the second operand's row of step 0
    int count;    // steps
};

// Second-operand word of reduction row j (its table row, or with the native multiply its value)
// for result column col.
__device__ __forceinline__ uint32_t Bd_word(const TabArgs &a, int j, int col)
{
    return a.Bd[int64_t(j) * a.Np + col];
}

// The first operand of every operation is decoded into one 12-byte record per lane row and step
// pair (j, j + 1), j even (backward weight: one record per pixel of the zero-bordered x and
// channel, pairing it with the pixel one stride to its right, so that every kernel column's steps
// pair up whatever its kw): j's 16-bit table-index field (an LDS byte offset on the bf16 path)
// as a word, the two mantissa-cleared operands as bf16 (pa(j) | pa(j+1) << 16), and j+1's index
// word (with the native multiply: the two raw operands in the first and last words).  The bf16
// path loads a record with one instruction and uses it as loaded: no masking of the indices, no
// pairing of the heads.  A single step is one 8-byte load at record offset 0 (j even) or 4
// (j odd) and one byte permute.
constexpr uint32_t kPairRecordBytes = 12;

// First-operand buffer and the lane rows' byte offsets in it.
template <int TM>
struct AView {
    __amdgpu_buffer_rsrc_t words;  // the pair records
    uint32_t aoff[TM];             // per lane row: byte offset of its record base
};

// Byte offset of the record holding step j, relative to the lane row's record base.
template <int OP>
__host__ __device__ __forceinline__ uint32_t a_step_offset(const TabTap &tp, int j)
{
    return uint32_t(tp.pbase + (j >> 1) * tp.ustride) * kPairRecordBytes;
}

// The first operand's word of step j for each lane row (head | index: j's index word with j's
// half of the head pair moved into the high half); so = a_step_offset of j (wave-uniform).
template <int OP, int TM>
__device__ __forceinline__ void load_a_words(uint32_t (&dst)[TM], const AView<TM> &av, uint32_t so, int j)
{
#pragma unroll
    for (int r = 0; r < TM; ++r) {
        // j even: (index, heads) -> index | pa(j) << 16; j odd: (heads, index) -> index | pa(j+1)'s half
        const u32x2 d = __builtin_amdgcn_raw_buffer_load_b64(av.words, av.aoff[r], so + (j & 1) * 4u, 0);
        dst[r] = __builtin_amdgcn_perm(d.y, d.x, (j & 1) ? 0x03020504u : 0x05040100u);
    }
}

// rec: the lane rows' record bases (tab_row_rec).
template <int OP, int TM>
__device__ __forceinline__ AView<TM> make_aview(const TabArgs &a, const int (&rec)[TM])
{
    AView<TM> av;
    av.words = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t *>(a.A), 0, int(a.a_bytes), 0x00020000);
#pragma unroll
    for (int r = 0; r < TM; ++r) av.aoff[r] = uint32_t(rec[r]) * kPairRecordBytes;
    return av;
}

// Rows of one stride phase of the backward-data pass.
__host__ __device__ __forceinline__ void phase_dims(const ConvShape &s, int ph, int pw, int &hq_n, int &wq_n)
{
    hq_n = ph < s.h ? (s.h - ph + s.sh - 1) / s.sh : 0;
    wq_n = pw < s.w ? (s.w - pw + s.sw - 1) / s.sw : 0;
}

// tile z = phase * splits + split (phase only for BWD_DATA, else 0)
__host__ __device__ __forceinline__ int tab_phase(const TabArgs &a) { return a.tz / a.splits; }
__host__ __device__ __forceinline__ int tab_split(const TabArgs &a) { return a.tz % a.splits; }

template <int OP>
__host__ __device__ __forceinline__ int tab_rows(const TabArgs &a)
{
    if constexpr (OP == OP_BWD_DATA) {
        int hq_n, wq_n;
        phase_dims(a.s, tab_phase(a) / a.s.sw, tab_phase(a) % a.s.sw, hq_n, wq_n);
        return a.s.n * hq_n * wq_n;
    } else {
        return a.R;
    }
}

// Lane row -> result element offset.
template <int OP>
__host__ __device__ __forceinline__ int64_t tab_row_out(const TabArgs &a, int row)
{
    const ConvShape &s = a.s;
    if constexpr (OP == OP_GEMM) {
        return int64_t(row) * a.ldc;
    } else if constexpr (OP == OP_BWD_DATA) {
        const int ph = tab_phase(a) / s.sw, pw = tab_phase(a) % s.sw;
        int hq_n, wq_n;
        phase_dims(s, ph, pw, hq_n, wq_n);
        const int wq = row % wq_n, hq = (row / wq_n) % hq_n, n = row / (wq_n * hq_n);
        return ((int64_t(n) * s.h + hq * s.sh + ph) * s.w + wq * s.sw + pw) * s.ci;
    } else {
        return int64_t(row) * s.co;  // FWD: (n, oh, ow) x co; BWD_WEIGHT: (kh, kw, ci) x co
    }
}

// Lane row -> its record base in the first operand's pair records.
template <int OP>
__host__ __device__ __forceinline__ int tab_row_rec(const TabArgs &a, int row)
{
    const ConvShape &s = a.s;
    if constexpr (OP == OP_GEMM) {
        return row;
    } else if constexpr (OP == OP_FWD) {
        const int ow = row % s.ow, oh = (row / s.ow) % s.oh, n = row / (s.ow * s.oh);
        return (n * a.Hp + oh * s.sh) * ((a.rec_c + 1) / 2) * a.Wp + ow * s.sw;  // records [n][hp][ci/2][wp]
    } else if constexpr (OP == OP_BWD_DATA) {
        const int ph = tab_phase(a) / s.sw, pw = tab_phase(a) % s.sw;
        int hq_n, wq_n;
        phase_dims(s, ph, pw, hq_n, wq_n);
        const int wq = row % wq_n, hq = (row / wq_n) % hq_n, n = row / (wq_n * hq_n);
        return (n * a.OHp + hq) * ((a.rec_c + 1) / 2) * a.OWp + wq;  // records [n][ohp][rec_c/2][owp]
    } else {
        const int ci = row % s.ci, kw = (row / s.ci) % s.kw, kh = row / (s.ci * s.kw);
        return (kh * a.Wp + kw) * s.ci + ci;  // records [n][hp][wp][ci], one per element
    }
}

// Taps of the reduction (BWD_DATA: of this workgroup's stride phase).
template <int OP>
__host__ __device__ __forceinline__ int tab_taps(const TabArgs &a)
{
    if constexpr (OP == OP_GEMM) {
        return 1;
    } else if constexpr (OP == OP_BWD_WEIGHT) {
        return a.s.n * a.s.oh;
    } else if constexpr (OP == OP_BWD_DATA) {
        const ConvShape &s = a.s;
        const int ph = tab_phase(a) / s.sw, pw = tab_phase(a) % s.sw;
        const int kh0 = (ph + s.pt) % s.sh, kw0 = (pw + s.pl) % s.sw;
        const int nvh = kh0 < s.kh ? (s.kh - kh0 + s.sh - 1) / s.sh : 0;
        const int nvw = kw0 < s.kw ? (s.kw - kw0 + s.sw - 1) / s.sw : 0;
        return nvh * nvw * a.csplit;
    } else {
        return a.s.kh * a.s.kw * a.csplit;
    }
}

// Steps per tap (the same for every tap of an operation).
template <int OP>
__host__ __device__ __forceinline__ int tab_count(const TabArgs &a)
{
    if constexpr (OP == OP_GEMM) return a.K;
    else if constexpr (OP == OP_FWD) return a.s.ci / a.csplit;
    else if constexpr (OP == OP_BWD_DATA) return a.s.co / a.csplit;
    else return a.s.ow;
}

// The tap's fields are wave-uniform (they depend on the workgroup and the tap only).
template <int OP>
__host__ __device__ __forceinline__ TabTap tab_tap_raw(const TabArgs &a, int tap)
{
    const ConvShape &s = a.s;
    TabTap t;
    if constexpr (OP == OP_GEMM) {
        t.count = a.K;
        t.ustride = a.Mp;
        t.bbase = 0;
        t.pbase = 0;
    } else if constexpr (OP == OP_FWD) {
        // chunk-major: every kernel position over one chunk of channels, then the next chunk, so
        // that the records one tap reads are read again by the next taps while still in L2
        const int kk = tap % (s.kh * s.kw), chunk = tap / (s.kh * s.kw);
        const int kh = kk / s.kw, kw = kk % s.kw, cnt = s.ci / a.csplit, c0 = chunk * cnt;
        t.count = cnt;
        t.ustride = a.Wp;
        t.bbase = kk * s.ci + c0;
        t.pbase = (kh * ((a.rec_c + 1) / 2) + c0 / 2) * a.Wp + kw;
    } else if constexpr (OP == OP_BWD_DATA) {
        const int ph = tab_phase(a) / s.sw, pw = tab_phase(a) % s.sw;
        const int kh0 = (ph + s.pt) % s.sh, kw0 = (pw + s.pl) % s.sw;
        const int nvh = (s.kh - kh0 + s.sh - 1) / s.sh, nvw = (s.kw - kw0 + s.sw - 1) / s.sw;
        const int kk = tap % (nvh * nvw), chunk = tap / (nvh * nvw);  // chunk-major, as FWD
        const int kh = kh0 + (kk / nvw) * s.sh, kw = kw0 + (kk % nvw) * s.sw;
        const int dh = (ph + s.pt - kh) / s.sh, dw = (pw + s.pl - kw) / s.sw;  // exact divisions
        const int cnt = s.co / a.csplit, c0 = chunk * cnt;
        t.count = cnt;
        t.ustride = a.OWp;
        t.bbase = (kh * s.kw + kw) * s.co + c0;
        // >= 0: the padding covers every dh, dw
        t.pbase = ((dh + a.pad_oh) * ((a.rec_c + 1) / 2) + c0 / 2) * a.OWp + dw + a.pad_ow;
    } else {
        // step j = ow reads x at column ow * sw + kw: the record of step pair (j, j + 1) is the one of
        // column j * sw + kw, 2 sw columns after the previous pair's
        const int n = tap / s.oh, oh = tap % s.oh;
        t.count = s.ow;
        t.ustride = 2 * s.sw * s.ci;
        t.bbase = tap * s.ow;
        t.pbase = (n * a.Hp + oh * s.sh) * a.Wp * s.ci;
    }
    return t;
}

template <int OP>
__device__ __forceinline__ TabTap tab_tap(const TabArgs &a, int tap)
{
    const TabTap t = tab_tap_raw<OP>(a, tap);
    return TabTap{__builtin_amdgcn_readfirstlane(t.pbase), __builtin_amdgcn_readfirstlane(t.ustride),
                  __builtin_amdgcn_readfirstlane(t.bbase), __builtin_amdgcn_readfirstlane(t.count)};
}

// The slab cursor is wave-uniform; saying so at the loop head keeps it, and the buffer loads'
// step offsets derived from it, in scalar registers (the compiler's uniformity analysis does not
// prove it through the backward-data phase math and would loop each load over the lanes).
__device__ __forceinline__ void uniform_cursor(TabTap &cur, int &tap, int &c0)
{
    cur = TabTap{__builtin_amdgcn_readfirstlane(cur.pbase), __builtin_amdgcn_readfirstlane(cur.ustride),
                 __builtin_amdgcn_readfirstlane(cur.bbase), __builtin_amdgcn_readfirstlane(cur.count)};
    tap = __builtin_amdgcn_readfirstlane(tap);
    c0 = __builtin_amdgcn_readfirstlane(c0);
}

// Steps per slab of the exact path, rows of 2^RL entries of EB bytes, TNW columns: 8 KiB slabs of
// 8 / EB steps for the 128-entry rows; wider rows (M = 8..11) take up to 32 KiB slabs of 1 to 8 steps
// (the step loop is unrolled, so it stays short).
constexpr int tab_slab_steps(int tnw, int rl, int eb)
{
    return rl == 7 ? 8 / eb
                   : (32768 / (tnw * (1 << rl) * eb) < 1 ? 1
                                                          : (32768 / (tnw * (1 << rl) * eb) > 8
                                                                 ? 8
                                                                 : 32768 / (tnw * (1 << rl) * eb)));
}

// Slab staging: each thread copies CPT 16-byte pieces of the rows selected by the second
// operand's mantissas (kb) for slots [0, nslots) of a slab, and that operand's head (pb).
// TNW = result columns of the workgroup.  Two parts, a slab apart: the second-operand words of
// the thread's pieces (tab_fetch_words), then the row pieces they select (tab_fetch_rows), so
// that a slab waits on one load latency rather than two dependent ones.
template <int TNW, int EB, int CPT, int NT, int RL>
__device__ __forceinline__ void tab_fetch_words(uint32_t (&bw)[CPT], const TabTap &tp, int c0,
                                                const uint32_t *__restrict__ Bd, int Np, int col0)
{
    constexpr int ROWB = (1 << RL) * EB;
    constexpr uint32_t kPad = RL == 7 ? kZeroRowWord : 0u;  // a padding step's second operand: +0
    constexpr int PIECES = ROWB / 16;
    constexpr int TOTAL = tab_slab_steps(TNW, RL, EB) * TNW * PIECES;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
        const int c = threadIdx.x + i * NT;
        if (CPT * NT > TOTAL && c >= TOTAL) break;  // the workgroup size does not divide the slab
        const int slot = c / (TNW * PIECES);
        const int t = (c / PIECES) % TNW;
        const int j = c0 + slot;
        bw[i] = j < tp.count ? Bd[int64_t(tp.bbase + j) * Np + col0 + t] : kPad;
    }
}

template <int TNW, int EB, int CPT, int NT, int RL>
__device__ __forceinline__ void tab_fetch_rows(u32x4 (&stage)[CPT], float (&stage_pb)[CPT], const uint32_t (&bw)[CPT],
                                               const unsigned char *__restrict__ rows)
{
    constexpr int ROWB = (1 << RL) * EB;
    constexpr int PIECES = ROWB / 16;
    constexpr int TOTAL = tab_slab_steps(TNW, RL, EB) * TNW * PIECES;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
        const int c = threadIdx.x + i * NT;
        if (CPT * NT > TOTAL && c >= TOTAL) break;
        const int piece = c % PIECES;
        stage_pb[i] = head_value(bw[i]);
        stage[i] = *reinterpret_cast<const u32x4 *>(rows + (bw[i] & kIdxMask) * EB + piece * 16);  // idx = kb << RL
    }
}

template <int TNW, int EB, int CPT, int NT, int RL>
__device__ __forceinline__ void tab_commit(const u32x4 (&stage)[CPT], const float (&stage_pb)[CPT],
                                           unsigned char *smem, float *pbs, int buf)
{
    constexpr int ROWB = (1 << RL) * EB;
    constexpr int KS = tab_slab_steps(TNW, RL, EB);
    constexpr int SLAB = KS * TNW * ROWB;
    constexpr int PIECES = ROWB / 16;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
        const int c = threadIdx.x + i * NT;
        if (CPT * NT > SLAB / 16 && c >= SLAB / 16) break;
        *reinterpret_cast<u32x4 *>(smem + buf * SLAB + c * 16) = stage[i];
        if (c % PIECES == 0) pbs[buf * KS * TNW + c / PIECES] = stage_pb[i];
    }
}

// Workgroup: NW waves as a WR x (NW/WR) grid -- WR row blocks of 64*TM rows, NW/WR column groups
// of TN columns.  All waves share the LDS tables of the workgroup's TN * NW/WR columns.
// Products: fma(v, pa * pb, acc) (ROUNDED = false), or t = v' * (pa * pb) rounded on its own, then
// acc = fma(t * su, sd, acc) (ROUNDED = true).  With FP32 operands v' = v and su = sd = 1: the
// product is Inf when the carry lifts its exponent to 255, whatever the sum.  With a narrower
// exponent (the decode lowered the heads' exponents by delta, 2 delta = 127 - beta) v' = v * 2^(2
// delta) makes t the format's product exactly, t * su = t * 2^(2 delta) overflows exactly when that
// product reaches 2^(beta + 1) (Algorithm 2's overflow rule in the format's constants), and sd =
// 2^(-2 delta) brings it back unchanged (Inf stays Inf).
template <int OP, int TM, int TN, int WR, int EB, int NW, int RL, bool ROUNDED>
__device__ __forceinline__ void tab_body(const TabArgs &a)
{
    constexpr int NT = 64 * NW;
    constexpr int WC = NW / WR;
    constexpr int TNW = TN * WC;                // result columns of the workgroup
    constexpr int ROWB = (1 << RL) * EB;        // a table row: 2^RL entries
    constexpr int KS = tab_slab_steps(TNW, RL, EB);
    constexpr int SLAB = KS * TNW * ROWB;
    constexpr int CPT = (SLAB / 16 + NT - 1) / NT;  // pieces per thread per slab (the last round partial)
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    float *pbs = reinterpret_cast<float *>(smem + 2 * SLAB);  // [2][KS][TNW] second-operand heads

    const int R = tab_rows<OP>(a);
    if (a.tx * 64 * TM * WR >= R) return;  // uniform over the workgroup
    const int lane = threadIdx.x & 63;
    const int wave = wave_id();
    const int rg = wave % WR, cg = wave / WR;
    const int row0 = a.tx * (64 * TM * WR) + rg * (64 * TM) + lane;
    const bool live = row0 - lane < R;  // wave-uniform: a wave past the end only stages
    const int colw = a.ty * TNW;  // first column of the workgroup
    const int col0 = colw + cg * TN;    // first column of this wave
    // First-operand reads are raw buffer loads: voffset = the lane row's byte offset (range-checked,
    // reads past the buffer return 0), soffset = the wave-uniform step offset, which every tap keeps
    // non-negative and inside the tensor, since the hardware does not range-check it.
    int abase[TM];  // each lane row's record base
#pragma unroll
    for (int r = 0; r < TM; ++r) {
        const int row = row0 + 64 * r;
        abase[r] = row < R ? tab_row_rec<OP>(a, row) : 0;  // rows past the end read record 0's run
    }
    const AView<TM> av = make_aview<OP, TM>(a, abase);
    // this split's chunks, as positions p = tap * (8 * chunks per tap) + step
    const int count = tab_count<OP>(a);
    const int ch = a.chunk;  // steps per reduction chunk
    const int cpt = (count + ch - 1) / ch;  // chunks per tap
    const int q_total = tab_taps<OP>(a) * cpt;
    const int q0 = tab_split(a) * a.chunks_per_split;
    const int p_end = min(q_total, q0 + a.chunks_per_split) * ch;

    // Second-operand words a slab ahead of their rows (tab_fetch_words), where the table fits an
    // XCD's L2 (rows of up to 1024 entries): measured on MI355X, the M = 10 GEMM 2048^3 14% and the
    // 2-byte ResNet 3x3 backward-weight pass 3% faster.  The M = 11 table (8 MiB at 2 bytes) is
    // read from beyond L2: with the words ahead its 4096^3 GEMM was 3% slower (19.15 against
    // 18.6 ms); it fetches both in the same slab, and with the slab cursors kept a slab ahead as
    // here it went to 17.85 ms.
    constexpr bool WORDS_AHEAD = RL <= 10;
    u32x4 stage[CPT];
    float stage_pb[CPT];
    uint32_t sbw[CPT];  // second-operand words of the next slab's pieces
    float acc[TM][TN];
    init_acc(acc);
    uint32_t acur[TM];
    // The slab after (t, tp_, c): its tap, cursor and whether it is in this split's range.
    auto advance = [&](const TabTap &t, int tp_, int c, TabTap &o, int &otap, int &oc, bool &ok)
                       __attribute__((always_inline)) {
        o = t;
        otap = tp_;
        oc = c + KS;
        if (oc >= count) {
            otap = tp_ + 1;
            oc = 0;
        }
        ok = otap * cpt * ch + oc < p_end;
        if (ok && otap != tp_) o = tab_tap<OP>(a, otap);
    };
    TabTap cur{0, 0, 0, 0};
    int tap = q0 / max(cpt, 1);
    int c0 = (q0 - tap * cpt) * ch;
    bool have = q0 * ch < p_end;
    TabTap nxt{0, 0, 0, 0};
    int ntap = 0, nc0 = 0;
    bool has_next = false;
    if (have) {
        cur = tab_tap<OP>(a, tap);
        tab_fetch_words<TNW, EB, CPT, NT, RL>(sbw, cur, c0, a.Bd, a.Np, colw);
        tab_fetch_rows<TNW, EB, CPT, NT, RL>(stage, stage_pb, sbw, a.rows);
        tab_commit<TNW, EB, CPT, NT, RL>(stage, stage_pb, smem, pbs, 0);
        load_a_words<OP, TM>(acur, av, __builtin_amdgcn_readfirstlane(a_step_offset<OP>(cur, c0)), c0);
        advance(cur, tap, c0, nxt, ntap, nc0, has_next);
        if (WORDS_AHEAD && has_next) tab_fetch_words<TNW, EB, CPT, NT, RL>(sbw, nxt, nc0, a.Bd, a.Np, colw);
    }
    __syncthreads();
    int buf = 0;
    while (have) {
        uniform_cursor(cur, tap, c0);
        uniform_cursor(nxt, ntap, nc0);
        // the slab after the next one, whose words are loaded while this one is computed (the
        // next slab's rows are fetched with the words loaded during the previous slab)
        TabTap nxt2 = nxt;
        int ntap2 = ntap, nc02 = nc0;
        bool has_next2 = false;
        if (has_next) advance(nxt, ntap, nc0, nxt2, ntap2, nc02, has_next2);
        if (has_next) {
            if constexpr (!WORDS_AHEAD) tab_fetch_words<TNW, EB, CPT, NT, RL>(sbw, nxt, nc0, a.Bd, a.Np, colw);
            tab_fetch_rows<TNW, EB, CPT, NT, RL>(stage, stage_pb, sbw, a.rows);
        }
        if (WORDS_AHEAD && has_next2) tab_fetch_words<TNW, EB, CPT, NT, RL>(sbw, nxt2, nc02, a.Bd, a.Np, colw);
        const unsigned char *tb = smem + buf * SLAB + cg * TN * ROWB;
        const float *pb_s = pbs + buf * KS * TNW + cg * TN;
        // the slab ends at the tap's end or, 8-step chunks being the unit of splits, at the split's
        const int nslots = live ? min(min(KS, cur.count - c0), p_end - (tap * cpt * ch + c0)) : 0;
        __builtin_amdgcn_s_setprio(3);  // computing waves first, as on the bf16 path
#pragma unroll
        for (int slot = 0; slot < KS; ++slot) {
            if (slot >= nslots) break;
            // next step's first-operand words: this slab's next slot or the next slab's first
            uint32_t anext[TM];
            const bool in_slab = slot + 1 < nslots;
            const uint32_t unext = __builtin_amdgcn_readfirstlane(in_slab ? a_step_offset<OP>(cur, c0 + slot + 1)
                                                                          : a_step_offset<OP>(nxt, nc0));
            const int jnext = __builtin_amdgcn_readfirstlane(in_slab ? c0 + slot + 1 : nc0);
            if (in_slab || has_next) {
                load_a_words<OP, TM>(anext, av, unext, jnext);
            } else {
#pragma unroll
                for (int r = 0; r < TM; ++r) anext[r] = 0u;
            }
            const unsigned char *vaddr[TM];
            float pa[TM];
#pragma unroll
            for (int r = 0; r < TM; ++r) {
                vaddr[r] = tb + __builtin_amdgcn_ubfe(acur[r], 4, RL) * EB;  // idx = ka << 4
                pa[r] = head_value(acur[r]);
            }
#pragma unroll
            for (int t = 0; t < TN; ++t) {
                const float pb = pb_s[slot * TNW + t];
#pragma unroll
                for (int r = 0; r < TM; ++r) {
                    if constexpr (ROUNDED) {
                        const float v = tab_value_scaled<EB>(vaddr[r] + (slot * TNW + t) * ROWB, a.vadd);
                        const float c = v * (pa[r] * pb);
                        acc[r][t] = __builtin_fmaf(c * a.su, a.sd, acc[r][t]);
                    } else {
                        const float v = tab_value<EB>(vaddr[r] + (slot * TNW + t) * ROWB);
                        acc[r][t] = __builtin_fmaf(v, pa[r] * pb, acc[r][t]);
                    }
                }
            }
#pragma unroll
            for (int r = 0; r < TM; ++r) acur[r] = anext[r];
        }
        __builtin_amdgcn_s_setprio(0);
        if (has_next) tab_commit<TNW, EB, CPT, NT, RL>(stage, stage_pb, smem, pbs, buf ^ 1);
        __syncthreads();
        cur = nxt;
        tap = ntap;
        c0 = nc0;
        buf ^= 1;
        have = has_next;
        nxt = nxt2;
        ntap = ntap2;
        nc0 = nc02;
        has_next = has_next2;
    }

    // results (with splits, each split's partial result is laid out like the final one)
    float *out = a.out + int64_t(tab_split(a)) * a.out_elems;
#pragma unroll
    for (int r = 0; r < TM; ++r) {
        const int row = row0 + 64 * r;
        if (row >= R) continue;
        float *dst = out + tab_row_out<OP>(a, row);  // recomputed rather than kept in registers
#pragma unroll
        for (int t = 0; t < TN; ++t) {
            const int col = col0 + t;
            if (col < a.N) dst[col] = acc[r][t];
        }
    }
}

// ------------------------------------------------------- sum-indexed wide tables
// For many approximate multipliers -- Mitchell's at every M among them -- an entry depends on the
// two mantissa indices only through their sum: T[ka][kb] = g(ka + kb), with
// g(s) = T[min(s, 2^M - 1)][s - min(s, 2^M - 1)].  The table preparation checks every entry for it
// (flags[3]).  Such a table is served from g alone: 2^(M+1) factors v (as floats, pre-scaled by vadd
// in the rounded form) copied into LDS once per workgroup, where the exact path stages a 2^M-entry
// row per column and step (4 KiB per column and step at M = 11, read from beyond L2).  Per product:
// one address add (the lane row's ka, the column's kb, both as byte offsets), one LDS gather, and the
// exact path's arithmetic.  The slabs hold only the second operand's (kb offset, head) pairs.
constexpr int kSumSlabSteps = 16;

constexpr size_t tab_sum_lds_bytes(int tnw, int rl)
{
    return (size_t(2) << rl) * 4 + size_t(2) * kSumSlabSteps * tnw * 8;
}

template <int OP, int TM, int TN, int WR, int NW, int RL, bool ROUNDED>
__device__ __forceinline__ void tab_body_sum(const TabArgs &a, int eb)
{
    constexpr int NT = 64 * NW;
    constexpr int WC = NW / WR;
    constexpr int TNW = TN * WC;            // result columns of the workgroup
    constexpr int KS = kSumSlabSteps;
    constexpr int GN = 2 << RL;             // g's entries (the last one unused)
    constexpr int WSLAB = KS * TNW;         // (kb offset, head) pairs per slab
    constexpr int WPT = (WSLAB + NT - 1) / NT;
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    float *g = reinterpret_cast<float *>(smem);
    u32x2 *wds = reinterpret_cast<u32x2 *>(smem + GN * 4);  // [2][KS][TNW]

    const int R = tab_rows<OP>(a);
    if (a.tx * 64 * TM * WR >= R) return;  // uniform over the workgroup
    const int lane = threadIdx.x & 63;
    const int wave = wave_id();
    const int rg = wave % WR, cg = wave / WR;
    const int row0 = a.tx * (64 * TM * WR) + rg * (64 * TM) + lane;
    const bool live = row0 - lane < R;  // wave-uniform: a wave past the end only stages
    const int colw = a.ty * TNW;
    const int col0 = colw + cg * TN;
    int abase[TM];
#pragma unroll
    for (int r = 0; r < TM; ++r) {
        const int row = row0 + 64 * r;
        abase[r] = row < R ? tab_row_rec<OP>(a, row) : 0;
    }
    const AView<TM> av = make_aview<OP, TM>(a, abase);
    const int count = tab_count<OP>(a);
    const int ch = a.chunk;
    const int cpt = (count + ch - 1) / ch;
    const int q_total = tab_taps<OP>(a) * cpt;
    const int q0 = tab_split(a) * a.chunks_per_split;
    const int p_end = min(q_total, q0 + a.chunks_per_split) * ch;

    // g from the transposed rows (row kb holds entry (ka, kb) at byte (kb * 2^RL + ka) * eb)
    for (int s = threadIdx.x; s < GN; s += NT) {
        const int ka = min(s, (1 << RL) - 1), kb = s - ka;
        float v = 0.0f;
        if (kb < (1 << RL)) {
            const unsigned char *src = a.rows + ((size_t(kb) << RL) + size_t(ka)) * eb;
            const uint32_t vadd = ROUNDED ? a.vadd : 0u;
            v = eb == 1 ? tab_value_scaled<1>(src, vadd)
                        : (eb == 2 ? tab_value_scaled<2>(src, vadd) : tab_value_scaled<4>(src, vadd));
        }
        g[s] = v;
    }
    // The second operand's pairs of a slab: thread -> (slot, column) c = threadIdx.x + i * NT.
    // A second-operand index outside the table is a zero's (its product is a signed zero whatever
    // it reads): it reads g(ka).
    uint32_t sw[WPT];
    auto fetch = [&](const TabTap &tp, int c0_) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < WPT; ++i) {
            const int c = threadIdx.x + i * NT;
            const int slot = c / TNW, t = c % TNW, j = c0_ + slot;
            sw[i] = (c < WSLAB && j < tp.count) ? Bd_word(a, tp.bbase + j, colw + t) : 0u;
        }
    };
    auto commit = [&](int buf_) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < WPT; ++i) {
            const int c = threadIdx.x + i * NT;
            if (WPT * NT > WSLAB && c >= WSLAB) break;
            const uint32_t kb = (sw[i] & kIdxMask) >> RL;
            wds[buf_ * WSLAB + c] = u32x2{(kb < (1u << RL) ? kb : 0u) * 4u, sw[i] & kHeadMask};
        }
    };
    float acc[TM][TN];
    init_acc(acc);
    uint32_t acur[TM];
    auto advance = [&](const TabTap &t, int tp_, int c, TabTap &o, int &otap, int &oc, bool &ok)
                       __attribute__((always_inline)) {
        o = t;
        otap = tp_;
        oc = c + KS;
        if (oc >= count) {
            otap = tp_ + 1;
            oc = 0;
        }
        ok = otap * cpt * ch + oc < p_end;
        if (ok && otap != tp_) o = tab_tap<OP>(a, otap);
    };
    TabTap cur{0, 0, 0, 0};
    int tap = q0 / max(cpt, 1);
    int c0 = (q0 - tap * cpt) * ch;
    bool have = q0 * ch < p_end;
    TabTap nxt{0, 0, 0, 0};
    int ntap = 0, nc0 = 0;
    bool has_next = false;
    if (have) {
        cur = tab_tap<OP>(a, tap);
        fetch(cur, c0);
        commit(0);
        load_a_words<OP, TM>(acur, av, __builtin_amdgcn_readfirstlane(a_step_offset<OP>(cur, c0)), c0);
        advance(cur, tap, c0, nxt, ntap, nc0, has_next);
    }
    __syncthreads();
    int buf = 0;
    while (have) {
        uniform_cursor(cur, tap, c0);
        uniform_cursor(nxt, ntap, nc0);
        if (has_next) fetch(nxt, nc0);
        const u32x2 *wb = wds + buf * WSLAB + cg * TN;
        const int nslots = live ? min(min(KS, cur.count - c0), p_end - (tap * cpt * ch + c0)) : 0;
        __builtin_amdgcn_s_setprio(3);
        for (int slot = 0; slot < nslots; ++slot) {
            uint32_t anext[TM];
            const bool in_slab = slot + 1 < nslots;
            const uint32_t unext = __builtin_amdgcn_readfirstlane(in_slab ? a_step_offset<OP>(cur, c0 + slot + 1)
                                                                          : a_step_offset<OP>(nxt, nc0));
            const int jnext = __builtin_amdgcn_readfirstlane(in_slab ? c0 + slot + 1 : nc0);
            if (in_slab || has_next) {
                load_a_words<OP, TM>(anext, av, unext, jnext);
            } else {
#pragma unroll
                for (int r = 0; r < TM; ++r) anext[r] = 0u;
            }
            uint32_t ao[TM];
            float pa[TM];
#pragma unroll
            for (int r = 0; r < TM; ++r) {
                ao[r] = __builtin_amdgcn_ubfe(acur[r], 4, RL) * 4u;  // idx = ka << 4
                pa[r] = head_value(acur[r]);
            }
            // every gather of the step before the first product: one LDS latency per step
            float v[TM][TN], pb[TN];
#pragma unroll
            for (int t = 0; t < TN; ++t) {
                const u32x2 w = wb[slot * TNW + t];
                pb[t] = __uint_as_float(w.y);
#pragma unroll
                for (int r = 0; r < TM; ++r) v[r][t] = *reinterpret_cast<const float *>(smem + ao[r] + w.x);
            }
            __builtin_amdgcn_sched_barrier(0);  // the scheduler would interleave them with the products
#pragma unroll
            for (int t = 0; t < TN; ++t) {
#pragma unroll
                for (int r = 0; r < TM; ++r) {
                    if constexpr (ROUNDED) {
                        const float c = v[r][t] * (pa[r] * pb[t]);
                        acc[r][t] = __builtin_fmaf(c * a.su, a.sd, acc[r][t]);
                    } else {
                        acc[r][t] = __builtin_fmaf(v[r][t], pa[r] * pb[t], acc[r][t]);
                    }
                }
            }
#pragma unroll
            for (int r = 0; r < TM; ++r) acur[r] = anext[r];
        }
        __builtin_amdgcn_s_setprio(0);
        if (has_next) commit(buf ^ 1);
        __syncthreads();
        cur = nxt;
        tap = ntap;
        c0 = nc0;
        buf ^= 1;
        have = has_next;
        if (have) advance(cur, tap, c0, nxt, ntap, nc0, has_next);
    }

    float *out = a.out + int64_t(tab_split(a)) * a.out_elems;
#pragma unroll
    for (int r = 0; r < TM; ++r) {
        const int row = row0 + 64 * r;
        if (row >= R) continue;
        float *dst = out + tab_row_out<OP>(a, row);
#pragma unroll
        for (int t = 0; t < TN; ++t) {
            const int col = col0 + t;
            if (col < a.N) dst[col] = acc[r][t];
        }
    }
}

// ------------------------------------------------------- native multiply (no table)
// The same kernels with the native FP32 multiply (the paper's ATnG configuration: its custom kernels
// with the `*` operator): operands are kept raw by the decode passes (pair records hold the two
// steps' values in their first and last words), the slab stages the second operand's values only,
// and every product is one fma into the sum.
constexpr int kNativeSlabSteps = 16;

template <int OP, int TM>
__device__ __forceinline__ void load_a_raw(float (&dst)[TM], const AView<TM> &av, uint32_t so, int j)
{
#pragma unroll
    for (int r = 0; r < TM; ++r) {
        const u32x2 d = __builtin_amdgcn_raw_buffer_load_b64(av.words, av.aoff[r], so + (j & 1) * 4u, 0);
        dst[r] = __uint_as_float((j & 1) ? d.y : d.x);
    }
}

template <int OP, int TM, int TN, int WR, int NW>
__device__ __forceinline__ void tab_body_native(const TabArgs &a)
{
    constexpr int NT = 64 * NW;
    constexpr int WC = NW / WR;
    constexpr int TNW = TN * WC;
    constexpr int KS = kNativeSlabSteps;
    constexpr int CPT = (KS * TNW + NT - 1) / NT;  // staged values per thread per slab
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    float *bs = reinterpret_cast<float *>(smem);  // [2][KS][TNW] second-operand values

    const int R = tab_rows<OP>(a);
    if (a.tx * 64 * TM * WR >= R) return;  // uniform over the workgroup
    const int lane = threadIdx.x & 63;
    const int wave = wave_id();
    const int rg = wave % WR, cg = wave / WR;
    const int row0 = a.tx * (64 * TM * WR) + rg * (64 * TM) + lane;
    const bool live = row0 - lane < R;
    const int colw = a.ty * TNW;
    const int col0 = colw + cg * TN;
    int abase[TM];
#pragma unroll
    for (int r = 0; r < TM; ++r) {
        const int row = row0 + 64 * r;
        abase[r] = row < R ? tab_row_rec<OP>(a, row) : 0;  // rows past the end read record 0's run
    }
    const AView<TM> av = make_aview<OP, TM>(a, abase);
    const int count = tab_count<OP>(a);
    const int ch = a.chunk;
    const int cpt = (count + ch - 1) / ch;
    const int q_total = tab_taps<OP>(a) * cpt;
    const int q0 = tab_split(a) * a.chunks_per_split;
    const int p_end = min(q_total, q0 + a.chunks_per_split) * ch;

    float stage[CPT];
    auto fetch = [&](const TabTap &tp, int c) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int e = int(threadIdx.x) + i * NT;
            const int slot = e / TNW, t = e % TNW;
            const int j = c + slot;
            stage[i] = (e < KS * TNW && j < tp.count) ? __uint_as_float(Bd_word(a, tp.bbase + j, colw + t)) : 0.0f;
        }
    };
    auto commit = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int e = int(threadIdx.x) + i * NT;
            if (e < KS * TNW) bs[buf * KS * TNW + e] = stage[i];
        }
    };
    float acc[TM][TN];
    init_acc(acc);
    TabTap cur{0, 0, 0, 0};
    int tap = q0 / max(cpt, 1);
    int c0 = (q0 - tap * cpt) * ch;
    bool have = q0 * ch < p_end;
    if (have) {
        cur = tab_tap<OP>(a, tap);
        fetch(cur, c0);
        commit(0);
    }
    __syncthreads();
    int buf = 0;
    while (have) {
        uniform_cursor(cur, tap, c0);
        TabTap nxt = cur;
        int ntap = tap, nc0 = c0 + KS;
        if (nc0 >= count) {
            ntap = tap + 1;
            nc0 = 0;
        }
        const bool has_next = ntap * cpt * ch + nc0 < p_end;
        if (has_next && ntap != tap) nxt = tab_tap<OP>(a, ntap);
        if (has_next) fetch(nxt, nc0);
        const int nslots = live ? min(min(KS, cur.count - c0), p_end - (tap * cpt * ch + c0)) : 0;
        const float *bsl = bs + buf * KS * TNW + cg * TN;
        float av0[TM];
        if (nslots > 0) load_a_raw<OP, TM>(av0, av, __builtin_amdgcn_readfirstlane(a_step_offset<OP>(cur, c0)), c0);
#pragma unroll
        for (int slot = 0; slot < KS; ++slot) {
            if (slot >= nslots) break;
            float an[TM];
            if (slot + 1 < nslots) {
                const uint32_t so = __builtin_amdgcn_readfirstlane(a_step_offset<OP>(cur, c0 + slot + 1));
                load_a_raw<OP, TM>(an, av, so, c0 + slot + 1);
            }
#pragma unroll
            for (int t = 0; t < TN; ++t) {
                const float b = bsl[slot * TNW + t];
#pragma unroll
                for (int r = 0; r < TM; ++r) acc[r][t] = __builtin_fmaf(av0[r], b, acc[r][t]);
            }
            if (slot + 1 < nslots) {
#pragma unroll
                for (int r = 0; r < TM; ++r) av0[r] = an[r];
            }
        }
        if (has_next) commit(buf ^ 1);
        __syncthreads();
        cur = nxt;
        tap = ntap;
        c0 = nc0;
        buf ^= 1;
        have = has_next;
    }

    float *out = a.out + int64_t(tab_split(a)) * a.out_elems;
#pragma unroll
    for (int r = 0; r < TM; ++r) {
        const int row = row0 + 64 * r;
        if (row >= R) continue;
        float *dst = out + tab_row_out<OP>(a, row);  // recomputed rather than kept in registers
#pragma unroll
        for (int t = 0; t < TN; ++t) {
            const int col = col0 + t;
            if (col < a.N) dst[col] = acc[r][t];
        }
    }
}

// ---------------------------------------------------------- bf16 pair path (1-byte tables)
// When every table entry fits 8 bits (its low 16 mantissa bits are zero) a table value v is a
// bfloat16, and so are v * pb (the second operand's sign and exponent added to v's bits) and pa.
// Products of such operands are exact in fp32, so two reduction steps k, k+1 can go through one
// v_dot2_f32_bf16:  acc += t(k) * pa(k) + t(k+1) * pa(k+1),  t = v * pb.
// The slab then holds, per step and first-operand mantissa ka, one 16-byte entry with t for the
// workgroup's 8 columns (8 bf16); a lane reads it with one ds_read_b128 and pairs the halves of
// two steps' entries with v_perm.
// Exactness needs every product of finite non-zero operands to stay normal (exponent field
// Ea + Eb - 127 + carry in [1, 254]) and v * pb not to overflow; the decode passes record the
// operands' exponent range and the kernel takes this path only when that holds (else the exact
// path).  Inside that range each product is the exact Algorithm 2 result; the sum is rounded
// per pair instead of per step.  A sum that comes out exactly zero gets its sign from a second
// pass over its products (the hardware returns +0 for zero sums; the sign of a sum of zeros is
// -0 exactly when every product is -0).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint16_t u16x2_t __attribute__((ext_vector_type(2)));

// Columns per entry DC: 8, or 4 for narrow outputs.  Entries sit 16 bytes apart either way (the
// first operand's index field is the byte offset ka * 16); a 4-column entry fills half a slot.
constexpr bool dot_cols_ok(int dc) { return dc == 8 || dc == 4; }
constexpr int kDotStepBytes = kTabRowEntries * 16;  // 128 entries, 16-byte slots
// Steps per slab: 2 per wave (each thread stages one step's entry group, 32 threads per step).
constexpr int dot_slab_steps(int nw) { return nw * 2; }

// 16 bytes of LDS at byte address off + imm.  The table kernels use no static LDS, so their
// dynamic allocation starts at LDS address 0 (checked on the host when the kernels are set up);
// addressing it as such lets the constant part land in the instruction's offset field.
typedef __attribute__((address_space(3))) const u32x4 lds_u32x4;
__device__ __forceinline__ u32x4 lds_load_b128(uint32_t off, uint32_t imm)
{
    return reinterpret_cast<lds_u32x4 *>(uintptr_t(off))[imm / 16];
}

// The same for 8 bytes (imm a multiple of 8).
typedef __attribute__((address_space(3))) const u32x2 lds_u32x2;
__device__ __forceinline__ u32x2 lds_load_b64(uint32_t off, uint32_t imm)
{
    return reinterpret_cast<lds_u32x2 *>(uintptr_t(off))[imm / 8];
}

__device__ __forceinline__ float dot2_bf16(uint32_t x, uint32_t y, float c)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, x), __builtin_bit_cast(bf16x2_t, y), c,
                                           false);
}

__device__ __forceinline__ uint32_t add_u16x2(uint32_t x, uint32_t y)
{
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2_t, x) + __builtin_bit_cast(u16x2_t, y));
}

// Staging of one slab: thread -> step slot (tid / 32) and entry group g (tid % 32), which builds
// the entries ka = g, g + 32, g + 64, g + 96.  Fetch, in two parts: the slot's DC second-operand
// words, then, per column, the 4 bytes of its table row that hold those entries.
template <int DC>
__device__ __forceinline__ void dot_fetch_b(u32x4 (&bw)[2], const TabTap &tp, int c0, const uint32_t *__restrict__ Bd,
                                            int Np, int colw)
{
    const int slot = threadIdx.x >> 5;
    const int j = c0 + slot;
    if (j < tp.count) {
        const u32x4 *src = reinterpret_cast<const u32x4 *>(Bd + int64_t(tp.bbase + j) * Np + colw);
        bw[0] = src[0];
        bw[1] = DC == 8 ? src[1] : bw[0];
    } else {  // a padding step: +0 operands, whose entries are +0
        bw[0] = u32x4{kZeroRowWord, kZeroRowWord, kZeroRowWord, kZeroRowWord};
        bw[1] = bw[0];
    }
}

template <int DC>
__device__ __forceinline__ void dot_fetch_rows(uint32_t (&rw)[DC], const u32x4 (&bw)[2], __amdgpu_buffer_rsrc_t rres)
{
    const int g = threadIdx.x & 31;
#pragma unroll
    for (int c = 0; c < DC; ++c) {
        const uint32_t w = bw[c / 4][c % 4];  // idx = kb * 128 (kZeroRow for zeros)
        rw[c] = __builtin_amdgcn_raw_buffer_load_b32(rres, (w & 0x7F80u) | uint32_t(g * 4), 0, 0);
    }
}

// Commit: t = v * pb as bf16 bits = table byte + (pb's bits >> 16); a zero second operand reads
// the zero row and gets signed zeros.  Entry dword q = (t of column 2q, t of column 2q + 1).
template <int DC>
__device__ __forceinline__ void dot_commit(const u32x4 (&bw)[2], const uint32_t (&rw)[DC], unsigned char *slab)
{
    const int slot = threadIdx.x >> 5, g = threadIdx.x & 31;
    const uint32_t(&w)[DC] = rw;
    uint32_t hb[DC / 2];
#pragma unroll
    for (int q = 0; q < DC / 2; ++q)
        hb[q] = __builtin_amdgcn_perm(bw[(2 * q + 1) / 4][(2 * q + 1) % 4], bw[(2 * q) / 4][(2 * q) % 4], 0x07060302u);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint32_t e[DC / 2];
#pragma unroll
        for (int q = 0; q < DC / 2; ++q) {
            // low half: byte i of the even column's word, high half: byte i of the odd one's
            const uint32_t d = __builtin_amdgcn_perm(w[2 * q + 1], w[2 * q], 0x0C000C00u | ((4u + i) << 16) | i);
            e[q] = add_u16x2(d, hb[q]);
        }
        unsigned char *dst = slab + slot * kDotStepBytes + (g + 32 * i) * 16;
        if constexpr (DC == 8)
            *reinterpret_cast<u32x4 *>(dst) = u32x4{e[0], e[1], e[2], e[3]};
        else
            *reinterpret_cast<u32x2 *>(dst) = u32x2{e[0], e[1]};
    }
}

// First-operand data of the step pair (j, j + 1) per lane row: the two indices and the head pair.  A step past the tap's end (the odd step of a pair, or a
// slab's unused slots) reads the tap's last step again: its slot in the slab holds +0 entries
// (staged from a +0 second operand), so it adds signed zeros only, and the loads stay
// branch-free and in bounds.
template <int OP, int TM>
__device__ __forceinline__ void dot_load_pair(uint32_t (&dst)[3][TM], const AView<TM> &av, const TabTap &tp, int j)
{
    // j even: one record holds both steps (past the end: the last record; an odd count's last
    // record has a decoded +0 for its missing step)
    const uint32_t so = __builtin_amdgcn_readfirstlane(a_step_offset<OP>(tp, min(j, tp.count - 1)));
#pragma unroll
    for (int r = 0; r < TM; ++r) {
        const u32x3 rec = __builtin_amdgcn_raw_buffer_load_b96(av.words, av.aoff[r], so, 0);
        dst[0][r] = rec.x;
        dst[1][r] = rec.z;
        dst[2][r] = rec.y;
    }
}

// The end of a pair-path body: the signs of exactly-zero sums, then the stores of the TM x TN
// outputs (or of the split's partial sums).
template <int OP, int TM, int TN>
__device__ __forceinline__ void dot_finish(const TabArgs &a, float (&acc)[TM][TN], const AView<TM> &av, int row0,
                                           int col0, int R, int q0, int cpt, int p_end, int ch)
{
    // Signs of zero sums: -0 when every product of the split's range is -0, else +0.  The first
    // product that is not -0 (non-zero, or +0) settles an output as +0, so the pass stops once no
    // output of the wave is pending -- after one step for a sum that cancelled to zero, after the
    // whole range only for outputs whose products are all -0.
    uint32_t pending = 0u;
#pragma unroll
    for (int r = 0; r < TM; ++r)
#pragma unroll
        for (int t = 0; t < TN; ++t)
            if (row0 + 64 * r < R && col0 + t < a.N && acc[r][t] == 0.0f) pending |= 1u << (r * TN + t);
    const uint32_t zero = pending;
    if (__builtin_amdgcn_ballot_w64(pending != 0u) != 0u) {
        bool open = true;
        for (int tp_i = q0 / max(cpt, 1); open && tp_i * cpt * ch < p_end; ++tp_i) {
            const int pbase = tp_i * cpt * ch;
            const TabTap tp = tab_tap<OP>(a, tp_i);
            const int j1 = min(tp.count, p_end - pbase);
            for (int j = max(q0 * ch - pbase, 0); j < j1; ++j) {
                uint32_t aw[TM];
                load_a_words<OP, TM>(aw, av, __builtin_amdgcn_readfirstlane(a_step_offset<OP>(tp, j)), j);
                const uint32_t *brow = a.Bd + int64_t(tp.bbase + j) * a.Np + col0;
#pragma unroll
                for (int t = 0; t < TN; ++t) {
                    const float pb = head_value(brow[t]);
#pragma unroll
                    for (int r = 0; r < TM; ++r)
                        if (__float_as_uint(head_value(aw[r]) * pb) != 0x80000000u) pending &= ~(1u << (r * TN + t));
                }
                if (__builtin_amdgcn_ballot_w64(pending != 0u) == 0u) {
                    open = false;
                    break;
                }
            }
        }
#pragma unroll
        for (int r = 0; r < TM; ++r)
#pragma unroll
            for (int t = 0; t < TN; ++t)
                if (zero & (1u << (r * TN + t))) acc[r][t] = (pending & (1u << (r * TN + t))) ? -0.0f : 0.0f;
    }

    float *out = a.out + int64_t(tab_split(a)) * a.out_elems;
#pragma unroll
    for (int r = 0; r < TM; ++r) {
        const int row = row0 + 64 * r;
        if (row >= R) continue;
        float *dst = out + tab_row_out<OP>(a, row);  // recomputed rather than kept in registers
#pragma unroll
        for (int t = 0; t < TN; ++t) {
            const int col = col0 + t;
            if (col < a.N) dst[col] = acc[r][t];
        }
    }
}

// Workgroup: NW waves along rows (64*TM rows each), all on the same 8 columns.  Every thread
// stages one step's entry group per slab (KS = 2 * NW steps x 32 groups).
template <int OP, int TM, int NW, int DC>
__device__ __forceinline__ void tab_body_dot(const TabArgs &a)
{
    static_assert(dot_cols_ok(DC), "8 or 4 columns per entry");
    constexpr int KS = dot_slab_steps(NW);
    constexpr int kDotSlab = KS * kDotStepBytes;
    constexpr int TN = DC;
    constexpr int NA = 3;  // first-operand registers per step pair and lane row (one record)
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

    const int R = tab_rows<OP>(a);
    if (a.tx * 64 * TM * NW >= R) return;  // uniform over the workgroup
    const int lane = threadIdx.x & 63;
    const int wave = wave_id();
    const int row0 = a.tx * (64 * TM * NW) + wave * (64 * TM) + lane;
    const bool live = row0 - lane < R;  // wave-uniform
    const int col0 = a.ty * TN;
    const __amdgpu_buffer_rsrc_t rres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<unsigned char *>(a.dot_rows), 0, int((kZeroRow + 1) * kTabRowEntries), 0x00020000);

    int abase[TM];
#pragma unroll
    for (int r = 0; r < TM; ++r) {
        const int row = row0 + 64 * r;
        abase[r] = row < R ? tab_row_rec<OP>(a, row) : 0;  // rows past the end read record 0's run
    }
    const AView<TM> av = make_aview<OP, TM>(a, abase);
    const int count = tab_count<OP>(a);
    const int ch = a.chunk;
    const int cpt = (count + ch - 1) / ch;
    const int q_total = tab_taps<OP>(a) * cpt;
    const int q0 = tab_split(a) * a.chunks_per_split;
    const int p_end = min(q_total, q0 + a.chunks_per_split) * ch;

    // Staging pipeline: while slab s is computed, the table bytes of slab s + 1 are fetched (its
    // second-operand words `sbw` having arrived during slab s - 1) and the second-operand words
    // of slab s + 2 are loaded into `sbw2`, so that the words' latency is not exposed once per
    // slab (8-step slabs lose most, 16-step slabs ~1%).  16-step slabs fetch both in slab s: their
    // registers go to the second gather set of the pair loop (the backward-data pass's, to its tap
    // arithmetic).
    constexpr bool AHEAD2 = NW <= 4;
    u32x4 sbw[2], sbw2[2];
    uint32_t srw[DC];
    float acc[TM][TN];
    init_acc(acc);
    // First-operand data of RS step pairs, as a ring: pair kp of a slab is in w[kp % RS]; while
    // it is used, pair kp + LA (of this slab, or one of the next slab's first LA pairs for the
    // last LA pairs) is loaded into w[(kp + LA) % RS].  A slab holds a multiple of RS pairs, so
    // after a full slab the next slab's first LA pairs sit in w[0] .. w[LA - 1].
    constexpr int RS = (KS / 2) % 4 == 0 ? 4 : KS / 2;
    // pairs loaded ahead: all of the ring but the pair in use, except in the backward-data pass,
    // whose tap arithmetic leaves registers for one pair less (with three its kernel spills)
    constexpr int LA = OP == OP_BWD_DATA ? RS - 2 : RS - 1;
    static_assert(RS >= 3 && (KS / 2) % RS == 0, "ring of step pairs");
    uint32_t w[RS][NA][TM];
    // The slab after (t, tp_, c): its tap, cursor and whether it is in this split's range (if not,
    // `o` stays `t`, so that loads aimed at it stay in bounds).
    auto advance = [&](const TabTap &t, int tp_, int c, TabTap &o, int &otap, int &oc, bool &ok)
                       __attribute__((always_inline)) {
        o = t;
        otap = tp_;
        oc = c + KS;
        if (oc >= count) {
            otap = tp_ + 1;
            oc = 0;
        }
        ok = otap * cpt * ch + oc < p_end;
        if (ok && otap != tp_) o = tab_tap<OP>(a, otap);
    };
    TabTap cur{0, 0, 0, 0};
    int tap = q0 / max(cpt, 1);
    int c0 = (q0 - tap * cpt) * ch;
    bool have = q0 * ch < p_end;
    TabTap nxt{0, 0, 0, 0};
    int ntap = 0, nc0 = 0;
    bool has_next = false;
    if (have) {
        cur = tab_tap<OP>(a, tap);
        dot_fetch_b<DC>(sbw, cur, c0, a.Bd, a.Np, col0);
        dot_fetch_rows<DC>(srw, sbw, rres);
        dot_commit<DC>(sbw, srw, smem);
#pragma unroll
        for (int k = 0; k < LA; ++k) dot_load_pair<OP, TM>(w[k], av, cur, c0 + 2 * k);
        advance(cur, tap, c0, nxt, ntap, nc0, has_next);
        if (AHEAD2 && has_next) dot_fetch_b<DC>(sbw, nxt, nc0, a.Bd, a.Np, col0);
    }
    __syncthreads();
    // One slab from buffer BUF (a compile-time LDS offset, folded into the gathers' immediate
    // offsets); the next slab is staged into the other buffer.
    auto slab = [&](auto buf_c) __attribute__((always_inline)) {
        constexpr uint32_t BOFF = uint32_t(decltype(buf_c)::value) * kDotSlab;
        constexpr uint32_t NEXT = uint32_t(decltype(buf_c)::value ^ 1) * kDotSlab;
        uniform_cursor(cur, tap, c0);
        uniform_cursor(nxt, ntap, nc0);
        TabTap nxt2 = nxt;
        int ntap2 = ntap, nc02 = nc0;
        bool has_next2 = false;
        if constexpr (AHEAD2) {
            advance(nxt, ntap, nc0, nxt2, ntap2, nc02, has_next2);
            has_next2 = has_next2 && has_next;
            if (has_next) dot_fetch_rows<DC>(srw, sbw, rres);
            if (has_next2) dot_fetch_b<DC>(sbw2, nxt2, nc02, a.Bd, a.Np, col0);
        } else if (has_next) {
            dot_fetch_b<DC>(sbw, nxt, nc0, a.Bd, a.Np, col0);
            dot_fetch_rows<DC>(srw, sbw, rres);
        }
        // the slab ends at the tap's end or, 8-step chunks being the unit of splits, at the split's
        const int nslots = min(min(KS, cur.count - c0), p_end - (tap * cpt * ch + c0));
        // a wave whose rows all lie past the end only stages and keeps the barriers
        const int npairs = live ? (nslots + 1) / 2 : 0;
        // Waves computing a slab issue ahead of waves staging the next one or waiting at the
        // barrier (measured on MI355X: the GEMM 3-4% and the conv passes 2-9% faster than at one
        // priority): the gathers of the slowest waves keep the LDS busy, and a workgroup reaches
        // its barrier sooner.
        __builtin_amdgcn_s_setprio(3);
        // The two gathers of lane row r of pair kp: the entry byte offset is the mantissa field
        // * 16 (the index plane, or the word's low half under its head) plus the slot's, which is
        // a constant.
        auto gather = [&](int kp, int r, uint32_t(&X)[DC / 2], uint32_t(&Y)[DC / 2]) __attribute__((always_inline)) {
            const uint32_t o0 = w[kp % RS][0][r];
            const uint32_t o1 = w[kp % RS][1][r];
            if constexpr (DC == 8) {
                const u32x4 x4 = lds_load_b128(o0, BOFF + (2 * kp) * kDotStepBytes);
                const u32x4 y4 = lds_load_b128(o1, BOFF + (2 * kp + 1) * kDotStepBytes);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    X[q] = x4[q];
                    Y[q] = y4[q];
                }
            } else {
                const u32x2 x2 = lds_load_b64(o0, BOFF + (2 * kp) * kDotStepBytes);
                const u32x2 y2 = lds_load_b64(o1, BOFF + (2 * kp + 1) * kDotStepBytes);
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    X[q] = x2[q];
                    Y[q] = y2[q];
                }
            }
        };
        // Gathers run one lane row ahead of the products (two register sets), so that a wave's
        // own permutes and dots cover part of its gathers' latency; scheduling barriers keep the
        // compiler from hoisting more gathers (which costs registers).  The gather for the first
        // row of pair kp + 1 is issued even when the slab ends at kp: its ring slot then holds a
        // record already loaded (of this slab or the next), whose index words address this slab's
        // buffer, and the entries read are not used.  The backward-data pass, whose tap
        // arithmetic leaves no registers for the second set, gathers each row just before use.
        constexpr bool PIPE = OP != OP_BWD_DATA;
        uint32_t GX[2][DC / 2], GY[2][DC / 2];
        if (PIPE && npairs > 0) gather(0, 0, GX[0], GY[0]);
#pragma unroll
        for (int kp = 0; kp < KS / 2; ++kp) {
            if (kp >= npairs) break;
            if (kp + LA < KS / 2)
                dot_load_pair<OP, TM>(w[(kp + LA) % RS], av, cur, c0 + 2 * (kp + LA));
            else
                dot_load_pair<OP, TM>(w[(kp + LA) % RS], av, nxt, nc0 + 2 * (kp + LA - KS / 2));
#pragma unroll
            for (int r = 0; r < TM; ++r) {
                const int cb = PIPE ? (kp * TM + r) & 1 : 0;
                if constexpr (PIPE) {
                    __builtin_amdgcn_sched_barrier(0);
                    if (r + 1 < TM)
                        gather(kp, r + 1, GX[cb ^ 1], GY[cb ^ 1]);
                    else if (kp + 1 < KS / 2)
                        gather(kp + 1, 0, GX[cb ^ 1], GY[cb ^ 1]);
                    __builtin_amdgcn_sched_barrier(0);
                } else {
                    gather(kp, r, GX[0], GY[0]);
                }
                const uint32_t(&X)[DC / 2] = GX[cb];
                const uint32_t(&Y)[DC / 2] = GY[cb];
                const uint32_t pa = w[kp % RS][NA - 1][r];  // (pa(k), pa(k+1)) as bf16
#pragma unroll
                for (int q = 0; q < TN / 2; ++q) {
                    acc[r][2 * q] = dot2_bf16(__builtin_amdgcn_perm(Y[q], X[q], 0x05040100u), pa, acc[r][2 * q]);
                    acc[r][2 * q + 1] =
                        dot2_bf16(__builtin_amdgcn_perm(Y[q], X[q], 0x07060302u), pa, acc[r][2 * q + 1]);
                }
            }
        }
        if (live && npairs < KS / 2 && has_next) {  // a short slab: the next slab's first LA pairs
#pragma unroll
            for (int k = 0; k < LA; ++k) dot_load_pair<OP, TM>(w[k], av, nxt, nc0 + 2 * k);
        }
        __builtin_amdgcn_s_setprio(0);
        if (has_next) dot_commit<DC>(sbw, srw, smem + NEXT);
        __syncthreads();
        cur = nxt;
        tap = ntap;
        c0 = nc0;
        have = has_next;
        if constexpr (AHEAD2) {
            nxt = nxt2;
            ntap = ntap2;
            nc0 = nc02;
            has_next = has_next2;
            sbw[0] = sbw2[0];
            sbw[1] = sbw2[1];
        } else {
            advance(cur, tap, c0, nxt, ntap, nc0, has_next);
        }
    };
    while (have) {
        slab(std::integral_constant<int, 0>{});
        if (!have) break;
        slab(std::integral_constant<int, 1>{});
    }

    dot_finish<OP, TM, TN>(a, acc, av, row0, col0, R, q0, cpt, p_end, ch);
}

// ------------------------------------------------------- bf16 hi/lo path (2-byte tables)
// A 2-byte entry's value v has up to 16 significant bits: too many for one bf16, but v is the sum
// of two bf16 values v_hi (its top 8 bits) and v_lo (the rest; where that is zero, v_hi is
// lowered by one bf16 unit and v_lo is that unit, so that neither half is ever zero).  The
// table-preparation kernel stores, per row kb and first-operand mantissa ka, both halves (less
// the bias 0x3F80) in one word; the staging adds the column's pb bits to each half, giving
// (t_hi, t_lo) = (v_hi * pb, v_lo * pb) as a bf16 pair, and one v_dot2_f32_bf16 against
// (pa, pa) adds t_hi * pa + t_lo * pa = v * pb * pa, exact, to the sum: one instruction per
// product and 4 bytes of LDS per product.  Exactness needs every half-product normal: pb's
// exponent field >= 16 and Ea + Eb >= 143 (v_lo >= 2^-15), besides the bf16 path's upper bounds;
// the table preparation checks it against the decode statistics.  8-column tiles of 8 or 4 waves,
// all along rows: an 8-column entry is two 16-byte halves, each in a 2 KiB region of the step (so
// that the index word, ka * 16, addresses both), and a slab holds NW steps.
constexpr int kHlStepBytes = 2 * kDotStepBytes;        // two 4-column halves of 128 entries x 16 bytes
constexpr int kHlRowBytes = 64 * 2 * 4;                // per row kb: 64 groups x 2 entries x 4 bytes

// Staging of one hi/lo slab: thread -> step slot (tid / 64) and entry group g (tid % 64), which
// builds the entries ka = g and g + 64.
__device__ __forceinline__ void hl_fetch_b(u32x4 (&bw)[2], const TabTap &tp, int c0, const uint32_t *__restrict__ Bd,
                                           int Np, int colw)
{
    const int j = c0 + (threadIdx.x >> 6);
    if (j < tp.count) {
        const u32x4 *src = reinterpret_cast<const u32x4 *>(Bd + int64_t(tp.bbase + j) * Np + colw);
        bw[0] = src[0];
        bw[1] = src[1];
    } else {  // a padding step: +0 operands, whose entries are +0
        bw[0] = u32x4{kZeroRowWord, kZeroRowWord, kZeroRowWord, kZeroRowWord};
        bw[1] = bw[0];
    }
}

// Per column, the 8 bytes of its row kb (idx = kb * 128) that hold the group's two entries.
__device__ __forceinline__ void hl_fetch_rows(u32x2 (&rw)[8], const u32x4 (&bw)[2], __amdgpu_buffer_rsrc_t rres)
{
    const uint32_t g = threadIdx.x & 63;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        const uint32_t w = bw[c / 4][c % 4];
        rw[c] = __builtin_amdgcn_raw_buffer_load_b64(rres, ((w & 0x7F80u) << 2) | (g * 8u), 0, 0);
    }
}

// Commit: (t_hi, t_lo) = each stored half + pb's bf16 bits (the word's high half, which is pb with
// its mantissa cleared); a zero second operand reads the all-zero row and gets +-0 halves.
__device__ __forceinline__ void hl_commit(const u32x4 (&bw)[2], const u32x2 (&rw)[8], unsigned char *slab)
{
    const int slot = threadIdx.x >> 6, g = threadIdx.x & 63;
    uint32_t hb[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) hb[c] = __builtin_amdgcn_perm(bw[c / 4][c % 4], bw[c / 4][c % 4], 0x03020302u);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        uint32_t t[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) t[c] = add_u16x2(rw[c][i], hb[c]);
        unsigned char *dst = slab + slot * kHlStepBytes + (g + 64 * i) * 16;
        *reinterpret_cast<u32x4 *>(dst) = u32x4{t[0], t[1], t[2], t[3]};
        *reinterpret_cast<u32x4 *>(dst + kDotStepBytes) = u32x4{t[4], t[5], t[6], t[7]};
    }
}

// Workgroup: NW (8 or 4) waves along rows (64*TM rows each), all on the same 8 columns; slabs of
// NW steps.
template <int OP, int TM, int NW>
__device__ __forceinline__ void tab_body_hl(const TabArgs &a)
{
    static_assert(NW == 8 || NW == 4, "8 or 4 waves");
    constexpr int TN = 8, KS = NW;
    constexpr int kSlab = KS * kHlStepBytes;
    constexpr int NA = 3;  // first-operand registers per step pair and lane row (one record)
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

    const int R = tab_rows<OP>(a);
    if (a.tx * 64 * TM * NW >= R) return;  // uniform over the workgroup
    const int lane = threadIdx.x & 63;
    const int wave = wave_id();
    const int row0 = a.tx * (64 * TM * NW) + wave * (64 * TM) + lane;
    const bool live = row0 - lane < R;  // wave-uniform
    const int col0 = a.ty * TN;
    const __amdgpu_buffer_rsrc_t rres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<unsigned char *>(a.hl_rows), 0, int((kZeroRow + 1) * kHlRowBytes), 0x00020000);

    int abase[TM];
#pragma unroll
    for (int r = 0; r < TM; ++r) {
        const int row = row0 + 64 * r;
        abase[r] = row < R ? tab_row_rec<OP>(a, row) : 0;  // rows past the end read record 0's run
    }
    const AView<TM> av = make_aview<OP, TM>(a, abase);
    const int count = tab_count<OP>(a);
    const int ch = a.chunk;
    const int cpt = (count + ch - 1) / ch;
    const int q_total = tab_taps<OP>(a) * cpt;
    const int q0 = tab_split(a) * a.chunks_per_split;
    const int p_end = min(q_total, q0 + a.chunks_per_split) * ch;

    // while slab s is computed, slab s + 1's second-operand words and row halves are fetched
    u32x4 sbw[2];
    u32x2 srw[8];
    float acc[TM][TN];
    init_acc(acc);
    // the first operand's step pairs as a ring of four (8 waves) or two (4 waves; pair kp in
    // w[kp % RS]), loaded LA ahead
    constexpr int RS = NW == 8 ? 4 : 2;
    constexpr int LA = NW == 8 ? (OP == OP_BWD_DATA ? 2 : 3) : 1;
    static_assert((KS / 2) % RS == 0, "ring of step pairs");
    uint32_t w[RS][NA][TM];
    auto advance = [&](const TabTap &t, int tp_, int c, TabTap &o, int &otap, int &oc, bool &ok)
                       __attribute__((always_inline)) {
        o = t;
        otap = tp_;
        oc = c + KS;
        if (oc >= count) {
            otap = tp_ + 1;
            oc = 0;
        }
        ok = otap * cpt * ch + oc < p_end;
        if (ok && otap != tp_) o = tab_tap<OP>(a, otap);
    };
    TabTap cur{0, 0, 0, 0};
    int tap = q0 / max(cpt, 1);
    int c0 = (q0 - tap * cpt) * ch;
    bool have = q0 * ch < p_end;
    TabTap nxt{0, 0, 0, 0};
    int ntap = 0, nc0 = 0;
    bool has_next = false;
    if (have) {
        cur = tab_tap<OP>(a, tap);
        hl_fetch_b(sbw, cur, c0, a.Bd, a.Np, col0);
        hl_fetch_rows(srw, sbw, rres);
        hl_commit(sbw, srw, smem);
#pragma unroll
        for (int k = 0; k < LA; ++k) dot_load_pair<OP, TM>(w[k], av, cur, c0 + 2 * k);
        advance(cur, tap, c0, nxt, ntap, nc0, has_next);
    }
    __syncthreads();
    auto slab = [&](auto buf_c) __attribute__((always_inline)) {
        constexpr uint32_t BOFF = uint32_t(decltype(buf_c)::value) * kSlab;
        constexpr uint32_t NEXT = uint32_t(decltype(buf_c)::value ^ 1) * kSlab;
        uniform_cursor(cur, tap, c0);
        uniform_cursor(nxt, ntap, nc0);
        if (has_next) {
            hl_fetch_b(sbw, nxt, nc0, a.Bd, a.Np, col0);
            hl_fetch_rows(srw, sbw, rres);
        }
        const int nslots = min(min(KS, cur.count - c0), p_end - (tap * cpt * ch + c0));
        const int npairs = live ? (nslots + 1) / 2 : 0;
        __builtin_amdgcn_s_setprio(3);  // computing waves first, as on the bf16 path
#pragma unroll
        for (int kp = 0; kp < KS / 2; ++kp) {
            if (kp >= npairs) break;
            if (kp + LA < KS / 2)
                dot_load_pair<OP, TM>(w[(kp + LA) % RS], av, cur, c0 + 2 * (kp + LA));
            else
                dot_load_pair<OP, TM>(w[(kp + LA) % RS], av, nxt, nc0 + 2 * (kp + LA - KS / 2));
            const uint32_t(&a0)[TM] = w[kp % RS][0];
            const uint32_t(&a1)[TM] = w[kp % RS][1];
#pragma unroll
            for (int r = 0; r < TM; ++r) {
                const uint32_t o0 = a0[r];
                const uint32_t o1 = a1[r];
                const uint32_t pp = w[kp % RS][NA - 1][r];  // (pa(k), pa(k+1)) as bf16
                const uint32_t pk0 = __builtin_amdgcn_perm(pp, pp, 0x01000100u);  // (pa(k), pa(k))
                const uint32_t pk1 = __builtin_amdgcn_perm(pp, pp, 0x03020302u);  // (pa(k+1), pa(k+1))
                const u32x4 x0 = lds_load_b128(o0, BOFF + (2 * kp) * kHlStepBytes);
                const u32x4 x1 = lds_load_b128(o0, BOFF + (2 * kp) * kHlStepBytes + kDotStepBytes);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    acc[r][q] = dot2_bf16(x0[q], pk0, acc[r][q]);
                    acc[r][4 + q] = dot2_bf16(x1[q], pk0, acc[r][4 + q]);
                }
                const u32x4 y0 = lds_load_b128(o1, BOFF + (2 * kp + 1) * kHlStepBytes);
                const u32x4 y1 = lds_load_b128(o1, BOFF + (2 * kp + 1) * kHlStepBytes + kDotStepBytes);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    acc[r][q] = dot2_bf16(y0[q], pk1, acc[r][q]);
                    acc[r][4 + q] = dot2_bf16(y1[q], pk1, acc[r][4 + q]);
                }
            }
        }
        if (live && npairs < KS / 2 && has_next) {  // a short slab: the next slab's first LA pairs
#pragma unroll
            for (int k = 0; k < LA; ++k) dot_load_pair<OP, TM>(w[k], av, nxt, nc0 + 2 * k);
        }
        __builtin_amdgcn_s_setprio(0);
        if (has_next) hl_commit(sbw, srw, smem + NEXT);
        __syncthreads();
        cur = nxt;
        tap = ntap;
        c0 = nc0;
        have = has_next;
        advance(cur, tap, c0, nxt, ntap, nc0, has_next);
    };
    while (have) {
        slab(std::integral_constant<int, 0>{});
        if (!have) break;
        slab(std::integral_constant<int, 1>{});
    }

    dot_finish<OP, TM, TN>(a, acc, av, row0, col0, R, q0, cpt, p_end, ch);
}

// Four waves per SIMD: the register budget (<= 128 VGPRs) the tiles are sized for.  Without the
// hint the scheduler minimises registers and serialises the LDS gathers.
// RL: log2 of the table row length, 7 (rows padded to 128 entries) for M <= 7, else M.
// VAR: kTabApprox (the table's products) or kTabNative (the native FP32 multiply, RL = 7 only).
// kTabApproxSelf: the table's products, with the path decided by the kernel itself (tab_paths)
// instead of read from the flags -- for small calls, where one launch fewer matters more.
enum { kTabApprox = 0, kTabNative = 1, kTabApproxSelf = 2 };

// The exact path's product form: 1 when a product must be rounded on its own before it is added
// (t = v * (pa * pb), then the sum), 0 when fma(v, pa * pb, acc) gives the same result.  They
// differ only where v * (pa * pb) overflows to Inf -- exponent field Ea + Eb - 127 = 254 plus a
// carry -- which an fma would fold into the sum unrounded: impossible when the largest finite
// exponent fields of the two operands add up to at most 380.  Inf and NaN operands give the same
// result either way, but their statistics carry no exponent range, so they take the rounded form;
// so do formats with fewer exponent bits (`narrow`), whose products are scaled before the add,
// and calls without statistics.
__device__ __forceinline__ int exact_needs_rounded_products(bool have_stats, bool special, uint32_t a_hi,
                                                            uint32_t b_hi, int narrow)
{
    return (narrow || !have_stats || special || a_hi + b_hi > 380u) ? 1 : 0;
}

// The call's path from the reduced decode statistics -- the smallest exponent field (lo) and the
// largest with the Inf/NaN flag above it (hs = special << 8 | hi) of each operand's non-zero
// operands -- and the table's entry width eb.  flags[1] and flags[2] of a call hold it.
//   path 1, the bf16 path (1-byte entries): every product of finite non-zero operands has
//     exponent field Ea + Eb - 127 + carry in [1, 254], and v * pb (Eb + carry) stays below 255;
//   path 2, the hi/lo path (2-byte entries): also the low halves' products normal -- v_lo >=
//     2^-15 times pb normal as a bf16 (Eb >= 16) and times pa normal (Ea + Eb - 127 - 15 >= 1);
//   path 0, the exact path, whose product form is `rounded`.
// have: the decode passes recorded statistics (not for the native multiply).
__device__ __forceinline__ void decide_paths(int eb, uint32_t a_lo, uint32_t a_hs, uint32_t b_lo, uint32_t b_hs,
                                             bool have, int narrow, int &path, int &rounded)
{
    const uint32_t a_hi = a_hs & 0xFFu, b_hi = b_hs & 0xFFu;
    const bool special = ((a_hs | b_hs) >> 8) != 0u;
    const bool window = have && !special && a_lo + b_lo >= 128u && a_hi + b_hi <= 380u && b_hi <= 253u;
    const bool window_hl = window && b_lo >= 16u && a_lo + b_lo >= 143u;
    path = narrow ? 0 : ((eb == 1 && window) ? 1 : ((eb == 2 && window_hl) ? 2 : 0));
    rounded = exact_needs_rounded_products(have, special, a_hi, b_hi, narrow);
}

// Reduction of n statistics words (lo | hi << 8 | special << 16 per decode workgroup) into a
// thread's lo / hs, NT threads striding, four loads in flight; a word past the end reads as that
// of a workgroup that saw no operand.
template <int NT>
__device__ __forceinline__ void stats_fold(const uint32_t *__restrict__ stats, int n, uint32_t &lo, uint32_t &hs)
{
    for (int i0 = threadIdx.x; i0 < n; i0 += 4 * NT) {
        uint32_t v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = i0 + u * NT < n ? stats[i0 + u * NT] : 0xFFu;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            lo = min(lo, v[u] & 0xFFu);
            hs = max(hs, (v[u] >> 8) & 0x1FFu);
        }
    }
}

// The path decided by every workgroup of a kTabApproxSelf kernel at its start, from the decode
// statistics (a.n_a + a.n_b words) -- so that no launch sits between the pre-pass and the table
// kernel.  NW: waves of the workgroup; red: 4 NW + 2 words of LDS, free until the body's first
// barrier.
template <int NW>
__device__ __forceinline__ void tab_paths(const TabArgs &a, int eb, uint32_t *red, int &path, int &rounded)
{
    uint32_t alo = 255u, ahs = 0u, blo = 255u, bhs = 0u;
    const bool have = a.stats_a != nullptr;  // uniform
    if (have) {
        stats_fold<64 * NW>(a.stats_a, a.n_a, alo, ahs);
        stats_fold<64 * NW>(a.stats_b, a.n_b, blo, bhs);
    }
    alo = wave_min(alo);
    ahs = wave_max(ahs);
    blo = wave_min(blo);
    bhs = wave_max(bhs);
    const int wave = int(threadIdx.x) >> 6;
    if ((threadIdx.x & 63) == 0) {
        red[4 * wave + 0] = alo;
        red[4 * wave + 1] = ahs;
        red[4 * wave + 2] = blo;
        red[4 * wave + 3] = bhs;
    }
    __syncthreads();
    if (threadIdx.x == 0) {  // the decision, handed to every wave through LDS
        uint32_t a_lo = 255u, a_hs = 0u, b_lo = 255u, b_hs = 0u;
        for (int w = 0; w < NW; ++w) {
            a_lo = min(a_lo, red[4 * w + 0]);
            a_hs = max(a_hs, red[4 * w + 1]);
            b_lo = min(b_lo, red[4 * w + 2]);
            b_hs = max(b_hs, red[4 * w + 3]);
        }
        int p, r;
        decide_paths(eb, a_lo, a_hs, b_lo, b_hs, have, a.narrow, p, r);
        red[4 * NW + 0] = uint32_t(p);
        red[4 * NW + 1] = uint32_t(r);
    }
    __syncthreads();
    path = __builtin_amdgcn_readfirstlane(int(red[4 * NW + 0]));
    rounded = __builtin_amdgcn_readfirstlane(int(red[4 * NW + 1]));
    __syncthreads();  // the body's first LDS stores may overwrite red
}

template <int OP, int TM, int TN, int WR, int NW, int RL, int VAR>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(4, 4))) void tab_kernel(TabArgs args)
{
    TabArgs a = args;
    tab_tile_id(a.splits, a.tx, a.ty, a.tz);
    if constexpr (VAR == kTabNative) {
        tab_body_native<OP, TM, TN, WR, NW>(a);
        return;
    }
    const int eb = __builtin_amdgcn_readfirstlane(a.eb[0]);
    int self_path = 0, self_rounded = 0;
    if constexpr (VAR == kTabApproxSelf) {
        extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
        tab_paths<NW>(a, eb, reinterpret_cast<uint32_t *>(smem), self_path, self_rounded);
    }
    if constexpr (RL == 7 && dot_cols_ok(TN) && WR == NW) {
        const int path = VAR == kTabApproxSelf ? self_path : __builtin_amdgcn_readfirstlane(a.eb[1]);
        if (path == 1) {
            tab_body_dot<OP, TM, NW, TN>(a);
            return;
        }
        if constexpr (TN == 8 && (NW == 8 || NW == 4)) {
            if (path == 2) {
                tab_body_hl<OP, TM, NW>(a);
                return;
            }
        }
    }
    const int rounded = VAR == kTabApproxSelf ? self_rounded : __builtin_amdgcn_readfirstlane(a.eb[2]);
    if constexpr (RL >= 8) {
        if (__builtin_amdgcn_readfirstlane(a.eb[3]) == 1) {  // a sum-indexed table
            if (rounded)
                tab_body_sum<OP, TM, TN, WR, NW, RL, true>(a, eb);
            else
                tab_body_sum<OP, TM, TN, WR, NW, RL, false>(a, eb);
            return;
        }
    }
    if (rounded) {
        if (eb == 1)
            tab_body<OP, TM, TN, WR, 1, NW, RL, true>(a);
        else if (eb == 2)
            tab_body<OP, TM, TN, WR, 2, NW, RL, true>(a);
        else
            tab_body<OP, TM, TN, WR, 4, NW, RL, true>(a);
    } else {
        if (eb == 1)
            tab_body<OP, TM, TN, WR, 1, NW, RL, false>(a);
        else if (eb == 2)
            tab_body<OP, TM, TN, WR, 2, NW, RL, false>(a);
        else
            tab_body<OP, TM, TN, WR, 4, NW, RL, false>(a);
    }
}

// Dynamic LDS of a table kernel with TN columns per wave, WR of its NW waves along rows and rows
// of 2^RL entries: two exact-path slabs (the widest entry width) plus the second-operand heads, or
// two bf16-path slabs where that path exists.
constexpr size_t tab_exact_lds_bytes(int tnw, int rl, int eb)
{
    return size_t(2) * tab_slab_steps(tnw, rl, eb) * tnw * ((size_t(1) << rl) * eb) +
           size_t(2) * tab_slab_steps(tnw, rl, eb) * tnw * 4;
}

constexpr size_t tab_native_lds_bytes(int tn, int wr, int nw)
{
    return size_t(2) * kNativeSlabSteps * tn * (nw / wr) * 4;
}

constexpr size_t tab_lds_bytes(int tn, int wr, int nw, int rl)
{
    const int tnw = tn * (nw / wr);
    size_t b = tab_exact_lds_bytes(tnw, rl, 1);
    b = tab_exact_lds_bytes(tnw, rl, 2) > b ? tab_exact_lds_bytes(tnw, rl, 2) : b;
    b = tab_exact_lds_bytes(tnw, rl, 4) > b ? tab_exact_lds_bytes(tnw, rl, 4) : b;
    const size_t dot = (rl == 7 && dot_cols_ok(tn) && wr == nw) ? size_t(2) * dot_slab_steps(nw) * kDotStepBytes : 0;
    const size_t hl = (rl == 7 && tn == 8 && (nw == 8 || nw == 4) && wr == nw) ? size_t(2) * nw * kHlStepBytes : 0;
    const size_t sum = rl >= 8 ? tab_sum_lds_bytes(tnw, rl) : 0;
    b = b > dot ? b : dot;
    b = b > sum ? b : sum;
    return b > hl ? b : hl;
}

// ------------------------------------------------------------------ instantiated tiles -----

// A table-kernel tile: TM rows per lane, TN columns per wave, WR of the NW waves along rows, and
// the reduction split the host chose for the launch.
struct Tile {
    int tm = 1, tn = 4, split = 1;
    int wr = 4;  // waves along rows (the rest take column groups)
    int nw = 4;  // waves per workgroup
};

// Tile candidates of the host's tile chooser, per table-row length: the instantiated
// (TM, TN, WR, NW) tiles.  Tiles whose registers would spill past the 128-VGPR budget are left
// out.
struct TabCand {
    int tm, tn, wr, nw;
};
constexpr TabCand kTabCands[] = {{4, 8, 8, 8}, {4, 8, 4, 4}, {3, 8, 4, 4}, {2, 8, 4, 4}, {1, 8, 4, 4},
                                 {4, 4, 8, 8}, {4, 4, 4, 4}, {2, 4, 4, 4}, {1, 4, 4, 4}, {4, 8, 2, 4}, {2, 8, 2, 4},
                                 {1, 8, 2, 4}, {2, 8, 1, 4}, {1, 8, 1, 4}};
// Wide rows (M = 8..10; 11 uses the 4-column tiles, whose 4-byte-entry slab of one step fits 32 KiB).
constexpr TabCand kWideCands[] = {{8, 4, 8, 8}, {4, 8, 8, 8}, {2, 8, 4, 4}, {1, 8, 4, 4}, {1, 4, 4, 4}};
constexpr TabCand kWide11Cands[] = {{8, 4, 8, 8}, {4, 4, 8, 8}, {2, 4, 4, 4}, {1, 4, 4, 4}};

// The instantiated (TM, TN, WR, NW, RL) tiles: every candidate above, with its row length.
#define AMSIM_FOR_TAB_TILES(X)                                                                                \
    X(4, 8, 8, 8, 7) X(4, 8, 4, 4, 7) X(3, 8, 4, 4, 7) X(2, 8, 4, 4, 7) X(1, 8, 4, 4, 7) X(4, 4, 8, 8, 7)     \
    X(4, 4, 4, 4, 7) X(2, 4, 4, 4, 7) X(1, 4, 4, 4, 7) X(4, 8, 2, 4, 7) X(2, 8, 2, 4, 7) X(1, 8, 2, 4, 7)     \
    X(2, 8, 1, 4, 7) X(1, 8, 1, 4, 7) AMSIM_WIDE_TILES(X, 8) AMSIM_WIDE_TILES(X, 9) AMSIM_WIDE_TILES(X, 10) X(8, 4, 8, 8, 11)     \
    X(4, 4, 8, 8, 11) X(2, 4, 4, 4, 11) X(1, 4, 4, 4, 11)
#define AMSIM_WIDE_TILES(X, RL)                                                                                \
    X(8, 4, 8, 8, RL) X(4, 8, 8, 8, RL) X(2, 8, 4, 4, RL) X(1, 8, 4, 4, RL) X(1, 4, 4, 4, RL)

// Every candidate the chooser can return is instantiated (checked at compile time).
constexpr bool tab_tile_listed(const TabCand &c, int rl)
{
#define X(TM, TN, WR, NW, RL) \
    if (c.tm == TM && c.tn == TN && c.wr == WR && c.nw == NW && rl == RL) return true;
    AMSIM_FOR_TAB_TILES(X)
#undef X
    return false;
}
template <size_t N>
constexpr bool tab_cands_listed(const TabCand (&cands)[N], int rl_lo, int rl_hi)
{
    for (size_t i = 0; i < N; ++i)
        for (int rl = rl_lo; rl <= rl_hi; ++rl)
            if (!tab_tile_listed(cands[i], rl)) return false;
    return true;
}
static_assert(tab_cands_listed(kTabCands, 7, 7) && tab_cands_listed(kWideCands, 8, 10) &&
                  tab_cands_listed(kWide11Cands, 11, 11),
              "a tile candidate is missing from AMSIM_FOR_TAB_TILES");

// Per operation (defined in amsim_tab.hip, one instantiation per operation): raise the dynamic
// LDS limit of every instantiated tile's kernel and check that none uses static LDS; launch the
// kernel of tile t with rows of 2^rl entries and variant var (kTabNative and kTabApproxSelf: rl = 7).  Both return the first HIP error, and the launch
// hipErrorInvalidConfiguration for a tile that is not instantiated.
template <int OP>
hipError_t tab_attributes();
template <int OP>
hipError_t tab_launch(const Tile &t, int rl, int var, const TabArgs &a, dim3 grid, hipStream_t st);

}  // namespace amsim_detail
