// crf_internal.h -- what the host plan code and the gfx950 kernels share.
//
// Not part of the public ABI (that is include/crf_inside.h).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "../../include/crf_inside.h"

namespace crf {

// Workgroup sizes.  Bundled LDS kernels run kThreadsDefault threads, two
// workgroups per CU when every bundle fits in half the LDS, else one; the
// workspace ("spill") kernels run kThreadsMax.  Every kernel is built for up
// to kThreadsMax threads and reads its size from blockDim.
constexpr int kThreadsDefault = 512;
constexpr int kThreadsMax = 1024;

// Most sentences per bundle (bounds the per-sentence tables in LDS; each
// thread of a bundle's workgroup fetches at most one sentence id).
constexpr int kMaxBundle = 256;
static_assert(kMaxBundle <= kThreadsDefault, "one sentence id per thread");

// LDS a bundle keeps besides its charts and per-sentence tables: n + 2
// words of room.  Masked tail loads of the last chart of a bundle reach
// past it, into the tables that follow it: up to masked_reach(n) float32
// (inside, whose tables and this room always cover that) or float64 (CKY,
// whose tail the plan pads to that size).
__host__ __device__ inline int64_t bundle_extra_bytes(int n) { return 4 * (int64_t)(n + 2); }

// LDS a workgroup holds besides its bundle (the fused kernel's claim slot)
// and slack.  Bundle budgets leave it free.
constexpr int kReservedLds = 256;

// LDS has 32 four-byte banks, and each 32-lane half of a wavefront is served
// on its own: lanes of one half that hit one bank with different addresses
// are served one after another.
//
// Inside chart geometry of a bundle of nb sentences of n words: row stride
// ld >= n + 1 and chart stride cs >= 2 ld^2 (elements) of the two squares.
// A width step numbers its spans sentence-minor, g = i nb + sb (span start i,
// sentence sb), and every operand run of span g starts at sb cs + i ld plus
// an offset uniform over the step.  With cs = sigma and ld = nb sigma
// (mod 32) that start is sigma g (mod 32) for every g, whatever the step:
// lanes that take g, g + q, g + 2q, ... with their G split lanes side by side
// then cover 32 distinct banks when sigma q = G times an odd number (the
// sweeps pick q = G >> e, where 2^e is the power of two in sigma).
// The strict layout: sigma odd (e = 0) and ld with the same power of two as
// nb, both the smallest that fit, except
//  - bundles of 32 or more sentences whose count has a factor 4: ld odd and
//    sigma = 1 (the start then jumps only where i changes, every nb spans);
//  - sentences of 98 and 99 words keep ld = n + 1: padded, their two float32
//    squares would no longer fit in half a CU, and one bundle that needs a
//    whole CU moves every bundle of the launch to one workgroup per CU.  A
//    single sentence then takes sigma = ld (e = 2 at n = 99: the sweeps then
//    lay spans side by side, and its 4-lane steps, most of its work, stay
//    conflict-free).
// Of the sigma that satisfy these, the one that needs the least padding.
// A count with a factor 2^b widens the strict ld by up to 2^(b+1) words;
// where the strict layout would not fit in half a CU, the plan takes the
// loose one instead: the smallest ld = 1 or 2 (mod 4) and sigma odd with one
// word of padding, spans side by side (e = 5; about 2-way conflicts on the
// steps of 2 and 4 lanes, where interleaving them does worse).
struct InsideLayout {
    int ld, cs, e;
};
__host__ __device__ inline int pow2_mod32(int x) {   // the power of two in x mod 32 (5 for 0)
    x &= 31;
    if (x == 0) return 5;
    int b = 0;
    while ((x & 1) == 0) {
        x >>= 1;
        ++b;
    }
    return b;
}
__host__ __device__ inline int inverse_mod32(int m) {   // m odd: m x = 1 (mod 32)
    // Newton: each step doubles the correct low bits.  Unsigned, since the
    // products wrap (only the low five bits are kept).
    const uint32_t mu = (uint32_t)m;
    uint32_t x = mu;
    for (int k = 0; k < 4; ++k) x *= 2u - mu * x;
    return (int)(x & 31u);
}
constexpr int kInsideLdCap = 100;
__host__ __device__ inline InsideLayout inside_layout(int n, int nb, bool strict) {
    const int bn = pow2_mod32(nb);
    if (!strict || (nb >= 32 && bn >= 2)) {
        // loose: the smallest ld = 1 or 2 (mod 4), one word of padding (2 ld^2
        // is even, so sigma = 2 ld^2 + 1 is odd), spans side by side (e = 5)
        int ld = n + 1;
        while ((ld & 3) == 0 || (ld & 3) == 3) ++ld;
        if (ld > kInsideLdCap && n + 1 <= kInsideLdCap) ld = n + 1;
        return InsideLayout{ld, 2 * ld * ld + 1, 5};
    }
    int ld = n + 1;
    while (pow2_mod32(ld) != bn) ++ld;
    if (ld > kInsideLdCap && n + 1 <= kInsideLdCap) ld = n + 1;
    const int sq2 = 2 * ld * ld;
    int e = 0, pad = (1 - sq2) & 31;   // sigma = 1 where no sigma solves it
    const int bl = pow2_mod32(ld);
    if (bl >= bn && bn < 5) {
        // nb sigma = ld (mod 32): (nb >> b) sigma = ld >> b (mod 2^(5-b)),
        // 2^b solutions mod 32; the one needing the least padding
        const int step = 32 >> bn;
        const int s0 = ((ld >> bn) * inverse_mod32(nb >> bn)) & (step - 1);
        pad = 32;
        for (int s = s0; s < 32; s += step) pad = ((s - sq2) & 31) < pad ? (s - sq2) & 31 : pad;
        e = bl - bn;
    }
    return InsideLayout{ld, sq2 + pad, e};
}
// Row stride of a float64 CKY chart on the workspace, and of a loose one
// in LDS: even, which makes the diagonal stride ld + 1 odd.
__host__ __device__ inline int cky_ld(int n) { return (n + 1) + ((n + 1) & 1); }

// Bytes of chart per sentence.
//   inside: two float32 squares, padded to the chart stride of its bundle
//           (inside_layout) -- alpha (upper triangle + mirrored lower
//           triangle) and the outside values (upper + mirrored; before the
//           outside sweep reaches a span its mirrored cell holds the span's
//           score, and cells no sweep reads park the forced-span scores);
//   cky:    one float64 square (beta, upper + mirror), followed by the
//           split table (cky_split_index) when split_bytes > 0: the best
//           split k of every span (i, j) of two or more words, stored as
//           k - i - 1 in split_bytes bytes (1 for n <= kMaxLenInLds, 2 in
//           the workspace).  A bundle whose tables do not fit in LDS beside
//           its charts keeps them in the workspace (Bundle::split_ws).
__host__ __device__ inline int64_t cky_split_bytes_of(int n, int split_bytes) {
    return ((int64_t)n * (n - 1) / 2 * split_bytes + 7) / 8 * 8;
}
// CKY chart geometry of a bundle in LDS: row stride ld, chart stride cs
// (bytes, the chart and its split table, if in LDS, padded), and e as for
// the inside.  8-byte reads are served 16 lanes at a time over 16 bank
// pairs.  A step's spans are numbered sentence-minor, g = i nb + sb, and
// span g's two operand runs start at sb cs/8 + i (ld + 1) doubles (plus an
// offset uniform over the step): with cs/8 = sigma and ld + 1 = nb sigma
// (mod 16) that is sigma g (mod 16), and sigma odd with the spans
// interleaved over the G 16-lane groups of a block keeps every group on 16
// distinct bank pairs.  Strict: the smallest ld whose ld + 1 has nb's power
// of two, the odd sigma needing the least padding.  Loose (where the strict
// layout does not fit in half a CU, and bundles of 16 or more sentences
// whose count has a factor 4): ld even, sigma odd, spans still interleaved
// (a bank model of such bundles: 1.7x the conflict-free read cycles, 1.8x
// side by side).
struct CkyLayout {
    int ld, cs, e;
};
__host__ __device__ inline int pow2_mod16(int x) { return pow2_mod32(x & 15) >= 4 ? 4 : pow2_mod32(x & 15); }
__host__ __device__ inline CkyLayout cky_layout(int n, int nb, int split_bytes, bool strict) {
    const int bn = pow2_mod16(nb);
    const int64_t split = cky_split_bytes_of(n, split_bytes);
    if (!strict || (nb >= 16 && bn >= 2)) {
        const int ld = cky_ld(n);
        const int64_t u = ((int64_t)ld * ld * 8 + split) / 8;
        return CkyLayout{ld, (int)(8 * (u + ((u & 1) ^ 1))), 0};
    }
    int ld = n + 1;
    while (pow2_mod16(ld + 1) != bn) ++ld;
    const int64_t u = ((int64_t)ld * ld * 8 + split) / 8;
    int pad = (int)((1 - u) & 15), e = 0;
    const int bl = pow2_mod16(ld + 1);
    if (bn < 4) {
        // nb sigma = ld + 1 (mod 16): 2^b solutions; the least padding
        const int step = 16 >> bn;
        const int s0 = (((ld + 1) >> bn) * inverse_mod32(nb >> bn)) & (step - 1);
        pad = 16;
        for (int sg = s0; sg < 16; sg += step) pad = (int)((sg - u) & 15) < pad ? (int)((sg - u) & 15) : pad;
        e = bl - bn;
    }
    return CkyLayout{ld, (int)(8 * (u + pad)), e};
}
// Byte offset of an inside bundle's per-sentence tables (the first holds
// float64): its charts, rounded up to 8 bytes (the chart stride may be odd).
__host__ __device__ inline int64_t inside_tables_offset(int nb, int cs) { return ((int64_t)nb * cs * 4 + 7) & ~(int64_t)7; }
// LDS of an inside bundle: the charts, then per sentence the forced sum
// (f64), gradient (f32), id (i32) and score shift (f32), then the room of
// bundle_extra_bytes.
__host__ __device__ inline int64_t inside_bundle_bytes(int n, int nb, bool strict) {
    return inside_tables_offset(nb, inside_layout(n, nb, strict).cs) + 20 * (int64_t)nb + bundle_extra_bytes(n);
}
__host__ __device__ inline int64_t cky_split_count(int n) { return (int64_t)n * (n - 1) / 2; }
// Entry of span (i, i + w), w >= 2, in the split table: all spans of width 2,
// then of width 3, and so on.
__host__ __device__ inline int cky_split_index(int n, int w, int i) {
    return (w - 2) * (n + 1) - ((w - 1) * w / 2 - 1) + i;
}
__host__ __device__ inline int64_t cky_chart_bytes(int n, int split_bytes) {
    const int64_t ld = cky_ld(n);
    return ld * ld * 8 + cky_split_bytes_of(n, split_bytes);
}

// Shape of a width step with K split points per span: G lanes per span (a
// power of two <= 64), C splits per lane (lane l takes splits l, l+G, ...),
// of which the first MF are in range for every lane (MF G <= K) and the rest
// are masked.  Every distinct shape is its own unrolled body, and entering
// one that a sweep has not run yet refills the instruction cache, so sweeps
// use few shapes; C grows in steps of a quarter or a third, which keeps the
// masked share of a step under a quarter.
struct StepShape {
    int G, C, MF;
};
__host__ __device__ constexpr StepShape step_shape_k(int K) {
    if (K <= 1) return StepShape{1, 1, 0};
    if (K <= 2) return StepShape{1, 2, 1};
    if (K <= 4) return StepShape{1, 4, 2};
    if (K <= 8) return StepShape{1, 8, 4};
    if (K <= 16) return StepShape{2, 8, 4};
    if (K <= 32) return StepShape{4, 8, 4};
    // 33..128 splits: 4 lanes per span, so that a lone sentence of up to 127
    // words takes one pass of a 512-thread workgroup per joint step
    if (K <= 48) return StepShape{4, 12, 8};
    if (K <= 64) return StepShape{4, 16, 12};
    if (K <= 96) return StepShape{4, 24, 16};
    if (K <= 128) return StepShape{4, 32, 24};
    int g = 8;
    while (16 * g < K && g < 64) g <<= 1;
    return 12 * g >= K ? StepShape{g, 12, 8} : StepShape{g, 16, 12};
}

// The step shapes of steps of up to 128 splits as runs of K in [LO, HI]:
// R(LO, HI, G, C, MF).  The sweeps call these runs one after the other,
// with no shape dispatch (sentences of up to 129 words); steps of more
// splits go through step_shape_k.
#define CRF_FIXED_RUNS_LOW(R) R(1, 1, 1, 1, 0) R(2, 2, 1, 2, 1) R(3, 4, 1, 4, 2) R(5, 8, 1, 8, 4)
#define CRF_FIXED_RUNS_MID(R) R(9, 16, 2, 8, 4) R(17, 32, 4, 8, 4)
#define CRF_FIXED_RUNS_HIGH(R) \
    R(33, 48, 4, 12, 8) R(49, 64, 4, 16, 12) R(65, 96, 4, 24, 16) R(97, 128, 4, 32, 24)
#define CRF_FIXED_RUNS(R) CRF_FIXED_RUNS_LOW(R) CRF_FIXED_RUNS_MID(R) CRF_FIXED_RUNS_HIGH(R)
constexpr int kFixedRunsMaxK = 128;
constexpr bool fixed_runs_match_step_shapes() {
    int next = 1;
#define CRF_CHECK_RUN(LO, HI, GG, CC, MM)                                                 \
    if (LO != next) return false;                                                       \
    for (int K = LO; K <= HI; ++K) {                                                    \
        const StepShape s = step_shape_k(K);                                            \
        if (s.G != GG || s.C != CC || s.MF != MM) return false;                         \
    }                                                                                   \
    next = HI + 1;
    CRF_FIXED_RUNS(CRF_CHECK_RUN)
#undef CRF_CHECK_RUN
    return next == kFixedRunsMaxK + 1;
}
static_assert(fixed_runs_match_step_shapes(), "CRF_FIXED_RUNS must list step_shape_k's runs");

// CKY's step shapes.  A CKY step has the n-w+1 inside spans only (the joint
// sweep's shapes are sized for its n+1 inside and outside spans), so from 33
// splits it gives each span twice or four times the lanes with half or a
// quarter of the splits each: shorter chains of float64 loads, sums and
// argmax per lane, one or two more group-reduction levels.  C G, and so the
// reach of the masked reads (C - MF) G, equal step_shape_k's at every K, so
// the CKY chart padding is the same.  Measured on the 5,000-sentence mixed
// batch: CKY decode 84 -> 76 us, identical trees; 16 lanes from 49 splits or
// 32 from 65 were slower.
__host__ __device__ constexpr StepShape step_shape_cky(int K) {
    if (K <= 32 || K > kFixedRunsMaxK) return step_shape_k(K);
    if (K <= 48) return StepShape{8, 6, 4};
    if (K <= 64) return StepShape{8, 8, 6};
    if (K <= 96) return StepShape{16, 6, 4};
    return StepShape{16, 8, 6};
}
#define CRF_CKY_FIXED_RUNS(R) \
    R(1, 1, 1, 1, 0) R(2, 2, 1, 2, 1) R(3, 4, 1, 4, 2) R(5, 8, 1, 8, 4) R(9, 16, 2, 8, 4) R(17, 32, 4, 8, 4) \
    R(33, 48, 8, 6, 4) R(49, 64, 8, 8, 6) R(65, 96, 16, 6, 4) R(97, 128, 16, 8, 6)
constexpr bool cky_runs_match_step_shapes() {
    int next = 1;
#define CRF_CHECK_CKY_RUN(LO, HI, GG, CC, MM)                                                \
    if (LO != next) return false;                                                          \
    for (int K = LO; K <= HI; ++K) {                                                       \
        const StepShape s = step_shape_cky(K), r = step_shape_k(K);                        \
        if (s.G != GG || s.C != CC || s.MF != MM) return false;                            \
        if (s.MF * s.G > K || s.C * s.G < K || s.C * s.G != r.C * r.G) return false;       \
        if ((s.C - s.MF) * s.G != (r.C - r.MF) * r.G) return false;                        \
    }                                                                                      \
    next = HI + 1;
    CRF_CKY_FIXED_RUNS(CRF_CHECK_CKY_RUN)
#undef CRF_CHECK_CKY_RUN
    return next == kFixedRunsMaxK + 1;
}
static_assert(cky_runs_match_step_shapes(),
              "CRF_CKY_FIXED_RUNS must list step_shape_cky's runs, with step_shape_k's reach");

// The joint sweep's shapes for bundles whose steps take several passes of
// the workgroup: a bundle of nb sentences of n words has nb (n + 1) spans in
// a joint step, 4 lanes each at step_shape_k's shapes from 17 splits, and
// short_bundle says when that exceeds the workgroup.  From 9 to 32 splits
// these shapes give each span half the lanes with twice the splits each (C G,
// and so the reach of the masked reads (C - MF) G, kept): fewer passes and one
// group-reduction level less per step.  A bundle whose steps fit one pass (a
// lone long sentence) keeps step_shape_k's shapes: its steps are latency-bound,
// and shorter per-lane chains serve it better.  Outside 9..32 both lists run
// the same code (a CU running both kinds of bundles fetches one copy of it).
// The labelled bundle kernel keeps step_shape_k's shapes throughout: beside
// its bundles' own label work the multi-pass shapes measured 1% slower.
__host__ __device__ constexpr bool short_bundle(int nb, int n, int threads) { return nb * (n + 1) * 4 > threads; }
__host__ __device__ constexpr StepShape step_shape_short(int K) {
    if (K <= 8 || K > 32) return step_shape_k(K);
    return K <= 16 ? StepShape{1, 16, 8} : StepShape{2, 16, 8};
}
#define CRF_SHORT_RUNS_MID(R) R(9, 16, 1, 16, 8) R(17, 32, 2, 16, 8)
#define CRF_SHORT_FIXED_RUNS(R) CRF_FIXED_RUNS_LOW(R) CRF_SHORT_RUNS_MID(R) CRF_FIXED_RUNS_HIGH(R)
constexpr bool short_runs_match_step_shapes() {
    int next = 1;
#define CRF_CHECK_SHORT_RUN(LO, HI, GG, CC, MM)                                              \
    if (LO != next) return false;                                                          \
    for (int K = LO; K <= HI; ++K) {                                                       \
        const StepShape s = step_shape_short(K), r = step_shape_k(K);                      \
        if (s.G != GG || s.C != CC || s.MF != MM) return false;                            \
        if (s.MF * s.G > K || s.C * s.G < K || s.C * s.G != r.C * r.G) return false;       \
        if ((s.C - s.MF) * s.G != (r.C - r.MF) * r.G) return false;                        \
    }                                                                                      \
    next = HI + 1;
    CRF_SHORT_FIXED_RUNS(CRF_CHECK_SHORT_RUN)
#undef CRF_CHECK_SHORT_RUN
    return next == kFixedRunsMaxK + 1;
}
static_assert(short_runs_match_step_shapes(),
              "CRF_SHORT_FIXED_RUNS must list step_shape_short's runs, with step_shape_k's reach");

// The first K' > K whose step shape differs from K's (the sweeps run the
// steps of one shape as one loop; a closed form, since a scan over the
// steps costs a chain of scalar instructions per step).
__host__ __device__ inline int shape_run_end(int K) {
    if (K <= 1) return 2;
    if (K <= 2) return 3;
    if (K <= 4) return 5;
    if (K <= 8) return 9;
    if (K <= 16) return 17;
    if (K <= 32) return 33;
    if (K <= 48) return 49;
    if (K <= 64) return 65;
    if (K <= 96) return 97;
    if (K <= 128) return 129;
    // workspace sentences: for g lanes per span (16 from 129 splits, doubling
    // past 16 g, at most 64), 12 splits per lane up to 12 g, then 16; the
    // widest shape never ends
    int g = 16;
    while (16 * g < K && g < 64) g <<= 1;
    if (K <= 12 * g) return 12 * g + 1;
    if (g < 64) return 16 * g + 1;
    return 1 << 30;
}

// Cells past its span's last split that a masked split read may reach, at
// the widest step of a sentence of n words: (C - MF) G.
__host__ __device__ inline int masked_reach(int n) {
    const StepShape sh = step_shape_k(n - 1 > 0 ? n - 1 : 0);
    return (sh.C - sh.MF) * sh.G;
}

// Biaffine scorer tiles: rows (left fence posts) and columns (right fence
// posts) per tile, representation dimensions per chunk of the inner product,
// and the largest d whose staged rows fit in LDS beside a chunk of W.
constexpr int kBiaRows = 64, kBiaCols = 64, kBiaChunk = 32;
constexpr int kBiaMaxD = 508;
static_assert(kBiaRows == kBiaCols, "packed tiles use their fence posts as both rows and columns");

// Threads per workgroup of the label passes, and floats of a row's label
// block per workgroup.
constexpr int kLabelChunk = 256;
// Labelled bundles of sentences of up to this many words read their label
// scores and write their per-label marginals themselves (in the inside
// kernel's prologue and epilogue); longer sentences, whose bundles set the
// launch's critical path, leave both to the chip-wide label passes.
constexpr int kLabInBundleMaxN = 48;
constexpr int kLabelRowChunk = 1024;

// Longest sentence whose CKY chart could sit in one CU's LDS (160 KiB):
// 8 (n+1)^2 <= 163840 (with row padding, its split table and tables the
// plan finds somewhat less).  The plan sends longer ones to the workspace
// kernels.
constexpr int kMaxLenInLds = 142;

// A bundle: `count` sentences of identical length `n`, processed together by
// one workgroup; their ids are order[first .. first+count).
struct Bundle {
    int32_t first;
    int32_t count;
    int32_t n;
    // CKY: where the bundle's split tables live -- -1: in LDS after each
    // chart; else at workspace byte 256 * split_ws, count tables of
    // cky_split_count(n) bytes back to back.  Unused for inside bundles.
    int32_t split_ws;
};

// What a bundle's workgroup reads first: one record of rec_stride ints --
// n, count, split_ws (CKY; -1 for inside), kind (kKindInside, kKindCky or
// kKindMbr), then its chart layout (inside_layout or cky_layout, as the plan
// chose it: e, ld, cs) and div_magic(count), then a second layout (the CKY
// chart of an MBR bundle, whose first layout is its inside chart), then the
// count sentence ids -- so that its sentence ids arrive with its shape, one
// memory round trip before its scores, and the workgroup computes none of it.
constexpr int kRecHeader = 12;
enum RecField {
    kRecN = 0, kRecCount, kRecSplitWs, kRecKind, kRecE, kRecLd, kRecCs, kRecMagic, kRecE2, kRecLd2, kRecCs2,
    kRecLab   // labelled inside bundles: 1 when the bundle reads and writes its own label scores
};
enum RecKind { kKindCky = 0, kKindInside = 1, kKindMbr = 2 };
// g / S by multiply-high: 2^32 / S + 1, exact for g < 2^18, 2 <= S <= 1024;
// 0 for S = 1 (the caller takes g itself).
__host__ __device__ inline uint32_t div_magic(int S) { return S > 1 ? 0xFFFFFFFFu / (uint32_t)S + 1u : 0u; }

// Which sentences run in LDS (in bundles) and which on the workspace kernel,
// for one kind of chart.  Bundles and spilled sentences are ordered most
// expensive first.
struct Schedule {
    const int32_t *recs;         // [n_bundles] records, rec_stride ints each
    const int32_t *order_spill;  // [n_spill] sentence ids
    const int64_t *ws_off;       // [n_spill] byte offset of each chart in the workspace
    int32_t n_bundles, n_spill;
    int32_t lds_bytes;           // dynamic LDS per workgroup (bundle budget)
    int32_t threads;             // workgroup size of the LDS kernels
};

// Device-side view of a plan, passed by value to every kernel.
//   mix: the records of the fused inside + CKY kernel, sorted by predicted
//   duration (both kinds merged); its fused_grid workgroups take them in
//   this order (see parse_kernel).
struct KernelPlan {
    const int32_t *len;          // [B] sentence lengths
    char *ws;                    // workspace base
    Schedule inside, cky;
    const int32_t *mix;          // [n_mix] records, or NULL when the fused kernel is not used
    int32_t n_mix;
    int32_t fused_grid;          // workgroups of the fused kernel (<= n_mix)
    // MBR decoding: records of bundles that run inside + marginals and then
    // CKY over the marginals, or NULL (then the two run as separate launches)
    const int32_t *mbr;
    int32_t n_mbr, mbr_grid, mbr_lds;
    int32_t *counter;            // the fused kernels' bundle claims; zero between launches
    // labelled plans: chunks of kLabelRowChunk floats of the label blocks of
    // the rows of the sentences whose label passes run chip-wide, (sentence,
    // row, first float, 0), and the workspace offsets of their label
    // log-sum-exps and marginals ([B][N1][N1] float32 each)
    const int32_t *lab_rows;
    int32_t n_lab_rows;
    // biaffine scorer tiles: kBiaRows row ids then kBiaCols column ids each
    // (b N1 + fence post, or -1)
    const int32_t *bia_tiles;
    int32_t n_bia_tiles;
    int64_t lab_sp_off, lab_mu_off;
    // set per labelled inside launch: the label scores [B][N1][N1][L], the
    // per-label marginals out (NULL for the forward pass) and L, for the
    // bundles that do their own label I/O (kRecLab)
    const float *lab_s4;
    float *lab_out;
    int32_t lab_L;
    int32_t rec_stride;          // ints per record: kRecHeader + the largest bundle
    int32_t B, n1, L;
    // Workspace launches by teams: the team area (kTeamAreaBytes, zeroed
    // before each team launch), how many workspace workgroups the device
    // holds at once, and the team size of the launch at hand (set by the
    // launcher; 1: a workgroup per sentence pass, no team area used).
    int32_t *team_area;
    int32_t team_cap, team_k;
};

// Teams for workspace sentences: up to kTeamMaxK workgroups of one XCD run a
// sentence's pass together.  The team area holds kTeamHeaderWords words
// (arrivals per XCD at [0, 16), all arrivals at 16, the abort flag at 17)
// and kTeamLineWords words per team (its barrier's arrivals at 0, at 1 the
// last of its jobs, plus one, whose linear-domain sweep left float32's range).
constexpr int kTeamMaxK = 16;
// Smallest team a launch forms.  A workspace step is bound by its memory
// round trips (operand loads, store acknowledgements, the team's arrival),
// not by one CU's issue, and a team reads the chart past its L1: teams pay
// where a few long sentences leave most of the chip idle (fused parse of a
// lone 512-word sentence 7.0 -> 2.1 ms, of a 1023-word one 60 -> 7.6 ms, at
// k = 16), not on batches that fill it (64 sentences of 256 words: 1.7 ms
// alone, 2.7 ms in teams of two).
constexpr int kTeamMinK = 8;
constexpr int kTeamHeaderWords = 64, kTeamLineWords = 64;
constexpr int kTeamMaxTeams = 1024;
constexpr int64_t kTeamAreaBytes = 4 * (int64_t)(kTeamHeaderWords + kTeamLineWords * kTeamMaxTeams);
// Workgroups of kThreadsMax threads of the workspace kernels one CU holds at
// once (the least over those kernels; 0 on error).
int spill_blocks_per_cu();

// Shape of a workspace launch of `jobs` sentence passes on a device that
// holds `cap` such workgroups at once.  With a team area: m = ceil(jobs / 8)
// teams per XCD (workgroups go to the eight XCDs in turn), k a power of two,
// as large as cap allows up to kTeamMaxK, grid 8 m k <= cap (a team barrier
// needs every member resident).  Without one, or with k below kTeamMinK:
// k = 1, a workgroup per job.
struct TeamShape {
    int k, grid;
};
inline TeamShape team_shape(int jobs, int64_t cap, bool has_area) {
    const int m = (jobs + 7) / 8;
    int k = 1;
    if (has_area && jobs >= 1 && 8 * m <= kTeamMaxTeams)
        while (2 * k <= kTeamMaxK && (int64_t)8 * m * 2 * k <= cap) k *= 2;
    if (k < kTeamMinK) return TeamShape{1, jobs};
    return TeamShape{k, 8 * m * k};
}

// The no-allocation entry point's scratch: a file-scope device array of
// kScratchBytes per GPU (the first kScratchCounterBytes hold the fused
// launch's claim counter, the rest stands in for the plan's workspace).
constexpr int64_t kScratchBytes = (int64_t)8 << 20;
constexpr int64_t kScratchCounterBytes = 256;
constexpr int kMaxDevices = 64;
// Device address of the current device's scratch array (resolved once per
// device, with that device current, and kept).
hipError_t scratch_address(int device, char **out);
// crf_inside_fwd_bwd_cky on the scratch array instead of the plan's
// workspace and counter: clears the counter with a kernel, then launches as
// launch_parse does.  The caller has checked the plan's workspace fits.
hipError_t launch_parse_scratch(const KernelPlan &p, char *scratch, const float *scores, const float *grad,
                                float *logZ, float *marg, int32_t *spans, float *best, hipStream_t stream);

hipError_t launch_inside(const KernelPlan &p, const float *scores, const float *grad,
                         float *logZ, float *marg, hipStream_t stream);
// CKY; labels != NULL: labelled scores, max over labels per span, and the
// tree's spans' best labels (one-stage labelled decoding)
hipError_t launch_cky(const KernelPlan &p, const float *scores, int32_t *spans, float *best,
                      hipStream_t stream, int32_t *labels = nullptr);
// MBR decoding: inside + marginals, then CKY over the marginals
hipError_t launch_mbr(const KernelPlan &p, const float *scores, float *logZ, float *marg, int32_t *spans,
                      float *best, hipStream_t stream);
// Gold-tree loss and its gradient (unlabelled)
hipError_t launch_loss(const KernelPlan &p, const float *scores, const int32_t *gold, const float *grad,
                       float *loss, float *grad_scores, hipStream_t stream);
// Labelling stage: labels of given spans from [B][N1][N1][L] label scores
hipError_t launch_label_spans(const KernelPlan &p, const float *label_scores, int L, const int32_t *spans,
                              int32_t *labels, hipStream_t stream);
hipError_t launch_parse(const KernelPlan &p, const float *scores, const float *grad, float *logZ,
                        float *marg, int32_t *spans, float *best, hipStream_t stream);
hipError_t set_kernel_attributes(int max_lds_bytes);
// The biaffine scorer (crf_biaffine.hip): dynamic LDS per workgroup for d,
// and the launch over the plan's tiles and L labels.
int64_t biaffine_lds_bytes(int d);
hipError_t set_biaffine_attributes();   // once per plan: the LDS of the largest d
hipError_t launch_biaffine(const KernelPlan &p, const uint16_t *rl, const uint16_t *rr, const uint16_t *w, int d,
                           int ldw, int L, float *scores, hipStream_t stream);

}  // namespace crf
