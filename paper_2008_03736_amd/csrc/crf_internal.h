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

// LDS a bundle needs besides its charts: a uint32 table of division magics
// for span counts 0..n+1.  (Masked tail loads stay inside a sentence's inside
// chart; those of the last CKY chart reach up to masked_reach(n) float64 past
// it, into the tables that follow it, which the plan pads to that size.)
__host__ __device__ inline int64_t bundle_extra_bytes(int n) { return 4 * (int64_t)(n + 2); }

// LDS a workgroup holds besides its bundle (the fused kernel's claim slot)
// and slack.  Bundle budgets leave it free.
constexpr int kReservedLds = 256;

// Row stride (in elements) of a sentence's square charts, at least n + 1.
// Spans of one width sit ld + 1 elements apart along the diagonal (the
// inside and CKY split operands) and ld apart down a column (the outside
// operands); LDS has 32 four-byte banks, so a stride with a factor 2^k
// makes 2^k lanes collide on a bank.  The inside chart takes ld = 1 or 2
// (mod 4) -- one stride odd, the other twice odd, at worst 2-way; the
// float64 CKY chart takes ld even, which makes ld + 1 odd and its
// 8-byte diagonal accesses conflict-free.  (Sentences of 98 and 99 words
// keep ld = n + 1 for the inside: padded, their two float32 squares would
// no longer fit in half a CU, and one bundle that needs a whole CU moves
// every bundle of the launch to one workgroup per CU.)
__host__ __device__ inline int inside_ld(int n) {
    int ld = n + 1;
    while ((ld & 3) == 0 || (ld & 3) == 3) ++ld;
    return (ld > 100 && n + 1 <= 100) ? n + 1 : ld;
}
__host__ __device__ inline int cky_ld(int n) { return (n + 1) + ((n + 1) & 1); }

// Bytes of chart per sentence.
//   inside: two float32 squares -- alpha (upper triangle + mirrored lower
//           triangle) and the outside values (upper + mirrored; before the
//           outside sweep reaches a span its mirrored cell holds the span's
//           score, and cells no sweep reads park the forced-span scores);
//   cky:    one float64 square (beta, upper + mirror), followed by the
//           split table (cky_split_index) when split_bytes > 0: the best
//           split k of every span (i, j) of two or more words, stored as
//           k - i - 1 in split_bytes bytes (1 for n <= kMaxLenInLds, 2 in
//           the workspace).  A bundle whose tables do not fit in LDS beside
//           its charts keeps them in the workspace (Bundle::split_ws).
__host__ __device__ inline int64_t inside_chart_bytes(int n) {
    const int64_t ld = inside_ld(n);
    return 2 * ld * ld * 4;
}
__host__ __device__ inline int64_t cky_split_count(int n) { return (int64_t)n * (n - 1) / 2; }
// Entry of span (i, i + w), w >= 2, in the split table: all spans of width 2,
// then of width 3, and so on.
__host__ __device__ inline int cky_split_index(int n, int w, int i) {
    return (w - 2) * (n + 1) - ((w - 1) * w / 2 - 1) + i;
}
__host__ __device__ inline int64_t cky_chart_bytes(int n, int split_bytes) {
    const int64_t ld = cky_ld(n);
    return ld * ld * 8 + (cky_split_count(n) * split_bytes + 7) / 8 * 8;
}
// The CKY tree walk follows the split table.  Bundles of fewer than
// kDfsMinBundle sentences walk breadth first, one wavefront per sentence,
// with a list of at most n - 1 internal nodes per wavefront; larger bundles
// walk depth first, one lane per sentence, with a stack of n ints each.
constexpr int kDfsMinBundle = 16;
__host__ __device__ inline int64_t cky_walk_bytes(int n, int64_t count, int waves) {
    return count < kDfsMinBundle ? 4 * (int64_t)(count < waves ? count : waves) * n : 4 * count * n;
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
__host__ __device__ inline StepShape step_shape_k(int K) {
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

// Cells past its span's last split that a masked split read may reach, at
// the widest step of a sentence of n words: (C - MF) G.
__host__ __device__ inline int masked_reach(int n) {
    const StepShape sh = step_shape_k(n - 1 > 0 ? n - 1 : 0);
    return (sh.C - sh.MF) * sh.G;
}

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
// n, count, split_ws (CKY; -1 for inside), kind (1 inside, 0 CKY), then the
// count sentence ids -- so that its sentence ids arrive with its shape, one
// memory round trip before its scores.
constexpr int kRecHeader = 4;

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
    int32_t *counter;            // the fused kernel's bundle claims; zero between launches
    int32_t rec_stride;          // ints per record: kRecHeader + the largest bundle
    int32_t B, n1, L;
};

hipError_t launch_inside(const KernelPlan &p, const float *scores, const float *grad,
                         float *logZ, float *marg, hipStream_t stream);
hipError_t launch_cky(const KernelPlan &p, const float *scores, int32_t *spans, float *best,
                      hipStream_t stream);
hipError_t launch_parse(const KernelPlan &p, const float *scores, const float *grad, float *logZ,
                        float *marg, int32_t *spans, float *best, hipStream_t stream);
hipError_t set_kernel_attributes(int max_lds_bytes);

}  // namespace crf
