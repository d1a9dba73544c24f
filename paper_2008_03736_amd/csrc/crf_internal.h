// crf_internal.h -- what the host plan code and the gfx950 kernels share.
//
// Not part of the public ABI (that is include/crf_inside.h).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace crf {

// Threads per workgroup of every kernel: four 64-wide wavefronts.
constexpr int kThreads = 256;

// The LDS kernels give a span at most 16 lanes and cache at most 12 split
// points per lane, so they take sentences of up to 16*12+1 words; longer
// ones always use the workspace kernels (which allow 64 lanes x 16).
constexpr int kMaxLenLds = 16 * 12 + 1;

// Row stride (in elements) of a sentence's square chart.  One place so the
// host's LDS sizing and the kernels' indexing cannot disagree.
__host__ __device__ inline int chart_ld(int n) { return n + 1; }

// Bytes of chart per sentence.
//   inside: two float32 squares -- alpha (upper triangle + mirrored lower
//           triangle) and the adjoint accumulators (scores during the
//           forward sweep);
//   cky:    one float64 square (beta, upper + mirror) + a uint16 square of
//           back-pointers.
__host__ __device__ inline int64_t inside_chart_bytes(int n) {
    const int64_t ld = chart_ld(n);
    return 2 * ld * ld * 4;
}
__host__ __device__ inline int64_t cky_chart_bytes(int n) {
    const int64_t ld = chart_ld(n);
    return ld * ld * 8 + ((ld * ld * 2 + 7) / 8) * 8;
}

// Which sentences run on the LDS kernel and which on the workspace kernel,
// for one kind of chart.  Both lists are ordered most expensive first.
struct Schedule {
    const int32_t *order_lds;    // [n_lds] sentence ids
    const int32_t *order_spill;  // [n_spill] sentence ids
    const int64_t *ws_off;       // [n_spill] byte offset of each chart in the workspace
    int32_t n_lds, n_spill;
    int32_t lds_bytes;           // dynamic LDS per workgroup of the LDS kernel
};

// Device-side view of a plan, passed by value to every kernel.
struct KernelPlan {
    const int32_t *len;          // [B] sentence lengths
    char *ws;                    // workspace base
    Schedule inside, cky;
    int32_t B, n1, L;
};

hipError_t launch_inside(const KernelPlan &p, const float *scores, const float *grad,
                         float *logZ, float *marg, hipStream_t stream);
hipError_t launch_cky(const KernelPlan &p, const float *scores, int32_t *spans, float *best,
                      hipStream_t stream);
hipError_t set_kernel_attributes(int max_lds_bytes);

}  // namespace crf
