// crf_ceilings.hip -- microbenchmarks of the gfx950 ceilings that the CRF
// kernels' roofline rests on (measurement infrastructure, not part of the
// CRF path).  Each kernel runs `iters` iterations of eight independent
// dependency chains per thread, so issue rate, not latency, bounds it (apart
// from the barrier kernel, which measures a latency).
//
//   kind 0  fp32 add          16 v_add_f32 per iteration
//   kind 1  fp32 FMA          16 v_fma_f32
//   kind 2  exp2              8 v_exp_f32 (x <- exp2(-x), a source modifier)
//   kind 3  log2              8 v_log_f32 (x <- log2(|x|))
//   kind 4  fp64 add          16 v_add_f64
//   kind 5  exp2 + adds       8 v_exp_f32 and 24 independent v_add_f32: if the
//                             transcendental co-issued, this would take the
//                             time of the adds alone
//   kind 6  LDS reads         8 ds_read_b32 per iteration, conflict-free
//                             (consecutive lanes, consecutive words)
//   kind 7  barrier step      one LDS store, workgroup barrier, one LDS load
//                             of another wavefront's word: the round trip
//                             that separates two width steps of a sweep
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/crf_ceilings.h"

namespace {

__global__ __launch_bounds__(1024) void k_add(float *out, float a, int iters) {
    float x[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) x[c] = (float)threadIdx.x + c;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int c = 0; c < 8; ++c) x[c] += a;
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < 8; ++c) s += x[c];
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(1024) void k_fma(float *out, float a, int iters) {
    float x[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) x[c] = (float)threadIdx.x + c;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int c = 0; c < 8; ++c) x[c] = __builtin_fmaf(x[c], a, a);
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < 8; ++c) s += x[c];
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(1024) void k_exp(float *out, float a, int iters) {
    float x[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) x[c] = a * (float)(threadIdx.x + c);
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int c = 0; c < 8; ++c) x[c] = __builtin_amdgcn_exp2f(-x[c]);
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < 8; ++c) s += x[c];
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(1024) void k_log(float *out, float a, int iters) {
    float x[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) x[c] = a + (float)(threadIdx.x + c);
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int c = 0; c < 8; ++c) x[c] = __builtin_amdgcn_logf(__builtin_fabsf(x[c]));
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < 8; ++c) s += x[c];
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(1024) void k_add64(float *out, float a, int iters) {
    double x[8];
    const double ad = a;
#pragma unroll
    for (int c = 0; c < 8; ++c) x[c] = (double)threadIdx.x + c;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int c = 0; c < 8; ++c) x[c] += ad;
    }
    double s = 0.0;
#pragma unroll
    for (int c = 0; c < 8; ++c) s += x[c];
    out[blockIdx.x * blockDim.x + threadIdx.x] = (float)s;
}

__global__ __launch_bounds__(1024) void k_exp_add(float *out, float a, int iters) {
    float x[8], y[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        x[c] = a * (float)(threadIdx.x + c);
        y[c] = (float)c;
    }
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int c = 0; c < 8; ++c) x[c] = __builtin_amdgcn_exp2f(-x[c]);
#pragma unroll
        for (int r = 0; r < 3; ++r)
#pragma unroll
            for (int c = 0; c < 8; ++c) y[c] += a;
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < 8; ++c) s += x[c] + y[c];
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(1024) void k_lds(float *out, float a, int iters) {
    __shared__ float buf[8 * 1024];
    for (int t = threadIdx.x; t < 8 * 1024; t += blockDim.x) buf[t] = a * t;
    __syncthreads();
    const int nt = blockDim.x;
    float s[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) s[c] = 0.f;
    int base = threadIdx.x;
    for (int i = 0; i < iters; ++i) {
        float v[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) v[c] = buf[base + c * nt];
#pragma unroll
        for (int c = 0; c < 8; ++c) s[c] += v[c];
        // keeps the eight reads of an iteration in range: base stays below nt
        base = (base + 64) & (nt - 1);
    }
    float r = 0.f;
#pragma unroll
    for (int c = 0; c < 8; ++c) r += s[c];
    out[blockIdx.x * blockDim.x + threadIdx.x] = r;
}

__global__ __launch_bounds__(1024) void k_barrier(float *out, float a, int iters) {
    __shared__ float buf[1024];
    float x = a * threadIdx.x;
    const int peer = (threadIdx.x + 64) & (blockDim.x - 1);   // a word of another wavefront
    for (int i = 0; i < iters; ++i) {
        buf[threadIdx.x] = x;
        __syncthreads();
        x = buf[peer] + a;
        __syncthreads();
    }
    out[blockIdx.x * blockDim.x + threadIdx.x] = x;
}

}  // namespace

extern "C" int crf_ceiling_run(int kind, int blocks, int threads, int iters, float *out, void *stream) {
    if (kind < 0 || kind > 7 || blocks < 1 || threads < 64 || threads > 1024 || (threads & (threads - 1)) != 0 ||
        iters < 1 || out == nullptr)
        return (int)hipErrorInvalidValue;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    const dim3 g(blocks), b(threads);
    const float a = 0.999f;
    switch (kind) {
        case 0: hipLaunchKernelGGL(k_add, g, b, 0, s, out, a, iters); break;
        case 1: hipLaunchKernelGGL(k_fma, g, b, 0, s, out, a, iters); break;
        case 2: hipLaunchKernelGGL(k_exp, g, b, 0, s, out, 1e-3f, iters); break;
        case 3: hipLaunchKernelGGL(k_log, g, b, 0, s, out, 1.5f, iters); break;
        case 4: hipLaunchKernelGGL(k_add64, g, b, 0, s, out, a, iters); break;
        case 5: hipLaunchKernelGGL(k_exp_add, g, b, 0, s, out, 1e-3f, iters); break;
        case 6: hipLaunchKernelGGL(k_lds, g, b, 0, s, out, a, iters); break;
        default: hipLaunchKernelGGL(k_barrier, g, b, 0, s, out, a, iters); break;
    }
    return (int)hipGetLastError();
}
