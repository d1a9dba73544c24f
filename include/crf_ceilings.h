/*
 * crf_ceilings.h -- microbenchmarks of the gfx950 ceilings behind the CRF
 * kernels' roofline (library libcrfceilings.so; measurement only, not part
 * of the CRF path).
 */
#ifndef CRF_CEILINGS_H
#define CRF_CEILINGS_H

#ifdef __cplusplus
extern "C" {
#endif

/*
 * crf_ceiling_run -- enqueue one microbenchmark kernel on `stream`.
 *   kind     0 fp32 add, 1 fp32 FMA, 2 exp2, 3 log2, 4 fp64 add,
 *            5 exp2 beside independent fp32 adds, 6 LDS reads,
 *            7 LDS store / barrier / load round trip.
 *   blocks   workgroups (>= 1); threads: a power of two in [64, 1024].
 *   iters    loop iterations (>= 1).  Per thread and iteration: kinds 0, 1
 *            and 4 issue 16 operations, kinds 2 and 3 issue 8, kind 5 issues
 *            8 exp2 and 24 adds, kind 6 issues 8 LDS reads, kind 7 one round
 *            trip (two barriers).
 *   out      device float32[blocks * threads], written once per thread (keeps
 *            the work live).
 * Returns 0 (hipSuccess) or a hipError_t code; bad arguments give
 * hipErrorInvalidValue before any launch.
 */
int crf_ceiling_run(int kind, int blocks, int threads, int iters, float *out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* CRF_CEILINGS_H */
