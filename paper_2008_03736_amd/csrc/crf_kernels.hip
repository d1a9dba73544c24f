// crf_kernels.hip -- gfx950 kernels for the batched tree-CRF.
//
// Method (Zhang, Zhou & Li, IJCAI 2020):
//   inside   alpha(i,j) = s(i,j) + log sum_{i<k<j} exp(alpha(i,k) + alpha(k,j)),
//            log Z = alpha(0,n)                           (Sec. 3.1, Algorithm 1)
//   reverse  p((i,j)|x) = d log Z / d s(i,j)              (Sec. 3.2, Eq. partial-derivative)
//   CKY      the same recursion under max, 1-best tree    (Sec. 3.3, Eq. tree-argmax)
//   labels   s'(i,j) = log sum_l exp s(i,j,l) feeds the inside; per-label
//            marginals are p((i,j)|x) * softmax_l s(i,j,l) (Sec. 4.2, Eq. tree-label-score)
//
// Design (one workgroup of 256 threads per sentence, longest first):
//   * The sentence's chart stays on chip for the whole call: LDS when it fits
//     ("lds" kernels), else a plan-owned global workspace that stays mostly
//     in L2/MALL ("spill" kernels, same code on global pointers).
//   * Width w is one barrier-separated step.  Each span of the width is
//     handled by a group of G lanes (G a power of two picked per width), each
//     lane taking the split points k = i+1+l, i+1+l+G, ...; the split-point
//     log-sum-exp is a lane-local max / sum-exp followed by a DPP butterfly
//     across the group.
//   * alpha is stored twice, at [i][j] and mirrored at [j][i], so both the
//     row alpha(i,.) and the column alpha(.,j) a span needs are contiguous.
//   * The chart holds log2-scaled values (v_exp_f32 / v_log_f32 are base 2).
//   * Forced spans -- every tree holds the n width-1 spans and the root -- are
//     factored out of the chart: their scores are summed in float64 and added
//     to log Z, and their marginal is exactly the upstream gradient.  This
//     keeps chart magnitudes small (an exact rewrite: Z = exp(forced) * Z').
//   * The reverse pass walks widths downwards.  For span (i,j) with adjoint
//     mu, each split gets p_k = exp(x_k - m) / sum exp(x - m) (normalised
//     with the span's own max), and mu * p_k flows to the left child (i,k)
//     and right child (k,j).  In one width a child has exactly one parent of
//     each kind, so left- and right-child adjoints are kept in the upper and
//     lower triangles of a second square: every write has a single writer
//     and no atomics are needed.
//   * CKY runs a float64 chart with the association order
//     beta(i,j) = (max_k (beta(i,k) + beta(k,j))) + s(i,j): only IEEE adds
//     and exact max, so the tree is reproducible bit for bit; ties keep the
//     lowest split.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "crf_internal.h"

namespace crf {
namespace {

constexpr int NT = kThreads;
constexpr int NWAVES = NT / 64;
constexpr float LOG2E_F = 1.4426950408889634f;
constexpr double LN2_D = 0.69314718055994530942;

// Split points cached in registers per lane (LDS kernels / spill kernels).
constexpr int MAXC_LDS = 12;
constexpr int MAXC_SPILL = 16;

// ---------------------------------------------------------------------------
// Cross-lane helpers.  Groups are aligned runs of G lanes; the butterflies
// leave the group's result in every lane of the group.

template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
    return __builtin_bit_cast(float, dpp_i<CTRL>(__builtin_bit_cast(int, v)));
}
template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const int lo = dpp_i<CTRL>((int)(uint32_t)u);
    const int hi = dpp_i<CTRL>((int)(uint32_t)(u >> 32));
    return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}
// xor 16 inside each 32-lane half: ds_swizzle bit-mask mode (and 0x1f, xor 0x10).
__device__ __forceinline__ int swz16_i(int v) { return __builtin_amdgcn_ds_swizzle(v, 0x401F); }
// xor 32: cross-half permute.
__device__ __forceinline__ int x32_i(int v) {
    const int lane = (int)__lane_id();
    return __builtin_amdgcn_ds_bpermute((lane ^ 32) << 2, v);
}
__device__ __forceinline__ float swz16_f(float v) {
    return __builtin_bit_cast(float, swz16_i(__builtin_bit_cast(int, v)));
}
__device__ __forceinline__ float x32_f(float v) {
    return __builtin_bit_cast(float, x32_i(__builtin_bit_cast(int, v)));
}
__device__ __forceinline__ double swz16_d(double v) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const int lo = swz16_i((int)(uint32_t)u), hi = swz16_i((int)(uint32_t)(u >> 32));
    return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}
__device__ __forceinline__ double x32_d(double v) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const int lo = x32_i((int)(uint32_t)u), hi = x32_i((int)(uint32_t)(u >> 32));
    return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// DPP controls: quad_perm [1,0,3,2] (xor 1), quad_perm [2,3,0,1] (xor 2),
// row_half_mirror (pairs the two quads of each 8 lanes), row_mirror (pairs
// the two halves of each 16-lane row).
constexpr int DPP_XOR1 = 0xB1, DPP_XOR2 = 0x4E, DPP_HMIRROR = 0x141, DPP_MIRROR = 0x140;

template <int G>
__device__ __forceinline__ float grp_max(float v) {
    if constexpr (G >= 2) v = fmaxf(v, dpp_f<DPP_XOR1>(v));
    if constexpr (G >= 4) v = fmaxf(v, dpp_f<DPP_XOR2>(v));
    if constexpr (G >= 8) v = fmaxf(v, dpp_f<DPP_HMIRROR>(v));
    if constexpr (G >= 16) v = fmaxf(v, dpp_f<DPP_MIRROR>(v));
    if constexpr (G >= 32) v = fmaxf(v, swz16_f(v));
    if constexpr (G >= 64) v = fmaxf(v, x32_f(v));
    return v;
}
template <int G>
__device__ __forceinline__ float grp_sum(float v) {
    if constexpr (G >= 2) v += dpp_f<DPP_XOR1>(v);
    if constexpr (G >= 4) v += dpp_f<DPP_XOR2>(v);
    if constexpr (G >= 8) v += dpp_f<DPP_HMIRROR>(v);
    if constexpr (G >= 16) v += dpp_f<DPP_MIRROR>(v);
    if constexpr (G >= 32) v += swz16_f(v);
    if constexpr (G >= 64) v += x32_f(v);
    return v;
}
template <int G>
__device__ __forceinline__ double grp_max_d(double v) {
    if constexpr (G >= 2) v = fmax(v, dpp_d<DPP_XOR1>(v));
    if constexpr (G >= 4) v = fmax(v, dpp_d<DPP_XOR2>(v));
    if constexpr (G >= 8) v = fmax(v, dpp_d<DPP_HMIRROR>(v));
    if constexpr (G >= 16) v = fmax(v, dpp_d<DPP_MIRROR>(v));
    if constexpr (G >= 32) v = fmax(v, swz16_d(v));
    if constexpr (G >= 64) v = fmax(v, x32_d(v));
    return v;
}
template <int G>
__device__ __forceinline__ int grp_min_i(int v) {
    if constexpr (G >= 2) v = min(v, dpp_i<DPP_XOR1>(v));
    if constexpr (G >= 4) v = min(v, dpp_i<DPP_XOR2>(v));
    if constexpr (G >= 8) v = min(v, dpp_i<DPP_HMIRROR>(v));
    if constexpr (G >= 16) v = min(v, dpp_i<DPP_MIRROR>(v));
    if constexpr (G >= 32) v = min(v, swz16_i(v));
    if constexpr (G >= 64) v = min(v, x32_i(v));
    return v;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// Lanes per span for one width: K = w-1 split points, S = n-w+1 spans.
// Minimises (rounds of spans) x (serial splits per lane + butterfly depth).
template <int GMAX, int MAXC>
__device__ __forceinline__ int pick_group(int K, int S) {
    int best = GMAX, best_cost = 0x7fffffff;
#pragma unroll
    for (int g = 1; g <= GMAX; g <<= 1) {
        const int cnt = (K + g - 1) / g;
        if (cnt > MAXC) continue;
        const int groups = NT / g;
        const int rounds = (S + groups - 1) / groups;
        const int depth = 31 - __builtin_clz(g);
        const int cost = rounds * (cnt * 4 + depth * 6 + 10);
        if (cost < best_cost) { best_cost = cost; best = g; }
    }
    return best;
}

// ---------------------------------------------------------------------------
// Inside sweep, one width.  al: chart (alpha upper [i][j], mirror [j][i]);
// before width w runs, al[i][j] of every width-w span holds its log2-scaled
// score (0 for the root, whose score is factored out).

template <int G, int MAXC, typename T>
__device__ __forceinline__ void inside_width(T *al, int ld, int n, int w, int tid) {
    constexpr int GROUPS = NT / G;
    const int K = w - 1, S = n - w + 1;
    const int cnt = (K + G - 1) / G;
    const int g = tid / G, l = tid % G;
    for (int s0 = 0; s0 < S; s0 += GROUPS) {
        const int sp = s0 + g;
        const bool act = sp < S;
        const int i = act ? sp : S - 1;
        const int j = i + w;
        const T *rp = al + (size_t)i * ld + (i + 1 + l);   // alpha(i, k)
        const T *cp = al + (size_t)j * ld + (i + 1 + l);   // alpha(k, j), mirrored
        const float sij = al[(size_t)i * ld + j];
        float x[MAXC];
        float m = -INFINITY;
#pragma unroll
        for (int c = 0; c < MAXC; ++c) {
            x[c] = -INFINITY;
            if (c < cnt && l + c * G < K) x[c] = rp[c * G] + cp[c * G];
            m = fmaxf(m, x[c]);
        }
        m = grp_max<G>(m);
        float sum = 0.f;
#pragma unroll
        for (int c = 0; c < MAXC; ++c)
            if (c < cnt) sum += fast_exp2(x[c] - m);
        sum = grp_sum<G>(sum);
        if (act && l == 0) {
            const float v = m + fast_log2(sum) + sij;
            al[(size_t)i * ld + j] = v;
            al[(size_t)j * ld + i] = v;
        }
    }
}

// Reverse sweep, one width.  ad: adjoints -- upper [i][k] accumulates what
// (i,k) receives as a left child, lower [j][k] what (k,j) receives as a
// right child.  gval is the upstream gradient (the root's adjoint).
template <int G, int MAXC, typename T>
__device__ __forceinline__ void reverse_width(const T *al, T *ad, int ld, int n, int w, int tid,
                                              float gval) {
    constexpr int GROUPS = NT / G;
    const int K = w - 1, S = n - w + 1;
    const int cnt = (K + G - 1) / G;
    const int g = tid / G, l = tid % G;
    for (int s0 = 0; s0 < S; s0 += GROUPS) {
        const int sp = s0 + g;
        const bool act = sp < S;
        const int i = act ? sp : S - 1;
        const int j = i + w;
        const T *rp = al + (size_t)i * ld + (i + 1 + l);
        const T *cp = al + (size_t)j * ld + (i + 1 + l);
        const float mu = (w == n) ? gval : ad[(size_t)i * ld + j] + ad[(size_t)j * ld + i];
        float x[MAXC];
        float m = -INFINITY;
#pragma unroll
        for (int c = 0; c < MAXC; ++c) {
            x[c] = -INFINITY;
            if (c < cnt && l + c * G < K) x[c] = rp[c * G] + cp[c * G];
            m = fmaxf(m, x[c]);
        }
        m = grp_max<G>(m);
        float sum = 0.f;
#pragma unroll
        for (int c = 0; c < MAXC; ++c) {
            if (c < cnt) {
                x[c] = fast_exp2(x[c] - m);
                sum += x[c];
            }
        }
        sum = grp_sum<G>(sum);
        const float coef = mu / sum;
        if (act) {
            T *lp = ad + (size_t)i * ld + (i + 1 + l);   // left-child slots (i, k)
            T *rq = ad + (size_t)j * ld + (i + 1 + l);   // right-child slots (k, j)
#pragma unroll
            for (int c = 0; c < MAXC; ++c) {
                if (c < cnt && l + c * G < K) {
                    const float v = coef * x[c];
                    lp[c * G] += v;
                    rq[c * G] += v;
                }
            }
        }
    }
}

template <int GMAX, int MAXC, typename T>
__device__ __forceinline__ void inside_sweep(T *al, int ld, int n, int tid) {
    for (int w = 2; w <= n; ++w) {
        const int g = pick_group<GMAX, MAXC>(w - 1, n - w + 1);
        switch (g) {
            case 1: inside_width<1, MAXC>(al, ld, n, w, tid); break;
            case 2: inside_width<2, MAXC>(al, ld, n, w, tid); break;
            case 4: inside_width<4, MAXC>(al, ld, n, w, tid); break;
            case 8: inside_width<8, MAXC>(al, ld, n, w, tid); break;
            case 16: inside_width<16, MAXC>(al, ld, n, w, tid); break;
            case 32: if constexpr (GMAX >= 32) inside_width<32, MAXC>(al, ld, n, w, tid); break;
            default: if constexpr (GMAX >= 64) inside_width<64, MAXC>(al, ld, n, w, tid); break;
        }
        __syncthreads();
    }
}

template <int GMAX, int MAXC, typename T>
__device__ __forceinline__ void reverse_sweep(const T *al, T *ad, int ld, int n, int tid,
                                              float gval) {
    for (int w = n; w >= 2; --w) {
        const int g = pick_group<GMAX, MAXC>(w - 1, n - w + 1);
        switch (g) {
            case 1: reverse_width<1, MAXC>(al, ad, ld, n, w, tid, gval); break;
            case 2: reverse_width<2, MAXC>(al, ad, ld, n, w, tid, gval); break;
            case 4: reverse_width<4, MAXC>(al, ad, ld, n, w, tid, gval); break;
            case 8: reverse_width<8, MAXC>(al, ad, ld, n, w, tid, gval); break;
            case 16: reverse_width<16, MAXC>(al, ad, ld, n, w, tid, gval); break;
            case 32: if constexpr (GMAX >= 32) reverse_width<32, MAXC>(al, ad, ld, n, w, tid, gval); break;
            default: if constexpr (GMAX >= 64) reverse_width<64, MAXC>(al, ad, ld, n, w, tid, gval); break;
        }
        __syncthreads();
    }
}

// Sum of a double over the workgroup (result valid in every thread).
__device__ __forceinline__ double block_sum_d(double v, double *red) {
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    const int tid = threadIdx.x;
    if ((tid & 63) == 0) red[tid >> 6] = v;
    __syncthreads();
    double t = 0.0;
#pragma unroll
    for (int q = 0; q < NWAVES; ++q) t += red[q];
    __syncthreads();
    return t;
}

// Log-sum-exp over labels of one span, in log2 units: returns m2 + log2 sum.
__device__ __forceinline__ float label_lse2(const float *s, int L) {
    float m = -INFINITY;
    for (int l = 0; l < L; ++l) m = fmaxf(m, s[l] * LOG2E_F);
    float acc = 0.f;
    for (int l = 0; l < L; ++l) acc += fast_exp2(s[l] * LOG2E_F - m);
    return m + fast_log2(acc);
}

// ---------------------------------------------------------------------------
// Inside (+ reverse) for one sentence per workgroup.
//   REV:  also run the reverse sweep and write marginals.
//   LAB:  labelled scores [B][N1][N1][L].
//   SPILL: chart in the plan workspace instead of LDS.
template <bool REV, bool LAB, bool SPILL>
__global__ __launch_bounds__(NT) void inside_kernel(KernelPlan p, const float *__restrict__ scores,
                                                    const float *__restrict__ grad,
                                                    float *__restrict__ logZ,
                                                    float *__restrict__ marg) {
    extern __shared__ __align__(16) char smem_raw[];
    __shared__ double red[NWAVES];
    const int item = blockIdx.x;
    const int b = SPILL ? p.inside.order_spill[item] : p.inside.order_lds[item];
    const int n = p.len[b];
    const int ld = chart_ld(n);
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int N1 = p.n1, L = p.L;

    float *al;
    if constexpr (SPILL)
        al = reinterpret_cast<float *>(p.ws + p.inside.ws_off[item]);
    else
        al = reinterpret_cast<float *>(smem_raw);
    float *ad = al + (size_t)ld * ld;

    const size_t row_stride = LAB ? (size_t)N1 * L : (size_t)N1;
    const float *sb = scores + (size_t)b * N1 * row_stride;

    // Prologue: scores of the valid triangle into the chart (log2-scaled),
    // forced spans (width 1 and the root) summed in float64 and replaced by 0.
    double forced = 0.0;
    for (int i = wave; i < n; i += NWAVES) {
        for (int j = i + 1 + lane; j <= n; j += 64) {
            float s2;
            if constexpr (LAB)
                s2 = label_lse2(sb + (size_t)i * row_stride + (size_t)j * L, L);
            else
                s2 = sb[(size_t)i * row_stride + j] * LOG2E_F;
            const bool root = (i == 0 && j == n);
            if (j == i + 1) {
                forced += LAB ? (double)s2 * LN2_D : (double)sb[(size_t)i * row_stride + j];
                al[(size_t)i * ld + j] = 0.f;
                al[(size_t)j * ld + i] = 0.f;
            } else if (root) {
                forced += LAB ? (double)s2 * LN2_D : (double)sb[(size_t)i * row_stride + j];
                al[(size_t)i * ld + j] = 0.f;
            } else {
                al[(size_t)i * ld + j] = s2;
            }
        }
    }
    forced = block_sum_d(forced, red);   // contains the barrier that publishes the chart

    inside_sweep<SPILL ? 64 : 16, SPILL ? MAXC_SPILL : MAXC_LDS>(al, ld, n, tid);

    if (logZ != nullptr && tid == 0) logZ[b] = (float)((double)al[n] * LN2_D + forced);
    if constexpr (!REV) return;

    // Reverse sweep.  Clear both triangles of the adjoint square first.
    const float gval = grad ? grad[b] : 1.0f;
    for (int c = tid; c < ld * ld; c += NT) ad[c] = 0.f;
    __syncthreads();
    reverse_sweep<SPILL ? 64 : 16, SPILL ? MAXC_SPILL : MAXC_LDS>(al, ad, ld, n, tid, gval);

    // Epilogue: marginals of the valid triangle, row by row (coalesced).
    float *mb = marg + (size_t)b * N1 * row_stride;
    for (int i = wave; i < n; i += NWAVES) {
        for (int j = i + 1 + lane; j <= n; j += 64) {
            const bool forced_span = (j == i + 1) || (i == 0 && j == n);
            const float mu = forced_span ? gval : ad[(size_t)i * ld + j] + ad[(size_t)j * ld + i];
            if constexpr (LAB) {
                const float *s = sb + (size_t)i * row_stride + (size_t)j * L;
                const float lse2 = label_lse2(s, L);
                float *o = mb + (size_t)i * row_stride + (size_t)j * L;
                for (int q = 0; q < L; ++q) o[q] = mu * fast_exp2(s[q] * LOG2E_F - lse2);
            } else {
                mb[(size_t)i * row_stride + j] = mu;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// CKY, one width: float64 max-plus with the lowest maximising split.
template <int G, int MAXC, typename DT, typename BT>
__device__ __forceinline__ void cky_width(DT *be, BT *bp, int ld, int n, int w, int tid) {
    constexpr int GROUPS = NT / G;
    const int K = w - 1, S = n - w + 1;
    const int cnt = (K + G - 1) / G;
    const int g = tid / G, l = tid % G;
    for (int s0 = 0; s0 < S; s0 += GROUPS) {
        const int sp = s0 + g;
        const bool act = sp < S;
        const int i = act ? sp : S - 1;
        const int j = i + w;
        const DT *rp = be + (size_t)i * ld + (i + 1 + l);
        const DT *cp = be + (size_t)j * ld + (i + 1 + l);
        const double sij = be[(size_t)i * ld + j];
        double lb = -INFINITY;
        int lk = 0x7fffffff;
#pragma unroll
        for (int c = 0; c < MAXC; ++c) {
            if (c < cnt && l + c * G < K) {
                const double v = rp[c * G] + cp[c * G];
                if (lk == 0x7fffffff || v > lb) { lb = v; lk = i + 1 + l + c * G; }
            }
        }
        const double m = grp_max_d<G>(lb);
        const int kk = grp_min_i<G>(lb == m ? lk : 0x7fffffff);
        if (act && l == 0) {
            const double v = m + sij;
            be[(size_t)i * ld + j] = v;
            be[(size_t)j * ld + i] = v;
            bp[(size_t)i * ld + j] = (BT)kk;
        }
    }
}

template <bool SPILL>
__global__ __launch_bounds__(NT) void cky_kernel(KernelPlan p, const float *__restrict__ scores,
                                                 int32_t *__restrict__ spans,
                                                 float *__restrict__ best) {
    extern __shared__ __align__(16) char smem_raw[];
    constexpr int GMAX = SPILL ? 64 : 16;
    constexpr int MAXC = SPILL ? MAXC_SPILL : MAXC_LDS;
    const int item = blockIdx.x;
    const int b = SPILL ? p.cky.order_spill[item] : p.cky.order_lds[item];
    const int n = p.len[b];
    const int ld = chart_ld(n);
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int N1 = p.n1;

    char *base = SPILL ? (p.ws + p.cky.ws_off[item]) : smem_raw;
    double *be = reinterpret_cast<double *>(base);
    uint16_t *bp = reinterpret_cast<uint16_t *>(base + (size_t)ld * ld * 8);

    const float *sb = scores + (size_t)b * N1 * N1;
    for (int i = wave; i < n; i += NWAVES) {
        for (int j = i + 1 + lane; j <= n; j += 64) {
            const double s = (double)sb[(size_t)i * N1 + j];
            be[(size_t)i * ld + j] = s;
            if (j == i + 1) be[(size_t)j * ld + i] = s;
        }
    }
    __syncthreads();

    for (int w = 2; w <= n; ++w) {
        const int g = pick_group<GMAX, MAXC>(w - 1, n - w + 1);
        switch (g) {
            case 1: cky_width<1, MAXC>(be, bp, ld, n, w, tid); break;
            case 2: cky_width<2, MAXC>(be, bp, ld, n, w, tid); break;
            case 4: cky_width<4, MAXC>(be, bp, ld, n, w, tid); break;
            case 8: cky_width<8, MAXC>(be, bp, ld, n, w, tid); break;
            case 16: cky_width<16, MAXC>(be, bp, ld, n, w, tid); break;
            case 32: if constexpr (GMAX >= 32) cky_width<32, MAXC>(be, bp, ld, n, w, tid); break;
            default: if constexpr (GMAX >= 64) cky_width<64, MAXC>(be, bp, ld, n, w, tid); break;
        }
        __syncthreads();
    }

    const int R = 2 * (N1 - 1) - 1;
    int32_t *out = spans + (size_t)b * R * 2;
    // Rows past the tree are -1.
    for (int r = 2 * n - 1 + tid; r < R; r += NT) {
        out[2 * r] = -1;
        out[2 * r + 1] = -1;
    }
    if (tid == 0) {
        if (best) best[b] = (float)be[n];
        // Preorder walk of the back-pointers; the stack reuses the (now dead)
        // beta square, which holds >= 2(n+1) ints.
        int32_t *stk = reinterpret_cast<int32_t *>(be);
        int top = 0, row = 0;
        stk[top++] = 0;
        stk[top++] = n;
        // Bounded: a tree has 2n-1 spans, and a split outside (i, j) ends the walk.
        while (top > 0 && row < 2 * n - 1) {
            const int j = stk[--top];
            const int i = stk[--top];
            out[2 * row] = i;
            out[2 * row + 1] = j;
            ++row;
            if (j - i > 1) {
                const int k = bp[(size_t)i * ld + j];
                if (k <= i || k >= j) break;
                stk[top++] = k;
                stk[top++] = j;
                stk[top++] = i;
                stk[top++] = k;
            }
        }
    }
}

}  // namespace

// ---------------------------------------------------------------------------
// Launchers.

hipError_t set_kernel_attributes(int max_lds_bytes) {
    const void *fns[] = {
        (const void *)inside_kernel<false, false, false>, (const void *)inside_kernel<true, false, false>,
        (const void *)inside_kernel<false, true, false>,  (const void *)inside_kernel<true, true, false>,
        (const void *)cky_kernel<false>,
    };
    for (const void *f : fns) {
        hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, max_lds_bytes);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_inside(const KernelPlan &p, const float *scores, const float *grad, float *logZ,
                         float *marg, hipStream_t stream) {
    const bool rev = marg != nullptr;
    const bool lab = p.L > 1;
    const Schedule &q = p.inside;
    if (q.n_lds > 0) {
        dim3 grid(q.n_lds), block(NT);
        const size_t lds = (size_t)q.lds_bytes;
        if (rev && lab) hipLaunchKernelGGL((inside_kernel<true, true, false>), grid, block, lds, stream, p, scores, grad, logZ, marg);
        else if (rev) hipLaunchKernelGGL((inside_kernel<true, false, false>), grid, block, lds, stream, p, scores, grad, logZ, marg);
        else if (lab) hipLaunchKernelGGL((inside_kernel<false, true, false>), grid, block, lds, stream, p, scores, grad, logZ, marg);
        else hipLaunchKernelGGL((inside_kernel<false, false, false>), grid, block, lds, stream, p, scores, grad, logZ, marg);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (q.n_spill > 0) {
        dim3 grid(q.n_spill), block(NT);
        if (rev && lab) hipLaunchKernelGGL((inside_kernel<true, true, true>), grid, block, 0, stream, p, scores, grad, logZ, marg);
        else if (rev) hipLaunchKernelGGL((inside_kernel<true, false, true>), grid, block, 0, stream, p, scores, grad, logZ, marg);
        else if (lab) hipLaunchKernelGGL((inside_kernel<false, true, true>), grid, block, 0, stream, p, scores, grad, logZ, marg);
        else hipLaunchKernelGGL((inside_kernel<false, false, true>), grid, block, 0, stream, p, scores, grad, logZ, marg);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_cky(const KernelPlan &p, const float *scores, int32_t *spans, float *best,
                      hipStream_t stream) {
    const Schedule &q = p.cky;
    if (q.n_lds > 0) {
        hipLaunchKernelGGL((cky_kernel<false>), dim3(q.n_lds), dim3(NT), (size_t)q.lds_bytes, stream, p, scores, spans, best);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (q.n_spill > 0) {
        hipLaunchKernelGGL((cky_kernel<true>), dim3(q.n_spill), dim3(NT), 0, stream, p, scores, spans, best);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace crf
