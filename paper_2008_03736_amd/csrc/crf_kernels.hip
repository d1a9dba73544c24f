// crf_kernels.hip -- gfx950 kernels for the batched tree-CRF.
//
// Method (Zhang, Zhou & Li, IJCAI 2020):
//   inside   alpha(i,j) = s(i,j) + log sum_{i<k<j} exp(alpha(i,k) + alpha(k,j)),
//            log Z = alpha(0,n)                           (Sec. 3.1, Algorithm 1)
//   marginal p((i,j)|x) = d log Z / d s(i,j)              (Sec. 3.2, Eq. partial-derivative)
//   CKY      the same recursion under max, 1-best tree    (Sec. 3.3, Eq. tree-argmax)
//   labels   s'(i,j) = log sum_l exp s(i,j,l) feeds the inside; per-label
//            marginals are p((i,j)|x) * softmax_l s(i,j,l) (Sec. 4.2, Eq. tree-label-score)
//
// Design.
//   * Bundles.  The host groups sentences of equal length into bundles that
//     fit one workgroup's LDS; a workgroup runs a whole bundle, all of its
//     sentences advancing one span width per barrier.  This is the paper's
//     batching of same-width spans (Sec. 3.1) done inside one CU, where the
//     chart never leaves LDS.  Sentences too long for LDS run alone on the
//     same code with the chart in a plan-owned workspace (L2/MALL resident).
//   * Lanes.  In width w every span has K = w-1 split points and gets G
//     lanes (a power of two <= 64) of C splits each, by the step-shape rule
//     step_shape_k; lane l takes splits l, l+G, ..., all loads issued before
//     the first use.  The split-point log-sum-exp is a max / sum-exp per lane
//     finished by a butterfly over the G lanes (DPP inside a 16-lane row,
//     ds_swizzle across rows, readlane across the two halves of the wave).
//   * Span order.  A step numbers its spans sentence-minor (span start i,
//     then sentence), spread over the 32-lane (4-byte words) or 16-lane
//     (8-byte words) groups of a wavefront, and the plan pads each bundle's
//     row and chart strides (inside_layout, cky_layout) so that every group
//     reads its split operands from distinct LDS banks.
//   * alpha and the outside values are each stored twice, in two squares
//     whose rows are stored rotated, so that every split operand of the
//     inside and of the outside is a contiguous run (see the inside chart
//     layout below).
//   * The chart holds log2-scaled values (v_exp_f32 / v_log_f32 are base 2).
//   * Forced spans -- every tree holds the n width-1 spans and the root -- are
//     factored out of the chart: their scores are summed in float64 and added
//     to log Z, and their marginal is exactly the upstream gradient.  This is
//     exact (Z = exp(forced) Z') and keeps chart magnitudes small.
//   * Marginals.  p((i,j)|x) = exp(alpha(i,j) + O(i,j) - log Z), with O the
//     log outside score (the derivative of Eq. partial-derivative written as
//     inside times outside).  The outside of a width-v span needs outside
//     values of wider spans and alpha of spans no wider than n - v, so the
//     outside of width n-t runs in the same barrier step as the inside of
//     width t+1: one joint sweep of n-1 steps instead of an inside sweep
//     followed by a reverse one.  A per-sentence score shift, estimated a
//     quarter of the way through the sweep, keeps the chart magnitudes (and
//     so the float32 rounding of the exponent) small; it moves log Z by a
//     known amount and leaves every marginal unchanged.
//   * CKY runs a float64 chart in the association order
//     beta(i,j) = (max_k (beta(i,k) + beta(k,j))) + s(i,j): only IEEE adds
//     and exact max, so the tree is reproducible bit for bit; ties keep the
//     lowest split, which the sweep records per span in a split table.  The
//     tree walk only looks splits up: a node (i,j) written at preorder row r
//     with split k puts (i,k) at row r+1 and (k,j) at row r+2(k-i).  One
//     lane per word p of every sentence walks down from the root towards p
//     and writes the nodes whose leftmost word is p.
//   * The fused launch is persistent: one workgroup per slot runs a chain of
//     bundles, claiming each next one from a device counter as it frees up.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

#include "crf_internal.h"

namespace crf {
namespace {

constexpr float LOG2E_F = 1.4426950408889634f;
constexpr double LN2_D = 0.69314718055994530942;

template <int G>
constexpr int ilog2() {
    return G <= 1 ? 0 : 1 + ilog2<G / 2>();
}

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
__device__ __forceinline__ float swz16_f(float v) {
    return __builtin_bit_cast(float, swz16_i(__builtin_bit_cast(int, v)));
}
__device__ __forceinline__ double swz16_d(double v) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const int lo = swz16_i((int)(uint32_t)u), hi = swz16_i((int)(uint32_t)(u >> 32));
    return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}
// The two 32-lane halves' values, for the last level of a 64-lane group.
__device__ __forceinline__ float half0_f(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
}
__device__ __forceinline__ float half1_f(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
}
__device__ __forceinline__ double readlane_d(double v, int lane) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, lane);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), lane);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// DPP controls: quad_perm [1,0,3,2] (xor 1), quad_perm [2,3,0,1] (xor 2),
// row_half_mirror (pairs the two quads of each 8 lanes), row_mirror (pairs
// the two halves of each 16-lane row).
constexpr int DPP_XOR1 = 0xB1, DPP_XOR2 = 0x4E, DPP_HMIRROR = 0x141, DPP_MIRROR = 0x140;

// Plain IEEE max (the library is built with -fno-honor-nans: no NaN reaches
// the chart, and the DPP moves fold into v_max_f32_dpp).
__device__ __forceinline__ float fmax_nn(float a, float b) { return __builtin_fmaxf(a, b); }

template <int G>
__device__ __forceinline__ float grp_max(float v) {
    if constexpr (G >= 2) v = fmax_nn(v, dpp_f<DPP_XOR1>(v));
    if constexpr (G >= 4) v = fmax_nn(v, dpp_f<DPP_XOR2>(v));
    if constexpr (G >= 8) v = fmax_nn(v, dpp_f<DPP_HMIRROR>(v));
    if constexpr (G >= 16) v = fmax_nn(v, dpp_f<DPP_MIRROR>(v));
    if constexpr (G >= 32) v = fmax_nn(v, swz16_f(v));
    if constexpr (G >= 64) v = fmax_nn(half0_f(v), half1_f(v));
    return v;
}
template <int G>
__device__ __forceinline__ float grp_sum(float v) {
    if constexpr (G >= 2) v += dpp_f<DPP_XOR1>(v);
    if constexpr (G >= 4) v += dpp_f<DPP_XOR2>(v);
    if constexpr (G >= 8) v += dpp_f<DPP_HMIRROR>(v);
    if constexpr (G >= 16) v += dpp_f<DPP_MIRROR>(v);
    if constexpr (G >= 32) v += swz16_f(v);
    if constexpr (G >= 64) v = half0_f(v) + half1_f(v);
    return v;
}
template <int G>
__device__ __forceinline__ double grp_max_d(double v) {
    if constexpr (G >= 2) v = fmax(v, dpp_d<DPP_XOR1>(v));
    if constexpr (G >= 4) v = fmax(v, dpp_d<DPP_XOR2>(v));
    if constexpr (G >= 8) v = fmax(v, dpp_d<DPP_HMIRROR>(v));
    if constexpr (G >= 16) v = fmax(v, dpp_d<DPP_MIRROR>(v));
    if constexpr (G >= 32) v = fmax(v, swz16_d(v));
    if constexpr (G >= 64) v = fmax(readlane_d(v, 0), readlane_d(v, 32));
    return v;
}
template <int G>
__device__ __forceinline__ double grp_sum_d(double v) {
    if constexpr (G >= 2) v += dpp_d<DPP_XOR1>(v);
    if constexpr (G >= 4) v += dpp_d<DPP_XOR2>(v);
    if constexpr (G >= 8) v += dpp_d<DPP_HMIRROR>(v);
    if constexpr (G >= 16) v += dpp_d<DPP_MIRROR>(v);
    if constexpr (G >= 32) v += swz16_d(v);
    if constexpr (G >= 64) v = readlane_d(v, 0) + readlane_d(v, 32);
    return v;
}
template <int G>
__device__ __forceinline__ int grp_min_i(int v) {
    if constexpr (G >= 2) v = min(v, dpp_i<DPP_XOR1>(v));
    if constexpr (G >= 4) v = min(v, dpp_i<DPP_XOR2>(v));
    if constexpr (G >= 8) v = min(v, dpp_i<DPP_HMIRROR>(v));
    if constexpr (G >= 16) v = min(v, dpp_i<DPP_MIRROR>(v));
    if constexpr (G >= 32) v = min(v, swz16_i(v));
    if constexpr (G >= 64) v = min(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 32));
    return v;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }
// log2 of a positive normal float, in float64: the exact binary exponent plus
// the float32 log2 of the mantissa in [0.5, 1) (good to about 1e-7 absolute
// at any exponent).  No float64 log: its polynomial's coefficients would be
// kept in a dozen VGPRs across a persistent kernel's loop.
__device__ __forceinline__ double log2_split(float x) {
    return (double)__builtin_amdgcn_frexp_expf(x) + (double)fast_log2(__builtin_amdgcn_frexp_mantf(x));
}

// a / d for 0 <= a < 2^24, 1 <= d, with inv = 1.0f / d: the float quotient is
// within one of the truth and is corrected exactly.
__device__ __forceinline__ int div_small(int a, int d, float inv) {
    int q = (int)((float)a * inv);
    q += ((q + 1) * d <= a) ? 1 : 0;
    q -= (q * d > a) ? 1 : 0;
    return q;
}

// Sentinel for "no split": far below any chart value, and finite so that
// differences of two sentinels stay finite (exp2 of the difference of a
// sentinel and a real value is 0).
constexpr float NEG = -1.0e30f;

__device__ __forceinline__ int next_pow2(int x) { return x <= 1 ? 1 : 1 << (32 - __builtin_clz(x - 1)); }
__device__ __forceinline__ int floor_pow2(int x) { return x <= 1 ? 1 : 1 << (31 - __builtin_clz(x)); }

// ---------------------------------------------------------------------------
// Teams.  A workspace sentence's pass can run on k workgroups of one XCD:
// member `rank` takes virtual threads rank * blockDim.x + threadIdx.x of
// k * blockDim.x in every step, and a team barrier replaces the workgroup
// barrier between steps.  The chart goes through the XCD's L2, which the
// members share: a member's stores are in L2 before its arrival is counted,
// and the members read the chart with device-coherent loads (chart_ld),
// which a CU's stale L1 lines cannot serve.  The arrival counters are
// updated by atomics and polled the same way.  k = 1: a lone workgroup,
// whose barriers are __syncthreads.
struct Team {
    int k = 1, rank = 0;
    int32_t *line = nullptr;   // the team's words: [0] arrivals, [1] last job (+1) that left float32's range
    int32_t *err = nullptr;    // the launch's abort flag
    int *ep = nullptr;         // (LDS) team barriers this workgroup has passed
    int job = 0;               // jobs this team has started
};

// A wait that lasts this many polls (a second or two) sets the abort flag;
// from then on no team barrier of the launch waits (the log Z and best
// score of its workspace sentences are NaN; a grid that never assembled
// forms no team and writes nothing).  Only a grid that is not resident at
// once can take that long.
constexpr int kTeamSpin = 1 << 21;

__device__ __forceinline__ int load_coherent(const int32_t *q) {
    return __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ bool team_aborted(const Team &tm) { return tm.k > 1 && load_coherent(tm.err) != 0; }

__device__ __forceinline__ void team_sync(const Team &tm) {
    if (tm.k == 1) {
        __syncthreads();
        return;
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this wave's stores are in L2
    __syncthreads();
    if (threadIdx.x == 0) {
        const int target = tm.k * ++*tm.ep;
        atomicAdd(tm.line, 1);
        for (int s = 0; load_coherent(tm.line) < target; ++s)
            if ((s & 63) == 63 && (s >= kTeamSpin || load_coherent(tm.err) != 0)) {
                atomicOr(tm.err, 1);
                break;
            }
    }
    __syncthreads();
}

// Barrier after a sweep step: the team's, or the workgroup's.
template <bool TEAM>
__device__ __forceinline__ void step_sync(const Team &tm) {
    if constexpr (TEAM) team_sync(tm);
    else __syncthreads();
}

// A chart read.  A team's members read each other's stores through device-
// coherent loads: they skip this CU's L1 (which nothing short of dropping
// the XCD's whole L2 invalidates) and are served by the XCD's L2.  Plain
// loads otherwise.
template <bool TEAM, typename T>
__device__ __forceinline__ T chart_ld(const T *q) {
    if constexpr (TEAM) return __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else return *q;
}

// The same with the choice made at run time (reads outside the steps).
template <typename T>
__device__ __forceinline__ T chart_ld_if(const T *q, bool coherent) {
    return coherent ? __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : *q;
}

// Virtual thread index and count of a step's lanes.
template <bool TEAM>
__device__ __forceinline__ int team_tid(const Team &tm) {
    if constexpr (TEAM) return tm.rank * (int)blockDim.x + (int)threadIdx.x;
    else return (int)threadIdx.x;
}
template <bool TEAM>
__device__ __forceinline__ int team_nt(const Team &tm) {
    if constexpr (TEAM) return tm.k * (int)blockDim.x;
    else return (int)blockDim.x;
}

// Joins the launch's teams (thread 0; every workgroup of the grid resident
// at once, the team area zeroed before the launch).  Each workgroup counts
// itself on its XCD (the XCC_ID hardware register) and waits for the whole
// grid; then the workgroups of each XCD form teams of k in arrival order.
// Returns the team (-1: left over, or the grid never assembled), the
// member's rank and the number of teams.
struct Team_slot {
    int team, rank, teams;
};
__device__ Team_slot join_team(int32_t *area, int k) {
    const int xcc = __builtin_amdgcn_s_getreg((3 << 11) | 20) & 15;   // hwreg(HW_REG_XCC_ID, 0, 4)
    const int slot = atomicAdd(area + xcc, 1);
    atomicAdd(area + 16, 1);
    for (int s = 0; load_coherent(area + 16) < (int)gridDim.x; ++s)
        if ((s & 63) == 63 && (s >= kTeamSpin || load_coherent(area + 17) != 0)) {
            atomicOr(area + 17, 1);
            return Team_slot{-1, 0, 0};
        }
    int before = 0, teams = 0;
    for (int x = 0; x < 16; ++x) {
        const int c = load_coherent(area + x) / k;
        if (x < xcc) before += c;
        teams += c;
    }
    if (slot >= (load_coherent(area + xcc) / k) * k) return Team_slot{-1, 0, teams};
    return Team_slot{before + slot / k, slot % k, teams};
}

// The jobs of a workspace launch by teams (sentence passes 0, 1, ...;
// launched when p.team_k > 1; otherwise each workgroup takes the job of its
// index): team t takes jobs t, t + T, ...  Sets this workgroup's team, first
// job and stride; false: it takes no job.  (The callers loop over the jobs
// themselves, with a barrier between jobs and ++tm.job.)  tm.k is at least 2,
// as the compiler can see, so a team build holds only the team sweeps (and a
// lone build, whose Team is the default, only the others).
__device__ __forceinline__ bool spill_jobs(const KernelPlan &p, Team &tm, int &first, int &stride) {
    __shared__ int slot[3];
    __shared__ int ep;
    tm = Team{};
    if (threadIdx.x == 0) {
        const Team_slot ts = join_team(p.team_area, p.team_k);
        slot[0] = ts.team;
        slot[1] = ts.rank;
        slot[2] = ts.teams;
        ep = 0;
    }
    __syncthreads();
    if (slot[0] < 0) return false;
    tm.k = max(2, p.team_k);
    tm.rank = slot[1];
    tm.line = p.team_area + kTeamHeaderWords + slot[0] * kTeamLineWords;
    tm.err = p.team_area + 17;
    tm.ep = &ep;
    first = slot[0];
    stride = slot[2];
    return true;
}

// ---------------------------------------------------------------------------
// Per-bundle context: nb sentences of length n; sentence sb's chart starts at
// chart0 + sb * cstride (elements).

template <typename T>
struct Bundle_ctx {
    T *chart0;
    int cstride;   // elements between consecutive sentences' charts
    int n, ld, nb;
    uint32_t mnb;   // div_magic(nb)
    int e;          // the inside layout's bank exponent (inside_layout); 5 on the workspace
    int *ovf;       // linear-domain sweeps: set to 1 (LDS) when a value leaves float32's range
    Team tm;        // workspace sentences: the team running the pass
};


// Where lane f of a step's region works.  The region's nsp spans are numbered
// sentence-minor, g = i nb + sb (sentence sb, span start i; g / nb by
// multiply-high with mnb = 2^32 / nb + 1, exact for g < 2^18, nb <= 1024).
// LDS serves a wavefront's accesses in groups of HW lanes (32 for 4-byte
// words, 16 for 8-byte ones), each over 32 banks.  Interleaved (IL, for
// layouts with e = 0), lanes come in blocks of G groups holding HW spans:
// group h of a block takes spans h, h + G, h + 2G, ..., each span's G lanes
// side by side, lane l of them taking split positions l, l + G, ...  With
// the chart layouts' strides span g's operand runs start sigma g banks (or
// bank pairs) apart, modulo the group's bank count, so for sigma odd the
// HW lanes of a group hit distinct banks.  Otherwise (e > 0, or spans of a
// whole group or more) spans lie side by side in lane order.  A lane past
// the region's spans (act = false) copies span and lane of an active lane
// of its group, or in a group with none the last span: its loads repeat
// addresses the group already reads, which costs no bank cycle.
struct Lane_at {
    int sb, i, l;
    bool act;
};
template <int G, bool IL, int HW>
struct Lane_map {
    static constexpr int LG = ilog2<G>(), LH = ilog2<HW>();
    static constexpr int lq = (IL && G < HW) ? LG : 0;   // log2 of the groups per block
    static constexpr int unit = HW << lq;                // lanes per block
};
template <int G, bool IL, int HW = 32>
__device__ __forceinline__ Lane_at lane_at(int f, int nsp, int nb, uint32_t mnb) {
    using M = Lane_map<G, IL, HW>;
    constexpr int LG = M::LG, LH = M::LH, lq = M::lq;
    const int l = f & (G - 1);
    int g;
    bool act;
    if constexpr (G >= HW) {   // a span fills one or more groups on its own
        g = f >> LG;
        act = g < nsp;
        if (!act) g = nsp - 1;
    } else {
        const int h = (f >> LH) & ((1 << lq) - 1);
        const int b0 = (f >> (LH + lq)) << (LH + lq - LG);
        g = b0 + h + (((f & (HW - 1)) >> LG) << lq);
        act = g < nsp;
        if (!act) {
            const int rem = nsp - b0;
            g = h < rem ? b0 + h + (((rem - 1 - h) >> lq) << lq) : nsp - 1;
        }
    }
    const int i = nb > 1 ? (int)__umulhi((uint32_t)g, mnb) : g;
    return Lane_at{g - (int)__umul24((uint32_t)i, (uint32_t)nb), i, l, act};
}
// Whether the wavefront whose first lane is f of a region (f a multiple of
// 64) holds any of its nsp spans (its first group's first span).
template <int G, bool IL, int HW = 32>
__device__ __forceinline__ bool wave_has_span(int f, int nsp) {
    using M = Lane_map<G, IL, HW>;
    constexpr int LG = M::LG, LH = M::LH, lq = M::lq;
    if constexpr (G >= HW) return (f >> LG) < nsp;
    else return ((f >> (LH + lq)) << (LH + lq - LG)) + ((f >> LH) & ((1 << lq) - 1)) < nsp;
}
// Lanes of a region of nsp spans: whole blocks.
template <int G, bool IL, int HW = 32>
__device__ __forceinline__ int region_lanes(int nsp) {
    constexpr int unit = Lane_map<G, IL, HW>::unit;
    return (nsp * G + unit - 1) & ~(unit - 1);
}

// Inside chart layout.  Two ld x ld float32 squares per sentence, P and Q,
// with P upper = alpha, P lower = O' mirrored, and Q = P transposed (Q upper
// = O', Q lower = alpha mirrored), where O'(a,b) = O(a,b) + s(a,b) + d is the
// outside score plus the span's own (shifted) score, zero at the root.  Row r
// of P is stored rotated left by r+1 and row r of Q by r (position p of row r
// holds column (p + r + 1) mod (n+1), resp. (p + r) mod (n+1)).  Then both
// recursions read two contiguous runs at offsets uniform over a step:
//   inside  (i,j), w = j-i:  alpha(i,k) + alpha(k,j) = P[i][p] + Q[j][p + n+2-w],
//                            p = k-i-1 in [0, w-1);
//   outside (i,j), v = j-i:  the parents' O' plus the siblings' alpha, over
//                            t in [0,i) u (j,n], = P[j][p] + Q[i][p + v+1],
//                            p in [0, n-v)
// (rows and positions in the rotated squares).  A span (a,b) of width w
// keeps alpha at P[a][w-1] and Q[b][n+1-w], O' at Q[a][w] and P[b][n-w];
// before the sweeps reach it those cells hold its (log2-scaled) score, which
// the steps read as the span's own term.  Cells no sweep reads park the
// natural-unit scores of the forced spans: width 1 at P[i+1][n-1], the root
// at P[0][n].
__host__ __device__ constexpr int rot_alpha_p(int w) { return w - 1; }
template <typename T>
__device__ __forceinline__ T *sq_p(const Bundle_ctx<T> &bx, int sb) {   // (sb < 256, cstride < 2^24)
    return bx.chart0 + __umul24((uint32_t)sb, (uint32_t)bx.cstride);
}

// One span's log-sum-exp over the K split terms of a step: lane l of the
// span's G lanes takes positions p = l + c*G, c < C, of the two runs a and b
// (terms c >= MF may fall past K: they count as exp2(-inf) = 0 and read at
// most (C - MF)*G cells past the run); the group's result plus `own` is
// returned to every lane of the group.
template <int G, int C, int MF, bool TEAM, typename T>
__device__ __forceinline__ float span_lse(const T *a, const T *b, int kl, float own) {
    float x[C], xa[C], xb[C];
#pragma unroll
    for (int c = 0; c < C; ++c) {
        xa[c] = chart_ld<TEAM>(&a[c * G]);
        xb[c] = chart_ld<TEAM>(&b[c * G]);
    }
    __builtin_amdgcn_sched_barrier(0);   // every load in flight before the first use
#pragma unroll
    for (int c = 0; c < C; ++c) x[c] = xa[c] + xb[c];
#pragma unroll
    for (int c = MF; c < C; ++c) x[c] = (c * G < kl) ? x[c] : NEG;
    float m = x[0];
#pragma unroll
    for (int c = 1; c < C; ++c) m = fmax_nn(m, x[c]);
    float s = fast_exp2(x[0] - m);
#pragma unroll
    for (int c = 1; c < C; ++c) s += fast_exp2(x[c] - m);
    const float mg = grp_max<G>(m);
    const float sg = grp_sum<G>(s * fast_exp2(m - mg));
    return mg + fast_log2(sg) + own;
}

// The same sum in the linear domain (the chart holding exp2 of the values
// above): one span's sum over its K split terms is the dot product of its
// two runs, sum_k a_k b_k, one FMA per term.  Terms c >= MF past K are
// dropped by a select on the accumulator, so whatever the masked reads find
// (other spans' scores, padding) never reaches the sum.  Two accumulators
// halve the dependent chain.  The span's own score (at po, log2 units) and
// its sentence's shift (at pd, added when `shifted`) are loaded with the
// operands, so that a step pays one LDS round trip; the group's sum times
// exp2(own + shift) is returned to every lane.
template <int G, int C, int MF, bool TEAM, typename T>
__device__ __forceinline__ float span_dot(const T *a, const T *b, int kl, const T *po, const float *pd,
                                          bool shifted) {
    float xa[C], xb[C];
#pragma unroll
    for (int c = 0; c < C; ++c) {
        xa[c] = chart_ld<TEAM>(&a[c * G]);
        xb[c] = chart_ld<TEAM>(&b[c * G]);
    }
    const float own = chart_ld<TEAM>(po), sh = *pd;
    __builtin_amdgcn_sched_barrier(0);   // every load in flight before the first use
    const float e = fast_exp2(shifted ? own + sh : own);
    float acc[2] = {0.f, 0.f};
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const float t = __builtin_fmaf(xa[c], xb[c], acc[c & 1]);
        acc[c & 1] = (c < MF || c * G < kl) ? t : acc[c & 1];
    }
    return e * grp_sum<G>(acc[0] + acc[1]);
}

// Bound of a stored linear-domain value: anything above it (infinity, NaN
// or a value whose products could overflow) sends the bundle to the
// log-domain sweep.
constexpr float kLinMax = 0x1p+100f;

// One span of a width-w inside step (K = w - 1 splits):
// alpha(i,j) = s(i,j) + d + log2 sum_k exp2(alpha(i,k) + alpha(k,j)), d the
// sentence's score shift (see rescale_chart); the root's own term is not
// shifted.  LIN: the chart holds exp2 of these values, and the span's value
// is exp2(own) * sum_k alpha(i,k) alpha(k,j).
template <bool LIN, int G, int C, int MF, bool IL, bool TEAM, typename T>
__device__ __forceinline__ void inside_span(const Bundle_ctx<T> &bx, int w, int nsp, int f, const float *dsh) {
    const int ld = bx.ld, n = bx.n, K = w - 1;
    const Lane_at at = lane_at<G, IL>(f, nsp, bx.nb, bx.mnb);
    const int i = at.i, l = at.l;
    T *pq = sq_p(bx, at.sb);
    const int rp = (int)__umul24((uint32_t)i, (uint32_t)ld);              // P row i
    const int rq = (int)__umul24((uint32_t)(i + ld + w), (uint32_t)ld);   // Q row j
    const int pa = rp + rot_alpha_p(w), qa = rq + n + 1 - w;                   // alpha(i,j) cells
    float v;
    if constexpr (LIN)
        v = span_dot<G, C, MF, TEAM>(pq + rp + l, pq + rq + (n + 2 - w) + l, K - l, pq + pa, dsh + at.sb, w < n);
    else
        v = span_lse<G, C, MF, TEAM>(pq + rp + l, pq + rq + (n + 2 - w) + l, K - l,
                                     chart_ld<TEAM>(&pq[pa]) + (w < n ? dsh[at.sb] : 0.f));
    // An unconditional use keeps the score load in the load block, where it
    // is issued with the operand loads instead of after the reductions.
    asm volatile("" ::"v"(v));
    if (at.act && l == 0) {
        pq[pa] = v;
        pq[qa] = v;
        if constexpr (LIN)
            if (!(v <= kLinMax)) *bx.ovf = 1;
    }
}

// One span (i,j) of a width-v outside step: K = n - v parent terms, every
// operand a parent of width > v or a sibling of width <= n - v, so this step
// runs beside the inside step of width n - v + 1.
template <bool LIN, int G, int C, int MF, bool IL, bool TEAM, typename T>
__device__ __forceinline__ void outside_span(const Bundle_ctx<T> &bx, int v, int nsp, int f, const float *dsh) {
    const int ld = bx.ld, n = bx.n, K = n - v;
    const Lane_at at = lane_at<G, IL>(f, nsp, bx.nb, bx.mnb);
    const int i = at.i, l = at.l;
    T *pq = sq_p(bx, at.sb);
    const int rp = (int)__umul24((uint32_t)(i + v), (uint32_t)ld);    // P row j
    const int rq = (int)__umul24((uint32_t)(i + ld), (uint32_t)ld);   // Q row i
    const int po = rp + n - v, qo = rq + v;                          // O'(i,j) cells
    float o;
    if constexpr (LIN)
        o = span_dot<G, C, MF, TEAM>(pq + rp + l, pq + rq + v + 1 + l, K - l, pq + po, dsh + at.sb, true);
    else
        o = span_lse<G, C, MF, TEAM>(pq + rp + l, pq + rq + v + 1 + l, K - l, chart_ld<TEAM>(&pq[po]) + dsh[at.sb]);
    asm volatile("" ::"v"(o));
    if (at.act && l == 0) {
        pq[qo] = o;
        pq[po] = o;
        if constexpr (LIN)
            if (!(o <= kLinMax)) *bx.ovf = 1;
    }
}

// Forward-only width step: every span of width w of every sentence.
template <bool LIN, int G, int C, int MF, bool IL, bool TEAM, typename T>
__device__ __forceinline__ void fwd_step(const Bundle_ctx<T> &bx, int w, const float *dsh) {
    const int tid = team_tid<TEAM>(bx.tm), nt = team_nt<TEAM>(bx.tm);
    const int nsp = bx.nb * (bx.n - w + 1);
    const int total = region_lanes<G, IL>(nsp);
    const int wq0 = __builtin_amdgcn_readfirstlane(tid & ~63);   // this wavefront's first thread
    for (int f0 = 0; f0 < total; f0 += nt) {
        const int fw = f0 + wq0;
        if (fw >= total) break;   // no span for this wavefront in this pass or later
        if (wave_has_span<G, IL>(fw, nsp)) inside_span<LIN, G, C, MF, IL, TEAM>(bx, w, nsp, f0 + tid, dsh);
    }
}

// Step t of the joint sweep: inside width t+1 and outside width n-t (when
// >= 2), both with K = t terms per span, so one step shape serves both.
// Inside spans take the first threads, outside spans start at the next
// wavefront boundary, so every wavefront runs one kind.
template <bool LIN, int G, int C, int MF, bool IL, bool TEAM, typename T>
__device__ __forceinline__ void io_step(const Bundle_ctx<T> &bx, int t, const float *dsh) {
    const int tid = team_tid<TEAM>(bx.tm), nt = team_nt<TEAM>(bx.tm);
    const int n = bx.n, w = t + 1, v = n - t;
    const int nin = bx.nb * (n - t), nout = v >= 2 ? bx.nb * (t + 1) : 0;
    const int obase = (region_lanes<G, IL>(nin) + 63) & ~63;
    const int total = obase + region_lanes<G, IL>(nout);
    const int wq0 = __builtin_amdgcn_readfirstlane(tid & ~63);
    for (int f0 = 0; f0 < total; f0 += nt) {
        const int fw = f0 + wq0;
        if (fw >= total) break;
        if (fw < obase) {
            if (wave_has_span<G, IL>(fw, nin)) inside_span<LIN, G, C, MF, IL, TEAM>(bx, w, nin, f0 + tid, dsh);
        } else {
            if (wave_has_span<G, IL>(fw - obase, nout))
                outside_span<LIN, G, C, MF, IL, TEAM>(bx, v, nout, f0 + tid - obase, dsh);
        }
    }
}

// A run of forward widths [w0, w1) sharing one step shape: a tight loop with
// no dispatch.
template <bool LIN, int G, int C, int MF, bool IL, bool TEAM, typename T>
__device__ __forceinline__ void fwd_run(const Bundle_ctx<T> &bx, int w0, int w1, const float *dsh) {
    for (int w = w0; w < w1; ++w) {
        fwd_step<LIN, G, C, MF, IL, TEAM>(bx, w, dsh);
        step_sync<TEAM>(bx.tm);
    }
}

// A run of joint steps [t0, t1) sharing one step shape.  Span counts are
// n - t (inside) and t + 1 (outside), both in [1, n+1].
template <bool LIN, int G, int C, int MF, bool IL, bool TEAM, typename T>
__device__ __forceinline__ void io_run(const Bundle_ctx<T> &bx, int t0, int t1, const float *dsh) {
    for (int t = t0; t < t1; ++t) {
        io_step<LIN, G, C, MF, IL, TEAM>(bx, t, dsh);
        step_sync<TEAM>(bx.tm);
    }
}

// Calls RUN(G, C, MF) for the shape of a step of more than 128 splits
// (the fixed runs take the others).  Charts in LDS hold at most 142 words
// (K <= 141), so their sweeps need only (16, 12); only the workspace (WIDE)
// kernels build the wider shapes.
#define CRF_DISPATCH_WIDE_SHAPE(SH, RUN)                     \
    do {                                                     \
        if (!WIDE || ((SH).G == 16 && (SH).C == 12)) {       \
            RUN(16, 12, 8);                                  \
        } else if constexpr (WIDE) {                         \
            if ((SH).G == 16) RUN(16, 16, 12);               \
            else if ((SH).G == 32) {                         \
                if ((SH).C == 12) RUN(32, 12, 8);            \
                else RUN(32, 16, 12);                        \
            } else {                                         \
                if ((SH).C == 12) RUN(64, 12, 8);            \
                else RUN(64, 16, 12);                        \
            }                                                \
        }                                                    \
    } while (0)

// Where a sweep stops for a rescale of the chart: after step t, the first
// rescale point >= lo, or 0 when no rescale is left.  One after step n/4
// (n >= 8).  The linear domain, whose shift starts from an estimate (see
// inside_block_impl), adds one after step 16 for sentences of 100 words or
// more, before a poor estimate can drift a whole width out of float32's
// range, and one after step n/2 for sentences of more than 128 words.
template <bool LIN>
__device__ __forceinline__ int next_rescale(int lo, int n) {
    if constexpr (LIN)
        if (n >= 100 && lo <= 16) return 16;
    const int t0 = n >= 8 ? n / 4 : 0;
    if (t0 >= lo) return t0;
    if constexpr (LIN)
        if (n > 128 && n / 2 >= lo) return n / 2;
    return 0;
}

template <bool LIN, bool REV, bool TEAM, typename T>
__device__ void rescale_chart(const Bundle_ctx<T> &bx, int t0, float *dsh, float *dl);

// The forward sweep alone: steps t = 1..n-1 (widths 2..n), one dispatch per
// run of steps sharing a step shape; the linear domain cuts the runs for its
// rescales (the log domain needs none here).
// WIDE: workspace charts (longer sentences), which may need 16 terms per lane.
// IL: interleaved span numbering (lane_at).
// dl: per-sentence scratch for the rescales.
template <bool LIN, bool WIDE, bool IL, bool TEAM, bool MULTI = true, typename T>
__device__ __forceinline__ void fwd_sweep(const Bundle_ctx<T> &bx, float *dsh, float *dl) {
    const int n = bx.n;
    for (int lo = 1; lo < n;) {
        const int tr = LIN ? next_rescale<true>(lo, n) : 0;
        const int hi = tr > 0 ? tr + 1 : n;   // steps [lo, hi), widths [lo + 1, hi + 1)
#define CRF_FWD_FIXED(LO, HI, GG, CC, MM)                                                  \
        if (max(lo, LO) < min(hi, HI + 1))                                                 \
            fwd_run<LIN, GG, CC, MM, IL, TEAM>(bx, max(lo, LO) + 1, min(hi, HI + 1) + 1, dsh);
        CRF_FIXED_RUNS_LOW(CRF_FWD_FIXED)
        if (MULTI && !WIDE && short_bundle(bx.nb, n, (int)blockDim.x)) {
            CRF_SHORT_RUNS_MID(CRF_FWD_FIXED)
        } else {
            CRF_FIXED_RUNS_MID(CRF_FWD_FIXED)
        }
        CRF_FIXED_RUNS_HIGH(CRF_FWD_FIXED)
#undef CRF_FWD_FIXED
        for (int t = max(lo, kFixedRunsMaxK + 1); t < hi;) {
            const StepShape sh = step_shape_k(t);
            const int t2 = min(shape_run_end(t), hi);
#define CRF_FWD_RUN(GG, CC, MM) fwd_run<LIN, GG, CC, MM, IL, TEAM>(bx, t + 1, t2 + 1, dsh)
            CRF_DISPATCH_WIDE_SHAPE(sh, CRF_FWD_RUN);
#undef CRF_FWD_RUN
            t = t2;
        }
        if (tr > 0) rescale_chart<LIN, false, TEAM>(bx, tr, dsh, dl);
        lo = hi;
    }
}


// Per-sentence work of a bundle on groups of GS lanes, GS the smallest of
// 8, 16, 32, 64 that covers `len` items per sentence (so that short
// sentences share a wavefront and reduce with DPP moves, not through LDS):
// group q of the workgroup takes sentences q, q + NG, ...  f(gs, sb, gl,
// valid) runs on every lane of a wavefront that holds a sentence; a group
// past the last sentence gets valid = false and the last sentence's index.
// GS depends on len only, so a group's summation order is fixed.
template <typename F>
__device__ __forceinline__ void by_sentence_groups(int len, int nb, F &&f) {
    auto run = [&](auto gs) {
        constexpr int GS = decltype(gs)::value;
        const int NG = blockDim.x / GS, q = threadIdx.x / GS, gl = threadIdx.x & (GS - 1);
        const int q_wave = __builtin_amdgcn_readfirstlane((threadIdx.x & ~63) / GS);   // the wavefront's first group
        for (int sb0 = 0; sb0 + q_wave < nb; sb0 += NG) {
            const int sb = sb0 + q;
            f(gs, sb < nb ? sb : nb - 1, gl, sb < nb);
        }
    };
    if (len <= 8) run(std::integral_constant<int, 8>{});
    else if (len <= 16) run(std::integral_constant<int, 16>{});
    else if (len <= 32) run(std::integral_constant<int, 32>{});
    else run(std::integral_constant<int, 64>{});
}

// Spans below a sentence's largest alpha of the probe width by more than this
// many log2 units per internal node are left out of its growth estimate (they
// hold near-forbidden scores, not the typical growth).
constexpr float kShiftBand = 30.0f;

// Score shift.  Adding one constant d to every non-forced score adds d times
// their number, n - 2, to the log score of every tree: log Z moves by
// (n-2) d and no marginal changes.  Chart values grow about linearly with the
// span width; the shift keeps them near zero (log domain: so that the
// float32 rounding of alpha + O - log Z, the exponent of a marginal, stays
// small; linear domain: so that exp2 of them stays in float32's range).
// After step t0 (inside widths <= t0+1 done, outside widths >= n-t0 done) a
// further shift delta is estimated from alpha at width w0 = t0+1 -- log
// domain: minus the mean growth per node of the spans within kShiftBand of
// the largest; linear domain: minus the midpoint of that mean and the
// largest, which keeps the largest values further from float32's limit --
// and the stored values move to the shifted problem:
//   alpha(i,j) += delta (w-1)   (w-1 non-forced nodes below and at (i,j))
//   O'(i,j)    += delta (n-w)   (n-1-w above it, plus its own score)
// (times exp2 of these in the linear domain), d += delta.  Later steps add d
// to each score as they read it; the root's O' stays 0.  dl holds delta per
// sentence meanwhile.
template <bool LIN, bool REV, bool TEAM, typename T>
__device__ void rescale_chart(const Bundle_ctx<T> &bx, int t0, float *dsh, float *dl) {
    const int n = bx.n, ld = bx.ld, nb = bx.nb, w0 = t0 + 1, S = n - t0;
    // (every member of a team estimates the shifts from the whole chart,
    // the same figures in the same order, then moves its share of cells)
    const int tid = team_tid<TEAM>(bx.tm), nt = team_nt<TEAM>(bx.tm);
    by_sentence_groups(S, nb, [&](auto gs, int sb, int gl, bool valid) {
        constexpr int GS = decltype(gs)::value;
        const T *P = bx.chart0 + (size_t)sb * bx.cstride;
        auto val = [&](int i) {
            const float a = chart_ld<TEAM>(&P[i * ld + w0 - 1]);
            if constexpr (LIN) return fast_log2(a);   // (0 gives -inf, below NEG)
            else return a;
        };
        float m = NEG;
        for (int i = gl; i < S; i += GS) m = fmax_nn(m, val(i));
        m = grp_max<GS>(m);
        const float floor_v = m - kShiftBand * (float)(w0 - 1);
        float acc = 0.f, cnt = 0.f;
        for (int i = gl; i < S; i += GS) {
            const float a = val(i);
            if (a >= floor_v) {
                acc += a;
                cnt += 1.f;
            }
        }
        acc = grp_sum<GS>(acc);
        cnt = grp_sum<GS>(cnt);
        float delta;
        if constexpr (LIN)   // (every value 0: no shift)
            delta = m > 0.5f * NEG ? -0.5f * (m + acc / cnt) / (float)(w0 - 1) : 0.f;
        else
            delta = -acc / (cnt * (float)(w0 - 1));
        if (valid && gl == 0) dl[sb] = delta;
    });
    step_sync<TEAM>(bx.tm);   // every member has read the chart before any cell moves
    auto moved = [&](float x, float dk) {
        // linear domain: x exp2(dk), as ldexp by the integer part of dk times
        // exp2 of the rest, so that a factor beyond float32's range (dk can
        // exceed 128 when x is small) never forms on its own
        if constexpr (LIN) {
            const float k = floorf(dk);
            return __builtin_amdgcn_ldexpf(x * fast_exp2(dk - k), (int)k);
        } else {
            return x + dk;
        }
    };
    // alpha of widths 2..w0: per sentence n rows x (w0-1) widths
    {
        const int A = w0 - 1, per = n * A, total = nb * per;
        const float inv_per = 1.0f / (float)per, inv_a = 1.0f / (float)A;
        for (int f = tid; f < total; f += nt) {
            const int sb = div_small(f, per, inv_per);
            const int r = f - sb * per;
            const int i = div_small(r, A, inv_a);
            const int w = 2 + r - i * A, j = i + w;
            if (j <= n) {
                T *P = bx.chart0 + (size_t)sb * bx.cstride, *Q = P + (size_t)ld * ld;
                const float a = moved(chart_ld<TEAM>(&P[i * ld + w - 1]), dl[sb] * (float)(w - 1));
                P[i * ld + w - 1] = a;
                Q[j * ld + n + 1 - w] = a;
            }
        }
    }
    // O' of widths n-t0..n-1: spans (i, i+v) with i + (v - (n-t0)) <= t0
    if constexpr (REV) {
        const int per = (t0 + 1) * t0, total = nb * per;
        const float inv_per = 1.0f / (float)per, inv_t = 1.0f / (float)t0;
        for (int f = tid; f < total; f += nt) {
            const int sb = div_small(f, per, inv_per);
            const int r = f - sb * per;
            const int i = div_small(r, t0, inv_t);
            const int e = r - i * t0, v = n - t0 + e, j = i + v;
            if (i + e <= t0) {
                T *P = bx.chart0 + (size_t)sb * bx.cstride, *Q = P + (size_t)ld * ld;
                const float o = moved(chart_ld<TEAM>(&Q[i * ld + v]), dl[sb] * (float)(n - v));
                Q[i * ld + v] = o;
                P[j * ld + n - v] = o;
            }
        }
    }
    for (int sb = threadIdx.x; sb < nb; sb += blockDim.x) dsh[sb] += dl[sb];   // (each member's own copy)
    step_sync<TEAM>(bx.tm);
}

// The joint sweep: steps t = 1..n-1 (inside widths 2..n, outside widths
// n-1..2), one dispatch per run of steps sharing a step shape; the runs are
// cut at the rescale points (next_rescale), each phase running the fixed list
// of runs (with the short-bundle runs of 9..32 splits for bundles whose
// steps take several passes, short_bundle), so that each run and the
// rescale appear once in the code.
template <bool LIN, bool WIDE, bool IL, bool TEAM, bool MULTI = true, typename T>
__device__ __forceinline__ void io_sweep(const Bundle_ctx<T> &bx, float *dsh, float *dl) {
    const int n = bx.n;
    for (int lo = 1; lo < n;) {
        const int tr = next_rescale<LIN>(lo, n);
        const int hi = tr > 0 ? tr + 1 : n;   // steps [lo, hi)
#define CRF_IO_FIXED(LO, HI, GG, CC, MM)                              \
        if (max(lo, LO) < min(hi, HI + 1))                            \
            io_run<LIN, GG, CC, MM, IL, TEAM>(bx, max(lo, LO), min(hi, HI + 1), dsh);
        CRF_FIXED_RUNS_LOW(CRF_IO_FIXED)
        if (MULTI && !WIDE && short_bundle(bx.nb, n, (int)blockDim.x)) {
            CRF_SHORT_RUNS_MID(CRF_IO_FIXED)
        } else {
            CRF_FIXED_RUNS_MID(CRF_IO_FIXED)
        }
        CRF_FIXED_RUNS_HIGH(CRF_IO_FIXED)
#undef CRF_IO_FIXED
        for (int t = max(lo, kFixedRunsMaxK + 1); t < hi;) {
            const StepShape sh = step_shape_k(t);
            const int t2 = min(shape_run_end(t), hi);
#define CRF_IO_RUN(GG, CC, MM) io_run<LIN, GG, CC, MM, IL, TEAM>(bx, t, t2, dsh)
            CRF_DISPATCH_WIDE_SHAPE(sh, CRF_IO_RUN);
#undef CRF_IO_RUN
            t = t2;
        }
        if (tr > 0) rescale_chart<LIN, true, TEAM>(bx, tr, dsh, dl);
        lo = hi;
    }
}

// Visit every valid cell (sb, i, j), 0 <= i < j <= n, of a bundle.  Rows r
// and n-1-r of the upper triangle (n-r and r+1 cells) share one folded row
// of n+1 slots: slot q < n-r is (r, r+1+q), slot q >= n-r is (n-1-r, q).
// So a walk touches (n+1) ceil(n/2) slots per sentence instead of n^2, and
// consecutive threads take consecutive j of one row.
struct Cell {
    int sb, i, j;
    bool ok;
};
struct Cell_walk {
    int n, W, per, total;
    float inv_per, inv_w;
    __device__ Cell_walk(int nb, int n_) : n(n_), W(n_ + 1) {
        per = ((n + 1) / 2) * W;
        total = nb * per;
        inv_per = 1.0f / (float)per;
        inv_w = 1.0f / (float)W;
    }
    // Cell c of the walk; past the end (ok = false) still a valid cell.
    __device__ __forceinline__ Cell at(int c) const {
        Cell e;
        const int cc = c < total ? c : 0;
        e.sb = div_small(cc, per, inv_per);
        const int rem = cc - e.sb * per;
        const int r = div_small(rem, W, inv_w);
        const int q = rem - r * W;
        if (q < n - r) {
            e.i = r;
            e.j = r + 1 + q;
            e.ok = c < total;
        } else {
            e.i = n - 1 - r;
            e.j = q;
            e.ok = c < total && e.i > r;   // odd n: the middle row is not folded twice
        }
        return e;
    }
};

// The walk, U cells per thread at a time: the U addresses first (`addr`,
// which may read LDS tables), then the U loads together (`load`: one memory
// latency per U cells), then `use` consumes them.  The loads are
// unconditional -- at() names a cell of the bundle even past the end -- so
// that no branch separates them (a load inside a branch is waited for
// before the branch joins).
// A team's member walks its share: virtual threads t of NT.
template <int U, typename AD, typename LD, typename F>
__device__ __forceinline__ void for_cells_loaded(int nb, int n, AD &&addr, LD &&load, F &&use,
                                                 int t = threadIdx.x, int NT = blockDim.x) {
    const Cell_walk cw(nb, n);
    using A = decltype(addr(0, 0, 1));
    using V = decltype(load(addr(0, 0, 1)));
    for (int c0 = t; c0 < cw.total; c0 += NT * U) {
        A a[U];
        V v[U];
        int cell[U];   // sb << 20 | i << 10 | j (sb < 256, i, j < 1024), or -1
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const Cell e = cw.at(c0 + u * NT);
            cell[u] = e.ok ? (e.sb << 20) | (e.i << 10) | e.j : -1;
            a[u] = addr(e.sb, e.i, e.j);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = load(a[u]);
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (cell[u] >= 0) use(cell[u] >> 20, (cell[u] >> 10) & 1023, cell[u] & 1023, v[u]);
    }
}

// In-bundle label work takes a span's labels kLabBlk at a time: each block's
// loads issued together (clamped to the last label, so every load is in
// bounds) and its terms kept in registers.  Sixteen fits in what the inside
// kernels have to spare at their prologue; 32 made them spill.
constexpr int kLabBlk = 16;
// Folds labels q0 .. q0+kLabBlk-1 of a span (v) into the running max m
// (log2 units) and sum acc of its log-sum-exp.
__device__ __forceinline__ void label_block(const float *v, int q0, int L, float &m, float &acc) {
    float mb = -INFINITY;
#pragma unroll
    for (int k = 0; k < kLabBlk; ++k) mb = q0 + k < L ? fmax_nn(mb, v[k]) : mb;
    const float mn = fmax_nn(m, mb * LOG2E_F);
    acc *= fast_exp2(m - mn);   // (0 * exp2(-inf) = 0 on the first block)
#pragma unroll
    for (int k = 0; k < kLabBlk; ++k) acc += q0 + k < L ? fast_exp2(v[k] * LOG2E_F - mn) : 0.f;
    m = mn;
}
// Labels q0 .. q0+kLabBlk-1 of a span into v (clamped to the last label),
// with 8-byte loads when `wide`: an even count on an 8-byte aligned score
// tensor (every span's offset is then a multiple of 2 floats; q0 is even).
// The values at valid labels are the same either way.
__device__ __forceinline__ void label_load_blk(const float *s, int q0, int L, bool wide, float *v) {
    if (wide) {
        const float2 *s2 = reinterpret_cast<const float2 *>(s);
        const int last = L / 2 - 1;
#pragma unroll
        for (int k = 0; k < kLabBlk / 2; ++k) {
            const float2 x = s2[min(q0 / 2 + k, last)];
            v[2 * k] = x.x;
            v[2 * k + 1] = x.y;
        }
    } else {
#pragma unroll
        for (int k = 0; k < kLabBlk; ++k) v[k] = s[min(q0 + k, L - 1)];
    }
}
// The first 32 labels of a span into v (clamped), 8-byte loads when `wide`.
__device__ __forceinline__ void label_load32(const float *s, int L, bool wide, float (&v)[32]) {
    label_load_blk(s, 0, L, wide, v);
    label_load_blk(s, kLabBlk, L, wide, v + kLabBlk);
}
// Log-sum-exp (log2 units) of the L label scores of one span at s.
__device__ __forceinline__ float label_lse2(const float *s, int L, bool wide) {
    float m = -INFINITY, acc = 0.f;
    for (int q0 = 0; q0 < L; q0 += kLabBlk) {
        float v[kLabBlk];
        label_load_blk(s, q0, L, wide, v);
        label_block(v, q0, L, m, acc);
    }
    return m + fast_log2(acc);
}
// o[q] = mu exp2(s[q] log2e - lse2) for the L labels of one span, a block
// at a time.
__device__ __forceinline__ void label_marginals(const float *s, int L, bool wide, float mu, float lse2, float *o) {
    for (int q0 = 0; q0 < L; q0 += kLabBlk) {
        float v[kLabBlk];
        label_load_blk(s, q0, L, wide, v);
#pragma unroll
        for (int k = 0; k < kLabBlk; ++k)
            if (q0 + k < L) o[q0 + k] = mu * fast_exp2(v[k] * LOG2E_F - lse2);
    }
}

// Max over the L labels of one span at s (an exact float32 max), for the
// one-stage labelled CKY: blocks of 32 labels, each block's loads issued
// together (clamped to the last label).
__device__ __forceinline__ float label_max(const float *s, int L, bool wide) {
    float m = -INFINITY;
    for (int q0 = 0; q0 < L; q0 += 32) {
        float v[32];
        if (q0 == 0) {
            label_load32(s, L, wide, v);
        } else {
#pragma unroll
            for (int k = 0; k < 32; ++k) v[k] = s[min(q0 + k, L - 1)];
        }
#pragma unroll
        for (int k = 0; k < 32; ++k) m = fmax_nn(m, v[k]);   // (clamped copies repeat the last label)
    }
    return m;
}
// The lowest label attaining the max of one span's L labels (Eq. label-argmax
// with the lowest-label tie rule): blocks of 32, strict '>' in label order.
__device__ __forceinline__ int label_argmax(const float *s, int L) {
    float m = -INFINITY;
    int bl = 0;
    for (int q0 = 0; q0 < L; q0 += 32) {
        float v[32];
#pragma unroll
        for (int k = 0; k < 32; ++k) v[k] = s[min(q0 + k, L - 1)];
#pragma unroll
        for (int k = 0; k < 32; ++k)
            if (q0 + k < L && v[k] > m) {
                m = v[k];
                bl = q0 + k;
            }
    }
    return bl;
}

// ---------------------------------------------------------------------------
// Inside (+ marginals).  One workgroup per bundle (or, SPILL, per long
// sentence with its chart in the workspace).
//   REV: also compute the marginals (joint inside/outside sweep) and write them.
//   LAB: a labelled plan's bundles.  Bundles of sentences of up to
//   kLabInBundleMaxN words (kRecLab) read their label scores and take each
//   span's log-sum-exp in the prologue and write the per-label marginals in
//   the epilogue; the others run on the label log-sum-exps that
//   label_reduce_kernel wrote beforehand (see launch_inside).
// Dynamic LDS (bundled): nb charts (chart stride from inside_layout), then
// nb x {forced (f64), grad (f32), id (i32), shift (f32)}, then the room
// bundle_extra_bytes gives every bundle.
// Chart of a sentence: the rotated squares P and Q of the inside chart
// layout (ld x ld floats each).
// GOLD (with REV, unlabelled): the gold-tree CRF loss (Sec. 2.3,
//   Eq. bracket-loss) L = log Z - s(x,y) into loss[b], and in marg its
//   gradient g (p((i,j)|x) - 1[(i,j) in y]), y = the first 2n-1 rows of the
//   sentence's span list in `gold` (rows that are not spans of the sentence
//   are skipped).  Gold spans are marked in their O' mirror cell P[j][n-w],
//   which nothing reads once the sweep is done, so the epilogue subtracts g
//   once per distinct span.
constexpr int kGoldMark = 0x7FBADBAD;   // a NaN bit pattern: no finite chart value has it
//
// LIN: the sweeps run in the linear domain -- the chart holds exp2 of the
// (shifted, log2-scaled) inside and outside values, a span's sum over its
// splits is a dot product (span_dot), and rescales at doubling steps keep the
// values near 1.  A value that leaves float32's range (or a root below
// kLinMin) sets the bundle's overflow flag, and the bundle returns false
// before it has written any output: the caller then runs it again in the log
// domain (LIN = false, max-shifted log-sum-exp per span).
constexpr float kLinMin = 0x1p-100f;
template <bool LIN, bool REV, bool SPILL, bool GOLD, bool LAB>
__device__ __forceinline__ bool inside_block_impl(const KernelPlan &p, int block, const int32_t *rec, char *smem_raw,
                                                  const float *__restrict__ scores,
                                                  const float *__restrict__ grad,
                                                  float *__restrict__ logZ, float *__restrict__ marg,
                                                  const int32_t *__restrict__ gold,
                                                  float *__restrict__ loss, const Team &tm) {
    static_assert(!GOLD || REV, "the gold-tree loss needs the marginals");
    static_assert(!LAB || (!SPILL && !GOLD), "label I/O is for labelled bundles in LDS");
    __shared__ int lin_ovf;
    __shared__ double spill_forced[1];
    __shared__ float spill_gv[1];
    __shared__ int spill_id[1];
    __shared__ float spill_dsh[1];
    const int NT = blockDim.x;
    const int tid = threadIdx.x;
    const int N1 = p.n1;

    int n, nb;
    float *chart0;
    int cstride;
    double *forced;
    float *gv, *dsh;
    int *sid;
    InsideLayout lay;
    uint32_t mnb = 0;   // div_magic(nb)
    if constexpr (SPILL) {
        const int b = p.inside.order_spill[block];
        n = p.len[b];
        nb = 1;
        chart0 = reinterpret_cast<float *>(p.ws + p.inside.ws_off[block]);
        lay = inside_layout(n, 1, true);
        lay.e = 5;   // a workspace chart: no banks, spans side by side
        cstride = 0;
        forced = spill_forced;
        gv = spill_gv;
        sid = spill_id;
        dsh = spill_dsh;
        if (tid == 0) sid[0] = b;
    } else {
        // the record's ids are fetched with its header (a bundle holds at
        // most kMaxBundle <= blockDim.x sentences)
        const int id0 = tid < p.rec_stride - kRecHeader ? rec[kRecHeader + tid] : 0;
        n = rec[kRecN];
        nb = rec[kRecCount];
        lay = InsideLayout{rec[kRecLd], rec[kRecCs], rec[kRecE]};
        mnb = (uint32_t)rec[kRecMagic];
        chart0 = reinterpret_cast<float *>(smem_raw);
        cstride = lay.cs;
        forced = reinterpret_cast<double *>(smem_raw + inside_tables_offset(nb, lay.cs));
        gv = reinterpret_cast<float *>(forced + nb);
        sid = reinterpret_cast<int *>(gv + nb);
        dsh = reinterpret_cast<float *>(sid + nb);
        if (tid < nb) sid[tid] = id0;
    }
    const int ld = lay.ld;
    const Bundle_ctx<float> bx{chart0, cstride, n, ld, nb, mnb, lay.e, LIN ? &lin_ovf : nullptr, tm};
    const bool coh = SPILL && tm.k > 1;   // a team's chart reads (chart_ld)
    if (tid == 0) lin_ovf = 0;
    __syncthreads();
    // (gv holds the rescales' per-sentence shifts during the sweep and the
    // upstream gradients after it)
    for (int t = tid; t < nb; t += NT) dsh[t] = 0.f;

    const size_t row_stride = (size_t)N1;
    const size_t sent_stride = (size_t)N1 * row_stride;

    // Prologue: scores of every valid cell into the charts (log2-scaled, in
    // the cells of alpha and, for the outside, of O'); forced spans get 0 in
    // alpha (1 in the linear domain) and park their natural-unit score.
    auto score_at = [&](int sb, int i, int j) -> const float * {
        return scores + (size_t)sid[sb] * sent_stride + (size_t)i * row_stride + (size_t)j;
    };
    auto load_score = [](const float *q) -> float { return *q; };
    // (cells of the rotated P / Q squares, see the inside chart layout)
    auto put_score = [&](int sb, int i, int j, float s) {
        float *P = chart0 + (size_t)sb * cstride, *Q = P + (size_t)ld * ld;
        const int w = j - i;
        const float zero = LIN ? 1.f : 0.f;   // log2 value 0
        if (w == 1) {   // forced: alpha 0, score parked in the O' cell no sweep uses
            P[i * ld] = zero;
            Q[j * ld + n] = zero;
            P[j * ld + n - 1] = s;
        } else if (i == 0 && j == n) {   // the root: own term 0 (a log2 score), O' 0, score parked
            P[n - 1] = 0.f;
            P[n] = s;
            if constexpr (REV) {
                Q[n] = zero;
                P[n * ld] = zero;
            }
        } else {
            const float s2 = s * LOG2E_F;
            P[i * ld + w - 1] = s2;
            if constexpr (REV) P[j * ld + n - w] = s2;
        }
    };
    // A labelled bundle that does its own label I/O (kRecLab) reads each
    // span's labels and takes their log-sum-exp (Sec. 4.2, Eq.
    // tree-label-score: the span's score in the one-stage Z); the others
    // read the [B][N1][N1] scores (the label passes' log-sum-exps for a
    // labelled plan).  Only the LAB build holds this code: its register
    // blocks would otherwise raise every other kernel's register pressure.
    const bool lab = LAB && rec[kRecLab] != 0;   // (uniform)
    const int L = p.lab_L;
    const size_t lab_sent = (size_t)N1 * N1 * (size_t)L;
    auto lab_at = [&](int sb, int i, int j) -> const float * {
        return p.lab_s4 + (size_t)sid[sb] * lab_sent + ((size_t)i * N1 + (size_t)j) * (size_t)L;
    };
    const bool wide_in = (L & 1) == 0 && ((uintptr_t)p.lab_s4 & 7) == 0;   // 8-byte label loads
    auto lab_lse = [&](const float *q) -> float { return label_lse2(q, L, wide_in) * (float)LN2_D; };
    if constexpr (LAB) {
        if (lab)
            for_cells_loaded<1>(nb, n, lab_at, lab_lse, put_score);
        else
            for_cells_loaded<8>(nb, n, score_at, load_score, put_score);
    } else {
        for_cells_loaded<8>(nb, n, score_at, load_score, put_score, team_tid<SPILL>(tm), team_nt<SPILL>(tm));
    }
    step_sync<SPILL>(tm);
    // Forced-span sums, a lane group per sentence, fixed order (deterministic).
    // The linear domain also seeds each sentence's shift d from its scores:
    // for independent scores of mean m and variance v (log2 units) the
    // expected tree weight grows by 4 (Catalan) times E[exp2(s)] =
    // exp2(m + v ln2 / 2) per node, so d = -(m + v ln2 / 2 + 2), from the
    // non-forced spans of widths 2..9 (near-forbidden scores left out); the
    // rescales then correct it from the chart itself.
    by_sentence_groups(n, nb, [&](auto gs, int sb, int gl, bool valid) {
        constexpr int GS = decltype(gs)::value;
        const float *P = chart0 + (size_t)sb * cstride;
        double acc = 0.0;
        for (int i = gl; i < n; i += GS) acc += (double)chart_ld_if(&P[(i + 1) * ld + n - 1], coh);
        if (gl == 0 && n >= 2) acc += (double)chart_ld_if(&P[n], coh);
        acc = grp_sum_d<GS>(acc);
        if (valid && gl == 0) forced[sb] = acc;
        if constexpr (LIN) {
            float s1 = 0.f, s2 = 0.f, c = 0.f;
            for (int i = gl; i < n - 1; i += GS)
                for (int w = 2; w <= 9 && i + w <= n; ++w) {
                    if (i == 0 && w == n) continue;   // the root: forced
                    const float x = chart_ld_if(&P[i * ld + w - 1], coh);
                    if (x > -1000.f) {
                        s1 += x;
                        s2 += x * x;
                        c += 1.f;
                    }
                }
            s1 = grp_sum<GS>(s1);
            s2 = grp_sum<GS>(s2);
            c = grp_sum<GS>(c);
            if (valid && gl == 0 && c > 0.f) {
                const float mean = s1 / c, var = fmaxf(s2 / c - mean * mean, 0.f);
                dsh[sb] = -(mean + 0.5f * (float)LN2_D * var + 2.0f);
            }
        }
    });
    if constexpr (LIN) __syncthreads();   // the seeds are read by the first step

    // Workspace charts lay spans side by side; LDS charts interleave them
    // when their layout allows (e = 0).
    if constexpr (!REV) {
        if constexpr (SPILL) {
            if (tm.k > 1) fwd_sweep<LIN, true, false, true>(bx, dsh, gv);
            else fwd_sweep<LIN, true, false, false>(bx, dsh, gv);
        } else if (lay.e == 0) fwd_sweep<LIN, false, true, false, !LAB>(bx, dsh, gv);
        else fwd_sweep<LIN, false, false, false, !LAB>(bx, dsh, gv);
    } else {
        if constexpr (SPILL) {
            if (tm.k > 1) io_sweep<LIN, true, false, true>(bx, dsh, gv);
            else io_sweep<LIN, true, false, false>(bx, dsh, gv);
        } else if (lay.e == 0) io_sweep<LIN, false, true, false, !LAB>(bx, dsh, gv);
        else io_sweep<LIN, false, false, false, !LAB>(bx, dsh, gv);
    }
    // (the sweep's last barrier published the chart and the flag)
    if constexpr (LIN) {
        for (int sb = tid; sb < nb; sb += NT) {
            const float r = chart_ld_if(&chart0[(size_t)sb * cstride + n - 1], coh);
            if (!(r >= kLinMin && r <= kLinMax)) lin_ovf = 1;
        }
        __syncthreads();
        if constexpr (SPILL) {
            if (tm.k > 1) {
                // One decision for the team: a member that saw a value
                // leave the range raises the team's word to this job + 1
                // (later jobs raise it only after this barrier's readers
                // are done, so the word needs no clearing).
                int32_t *fl = tm.line + 1;
                if (tid == 0 && lin_ovf) atomicMax(fl, tm.job + 1);
                team_sync(tm);
                if (tid == 0 && load_coherent(fl) > tm.job) lin_ovf = 1;
                __syncthreads();
            }
        }
        if (lin_ovf) return false;   // nothing written yet: the log domain redoes the bundle
    }
    for (int t = tid; t < nb; t += NT) gv[t] = grad ? grad[sid[t]] : 1.0f;
    __syncthreads();
    // log Z = (alpha~(0,n) - (n-2) d) ln 2 + forced sum, alpha~(0,n) the
    // root's log2 value.
    auto log_z = [&](int sb) {
        const float r = chart_ld_if(&chart0[(size_t)sb * cstride + n - 1], coh);
        const double lr = LIN ? log2_split(r) : (double)r;
        const double z2 = lr - (double)dsh[sb] * (n >= 2 ? n - 2 : 0);
        return z2 * LN2_D + forced[sb];
    };
    if (logZ != nullptr && tm.rank == 0) {
        const bool aborted = SPILL && team_aborted(tm);
        for (int sb = tid; sb < nb; sb += NT)
            logZ[sid[sb]] = aborted ? __builtin_bit_cast(float, 0x7fc00000) : (float)log_z(sb);
    }
    if constexpr (!REV) return true;

    if constexpr (GOLD) {
        // Gold rows of each sentence: mark the span, sum its score (float64,
        // a lane group per sentence in a fixed order), loss = log Z - sum.
        // (a team's first member marks and sums)
        const int R = 2 * (N1 - 1) - 1, rows = 2 * n - 1;
        if (tm.rank == 0) by_sentence_groups(rows, nb, [&](auto gs, int sb, int gl, bool valid) {
            constexpr int GS = decltype(gs)::value;
            float *P = chart0 + (size_t)sb * cstride;
            const int32_t *g2 = gold + (size_t)sid[sb] * R * 2;
            double acc = 0.0;
            for (int r = gl; r < rows; r += GS) {
                const int i = g2[2 * r], j = g2[2 * r + 1];
                if (0 <= i && i < j && j <= n) {
                    acc += (double)*score_at(sb, i, j);
                    if (valid) P[j * ld + n - (j - i)] = __builtin_bit_cast(float, kGoldMark);
                }
            }
            acc = grp_sum_d<GS>(acc);
            if (valid && gl == 0) loss[sid[sb]] = (float)(log_z(sb) - acc);
        });
        step_sync<SPILL>(tm);
    }

    // Epilogue: marginals of the valid cells (coalesced stores along rows),
    //   mu(i,j) = g exp2(alpha~(i,j) + O'(i,j) - (s(i,j) + d) - alpha~(0,n)),
    // and exactly g on forced spans.
    // mu of a valid cell whose own score (log2 units) is own2
    auto lg = [](float x) {   // a chart value as its log2 value
        if constexpr (LIN) return fast_log2(x);   // (0 gives -inf, and exp2 of the exponent 0)
        else return x;
    };
    auto span_mu = [&](int sb, int i, int j, float own2) {
        const float *P = chart0 + (size_t)sb * cstride, *Q = P + (size_t)ld * ld;
        const bool forced_span = (j == i + 1) || (i == 0 && j == n);
        const int w = j - i;
        float mu = gv[sb];
        if (!forced_span)
            mu *= fast_exp2(((lg(chart_ld_if(&P[i * ld + w - 1], coh)) - lg(chart_ld_if(&P[n - 1], coh))) +
                             lg(chart_ld_if(&Q[i * ld + w], coh))) - (own2 + dsh[sb]));
        if constexpr (GOLD)
            if (__builtin_bit_cast(int, chart_ld_if(&P[j * ld + n - w], coh)) == kGoldMark) mu -= gv[sb];
        return mu;
    };
    if constexpr (LAB) if (lab) {
        // per-label marginals mu(i,j) exp(s(i,j,l) - s'(i,j)).  Up to 32
        // labels: one load of a span's labels serves its log-sum-exp (the
        // prologue's blocks and arithmetic, so the same own score as the
        // chart's) and its outputs.
        float *const out0 = p.lab_out;
        const bool wide_out = wide_in && ((uintptr_t)out0 & 7) == 0;
        if (L <= 2 * kLabBlk) {
            const Cell_walk cw(nb, n);
            for (int c = tid; c < cw.total; c += NT) {
                const Cell e = cw.at(c);
                const float *q = lab_at(e.sb, e.i, e.j);
                float v[2 * kLabBlk];
                label_load32(q, L, wide_in, v);
                __builtin_amdgcn_sched_barrier(0);
                float m = -INFINITY, acc = 0.f;
                label_block(v, 0, L, m, acc);
                if (L > kLabBlk) label_block(v + kLabBlk, kLabBlk, L, m, acc);
                const float own2 = ((m + fast_log2(acc)) * (float)LN2_D) * LOG2E_F;   // as the chart holds it
                const float mu = span_mu(e.sb, e.i, e.j, own2);
                if (!e.ok) continue;
                float *o = out0 + (q - p.lab_s4);
                if (wide_out) {   // 8-byte stores
                    float2 *o2 = reinterpret_cast<float2 *>(o);
#pragma unroll
                    for (int k = 0; k < kLabBlk; ++k)
                        if (2 * k < L)
                            o2[k] = make_float2(mu * fast_exp2(v[2 * k] * LOG2E_F - own2),
                                                mu * fast_exp2(v[2 * k + 1] * LOG2E_F - own2));
                } else {
#pragma unroll
                    for (int k = 0; k < 2 * kLabBlk; ++k)
                        if (k < L) o[k] = mu * fast_exp2(v[k] * LOG2E_F - own2);
                }
            }
        } else {
            for_cells_loaded<1>(nb, n, lab_at, lab_lse, [&](int sb, int i, int j, float s) {
                const float *q = lab_at(sb, i, j);
                label_marginals(q, L, wide_in, span_mu(sb, i, j, s * LOG2E_F), s * LOG2E_F, out0 + (q - p.lab_s4));
            });
        }
        return true;
    }
    for_cells_loaded<8>(
        nb, n, score_at, load_score,
        [&](int sb, int i, int j, float s) {
            marg[(size_t)sid[sb] * sent_stride + (size_t)i * row_stride + j] = span_mu(sb, i, j, s * LOG2E_F);
        },
        team_tid<SPILL>(tm), team_nt<SPILL>(tm));
    return true;
}

// A bundle (or a workspace sentence): the linear-domain sweeps, and the log
// domain if they leave float32's range (see inside_block_impl).
template <bool REV, bool SPILL, bool GOLD = false, bool LAB = false>
__device__ __forceinline__ void inside_block(const KernelPlan &p, int block, const int32_t *rec, char *smem_raw,
                                             const float *__restrict__ scores,
                                             const float *__restrict__ grad,
                                             float *__restrict__ logZ, float *__restrict__ marg,
                                             const int32_t *__restrict__ gold = nullptr,
                                             float *__restrict__ loss = nullptr, const Team &tm = Team{}) {
    if (inside_block_impl<true, REV, SPILL, GOLD, LAB>(p, block, rec, smem_raw, scores, grad, logZ, marg, gold, loss,
                                                       tm))
        return;
    __syncthreads();   // every thread has left the linear attempt
    inside_block_impl<false, REV, SPILL, GOLD, LAB>(p, block, rec, smem_raw, scores, grad, logZ, marg, gold, loss, tm);
}

// ---------------------------------------------------------------------------
// CKY.  Each sentence's chart is one float64 square (beta upper + mirror);
// its split table (entries SP: uint8_t for bundles, uint16_t on the
// workspace kernel) follows the chart or sits in the workspace.
template <typename SP>
struct Cky_ctx {
    char *chart0;
    int cstride;   // bytes between consecutive sentences' charts
    char *split0;
    int sstride;   // bytes between consecutive sentences' split tables
    int n, ld, nb;
    uint32_t mnb;     // div_magic(nb)
    bool split_lds;   // split tables in LDS (else in global memory)
    Team tm;          // workspace sentences: the team running the pass
    __device__ double *beta(int sb) const {   // (sb < 256, cstride < 2^24)
        return reinterpret_cast<double *>(chart0 + __umul24((uint32_t)sb, (uint32_t)cstride));
    }
    // Split table entry e of sentence sb, through an LDS or a global pointer
    // (not a generic one: flat accesses cost more, and a flat store to LDS
    // holds up the next barrier).
    __device__ void put_split(int sb, int e, int v) const {
        if (split_lds) {   // 32-bit LDS address arithmetic
            const uint32_t a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)split0 +
                               __umul24((uint32_t)sb, (uint32_t)sstride) + (uint32_t)e * sizeof(SP);
            *(__attribute__((address_space(3))) SP *)(uintptr_t)a = (SP)v;
        } else {
            SP *q = reinterpret_cast<SP *>(split0 + (size_t)sb * sstride) + e;
            *(__attribute__((address_space(1))) SP *)q = (SP)v;
        }
    }
    __device__ int get_split(int sb, int e, bool coherent = false) const {
        if (split_lds) {
            const uint32_t a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)split0 +
                               __umul24((uint32_t)sb, (uint32_t)sstride) + (uint32_t)e * sizeof(SP);
            return (int)*(const __attribute__((address_space(3))) SP *)(uintptr_t)a;
        }
        const SP *q = reinterpret_cast<const SP *>(split0 + (size_t)sb * sstride) + e;
        if (coherent) return (int)chart_ld<true>(q);
        return (int)*(const __attribute__((address_space(1))) SP *)q;
    }
};

// Max of x[LO .. LO+N) and the first index attaining it (as (c0 + c) * G),
// paired as a balanced tree.  Indices are template constants, so no select
// ever picks between array slots (the compiler would then index the array
// dynamically).
struct Arg_max {
    double v;
    int k;
};
template <int LO, int N>
__device__ __forceinline__ Arg_max tree_arg_max(const double *x, int c0, int G) {
    if constexpr (N == 1) {
        return Arg_max{x[LO], (c0 + LO) * G};
    } else {
        constexpr int H = (N + 1) / 2;
        const Arg_max a = tree_arg_max<LO, H>(x, c0, G), b = tree_arg_max<LO + H, N - H>(x, c0, G);
        return Arg_max{fmax(a.v, b.v), b.v > a.v ? b.k : a.k};
    }
}

// One width: float64 max-plus, beta(i,j) = (max_k fl(beta(i,k) + beta(k,j)))
// + s(i,j), and the lowest k attaining the max into the split table (entry
// sp0 + i).  Each lane keeps its running max and the first of its terms to
// reach it; the group then takes the lowest split among its lanes at the
// group's max.
template <int G, int C, int MF, bool IL, bool TEAM, typename SP>
__device__ __forceinline__ void cky_step(const Cky_ctx<SP> &cx, int w, int sp0) {
    const int tid = team_tid<TEAM>(cx.tm), nt = team_nt<TEAM>(cx.tm);
    const int n = cx.n, ld = cx.ld;
    const int K = w - 1, nsp = cx.nb * (n - w + 1);
    const int total = region_lanes<G, IL, 16>(nsp);
    const int wq0 = __builtin_amdgcn_readfirstlane(tid & ~63);
    for (int f0 = 0; f0 < total; f0 += nt) {
        if (f0 + wq0 >= total) break;
        if (!wave_has_span<G, IL, 16>(f0 + wq0, nsp)) continue;
        const Lane_at at = lane_at<G, IL, 16>(f0 + tid, nsp, cx.nb, cx.mnb);
        const int i = at.i, l = at.l;
        double *be = cx.beta(at.sb);
        // every index from the diagonal cell [i][i] and the uniform w * ld
        const int rb = (int)__umul24((uint32_t)i, (uint32_t)(ld + 1));   // [i][i]
        const int cb = rb + (int)__umul24((uint32_t)w, (uint32_t)ld);    // [j][i]
        const int rowo = rb + 1 + l, colo = cb + 1 + l;
        const double sij = chart_ld<TEAM>(&be[rb + w]);
        const int kl = K - l;
        // Terms in chunks of 16 (the last one shorter).  Up to 16 splits per
        // lane (one chunk), every float64 operand is loaded before the first
        // is used; longer lanes interleave loads and arithmetic.  A chunk's
        // max and its lowest term at the max pair up as a tree; chunks merge
        // in order.
        double m = -INFINITY;
        int kc = 0;   // this lane's first term at its max, as c * G
        auto chunk = [&](auto c0_c, auto n_c) {
            constexpr int c0 = decltype(c0_c)::value, CN = decltype(n_c)::value;
            double xr[CN], xc[CN];
#pragma unroll
            for (int c = 0; c < CN; ++c) {
                xr[c] = chart_ld<TEAM>(&be[rowo + (c0 + c) * G]);
                xc[c] = chart_ld<TEAM>(&be[colo + (c0 + c) * G]);
            }
            if constexpr (C <= 16) __builtin_amdgcn_sched_barrier(0);
            double x[CN];
#pragma unroll
            for (int c = 0; c < CN; ++c) {
                x[c] = xr[c] + xc[c];
                // a split past the span's last: the high word alone makes it
                // about -1.8e308, below any chart value (one select, not two)
                if (c0 + c >= MF) {
                    const uint64_t u = __builtin_bit_cast(uint64_t, x[c]);
                    const uint32_t hi = (c0 + c) * G >= kl ? 0xFFEFFFFFu : (uint32_t)(u >> 32);
                    x[c] = __builtin_bit_cast(double, ((uint64_t)hi << 32) | (uint32_t)u);
                }
            }
            const Arg_max a = tree_arg_max<0, CN>(x, c0, G);
            if constexpr (c0 == 0) {
                m = a.v;
                kc = a.k;
            } else {
                kc = a.v > m ? a.k : kc;
                m = fmax(m, a.v);
            }
        };
        static_assert(C <= 48, "at most three chunks");
        chunk(std::integral_constant<int, 0>{}, std::integral_constant<int, (C < 16 ? C : 16)>{});
        if constexpr (C > 16) chunk(std::integral_constant<int, 16>{}, std::integral_constant<int, (C < 32 ? C - 16 : 16)>{});
        if constexpr (C > 32) chunk(std::integral_constant<int, 32>{}, std::integral_constant<int, C - 32>{});
        const double mg = grp_max_d<G>(m);
        const int kb = min(grp_min_i<G>(m == mg ? kc + l : 0x7fffffff), K - 1);
        const double v = mg + sij;
        asm volatile("" ::"v"(v));   // keeps the score load with the operand loads
        if (at.act && l == 0) {
            be[rb + w] = v;
            be[cb] = v;
            cx.put_split(at.sb, sp0 + i, kb);
        }
    }
}

template <int G, int C, int MF, bool IL, bool TEAM, typename SP>
__device__ __forceinline__ void cky_run(const Cky_ctx<SP> &cx, int w0, int w1) {
    for (int w = w0; w < w1; ++w) {
        cky_step<G, C, MF, IL, TEAM>(cx, w, cky_split_index(cx.n, w, 0));
        step_sync<TEAM>(cx.tm);
    }
}

template <bool WIDE, bool IL, bool TEAM, typename SP>
__device__ __forceinline__ void cky_sweep(const Cky_ctx<SP> &cx) {
    const int n = cx.n;
#define CRF_CKY_FIXED(LO, HI, GG, CC, MM) \
    if (n >= LO + 1) cky_run<GG, CC, MM, IL, TEAM>(cx, LO + 1, min(HI + 2, n + 1));
    CRF_CKY_FIXED_RUNS(CRF_CKY_FIXED)
#undef CRF_CKY_FIXED
    for (int w = kFixedRunsMaxK + 2; w <= n;) {
        const StepShape sh = step_shape_k(w - 1);
        const int w2 = min(shape_run_end(w - 1) + 1, n + 1);
#define CRF_CKY_RUN(GG, CC, MM) cky_run<GG, CC, MM, IL, TEAM>(cx, w, w2)
        CRF_DISPATCH_WIDE_SHAPE(sh, CRF_CKY_RUN);
#undef CRF_CKY_RUN
        w = w2;
    }
}

// Order one wavefront's LDS accesses across its lanes.
template <typename SP>
__device__ __forceinline__ int split_of(const Cky_ctx<SP> &cx, int sb, int i, int j) {
    return i + 1 + cx.get_split(sb, cky_split_index(cx.n, j - i, i), cx.tm.k > 1);
}

// Write the trees of all the bundle's sentences in preorder (the 2n-1 rows
// of each sentence's spans output), one lane per word p of a sentence.  A
// node (i, j) at row r with split k has its left child (i, k) at row r + 1
// and its right child (k, j) at row r + 2(k - i) (a subtree of m words
// holds 2m - 1 nodes).  Every node has one leftmost word; lane p walks down
// from the root towards word p, following the split table and counting
// rows, and writes the nodes whose leftmost word is p: once the walk reaches
// a node starting at p, that node and its chain of left children down to
// the word itself.  So each row is written once, and a lane's chain of
// split lookups is as long as its word's depth.
// With labels (one-stage labelled decoding), every node written also gets
// the lowest of its span's best labels, from the [B][N1][N1][L] scores s4.
template <bool LAB, typename SP>
__device__ void walk_trees(const Cky_ctx<SP> &cx, const int *sid, int32_t *spans, int R, int32_t *labels,
                           const float *s4, int N1, int L) {
    const int n = cx.n, total = cx.nb * n;
    const float inv_n = 1.0f / (float)n;
    for (int t = threadIdx.x; t < total; t += blockDim.x) {
        const int sb = div_small(t, n, inv_n), p = t - sb * n;
        int2 *out = reinterpret_cast<int2 *>(spans + (size_t)sid[sb] * R * 2);
        int32_t *lab = LAB ? labels + (size_t)sid[sb] * R : nullptr;
        const float *sent = LAB ? s4 + (size_t)sid[sb] * N1 * N1 * L : nullptr;
        int i = 0, j = n, row = 0;
        // (every split k lies in (i, j), so each pass moves i up or j down;
        // the pass bounds only guard against a corrupt table)
        for (int it = 0; i < p && it < n; ++it) {   // i < p < j: a node not starting at p
            const int k = split_of(cx, sb, i, j);
            if (p < k) {
                ++row;
                j = k;
            } else {
                row += 2 * (k - i);
                i = k;
            }
        }
        for (int it = 0; it < n; ++it) {
            out[row] = make_int2(i, j);
            if constexpr (LAB) lab[row] = label_argmax(sent + ((size_t)i * N1 + j) * L, L);
            if (j - i < 2) break;
            j = split_of(cx, sb, i, j);
            ++row;
        }
    }
}

// LAB: labelled scores [B][N1][N1][L]; each span's score is its best label's
// (an exact max), and the tree's spans get their best labels (one-stage
// labelled decoding, Sec. 4.2, Eq. tree-label-score).  second: take the chart
// layout from the record's second layout (an MBR bundle's CKY chart).
template <bool SPILL, bool LAB = false>
__device__ __forceinline__ void cky_block(const KernelPlan &p, int block, const int32_t *rec, char *smem_raw,
                                          const float *__restrict__ scores,
                                          int32_t *__restrict__ spans, float *__restrict__ best,
                                          int32_t *__restrict__ labels = nullptr, bool second = false,
                                          const Team &tm = Team{}) {
    __shared__ int spill_id[1];
    const int NT = blockDim.x;
    const int tid = threadIdx.x;
    const int N1 = p.n1;
    const int L = LAB ? p.L : 1;

    int n, nb, *sid;
    char *chart0, *split0;
    int cstride, sstride;
    bool split_lds = false;
    CkyLayout lay;
    uint32_t mnb = 0;   // div_magic(nb)
    if constexpr (SPILL) {
        const int b = p.cky.order_spill[block];
        n = p.len[b];
        nb = 1;
        lay = CkyLayout{cky_ld(n), 0, 5};   // a workspace chart: no banks, spans side by side
        chart0 = p.ws + p.cky.ws_off[block];
        cstride = 0;
        split0 = chart0 + (size_t)8 * lay.ld * lay.ld;
        sstride = 0;
        sid = spill_id;
        if (tid == 0) sid[0] = b;
    } else {
        const int id0 = tid < p.rec_stride - kRecHeader ? rec[kRecHeader + tid] : 0;
        n = rec[kRecN];
        nb = rec[kRecCount];
        const int split_ws = rec[kRecSplitWs];
        split_lds = split_ws < 0;
        lay = second ? CkyLayout{rec[kRecLd2], rec[kRecCs2], rec[kRecE2]} : CkyLayout{rec[kRecLd], rec[kRecCs], rec[kRecE]};
        mnb = (uint32_t)rec[kRecMagic];
        chart0 = smem_raw;
        cstride = lay.cs;
        split0 = split_lds ? chart0 + (size_t)8 * lay.ld * lay.ld : p.ws + (size_t)split_ws * 256;
        sstride = split_lds ? cstride : (int)cky_split_count(n);
        sid = reinterpret_cast<int *>(smem_raw + (size_t)nb * cstride);
        if (tid < nb) sid[tid] = id0;
    }
    const int ld = lay.ld;
    typedef typename std::conditional<SPILL, uint16_t, uint8_t>::type SP;
    const Cky_ctx<SP> cx{chart0, cstride, split0, sstride, n, ld, nb, mnb, !SPILL && split_lds, tm};
    const bool coh = SPILL && tm.k > 1;   // a team's chart reads (chart_ld)
    __syncthreads();

    auto score_at = [&](int sb, int i, int j) -> const float * {
        return scores + (((size_t)sid[sb] * N1 + i) * N1 + j) * L;
    };
    const bool wide_in = LAB && (L & 1) == 0 && ((uintptr_t)scores & 7) == 0;
    auto load_score = [&](const float *q) -> float {
        if constexpr (LAB) return label_max(q, L, wide_in);
        else return *q;
    };
    auto put_score = [&](int sb, int i, int j, float sf) {
        double *be = cx.beta(sb);
        const double s = (double)sf;
        be[i * ld + j] = s;
        if (j == i + 1) be[j * ld + i] = s;
    };
    for_cells_loaded<LAB ? 1 : 8>(nb, n, score_at, load_score, put_score, team_tid<SPILL>(tm), team_nt<SPILL>(tm));
    step_sync<SPILL>(tm);
    // Workspace charts lay spans side by side; LDS charts interleave them
    // when their layout allows (e = 0).
    if constexpr (SPILL) {
        if (tm.k > 1) cky_sweep<true, false, true>(cx);
        else cky_sweep<true, false, false>(cx);
    } else if (lay.e == 0) cky_sweep<false, true, false>(cx);
    else cky_sweep<false, false, false>(cx);
    if (tm.rank != 0) return;   // a team's first member writes the outputs

    const int R = 2 * (N1 - 1) - 1;
    const int pad_rows = R - (2 * n - 1);   // rows past the tree are -1
    if (pad_rows > 0) {
        const float inv_pad = 1.0f / (float)pad_rows;
        for (int c = tid; c < nb * pad_rows; c += NT) {
            const int sbb = div_small(c, pad_rows, inv_pad);
            const int r = 2 * n - 1 + (c - sbb * pad_rows);
            int32_t *o = spans + ((size_t)sid[sbb] * R + r) * 2;
            o[0] = -1;
            o[1] = -1;
            if constexpr (LAB) labels[(size_t)sid[sbb] * R + r] = -1;
        }
    }
    if (best != nullptr) {
        const bool aborted = SPILL && team_aborted(tm);
        for (int sb = tid; sb < nb; sb += NT)
            best[sid[sb]] = aborted ? __builtin_bit_cast(float, 0x7fc00000) : (float)chart_ld_if(&cx.beta(sb)[n], coh);
    }
    // (the sweep's last barrier published the splits)
    walk_trees<LAB>(cx, sid, spans, R, labels, scores, N1, L);
}

// Workgroups of 256, 512 or 1024 threads (the plan's choice) share one
// build of each kernel.  LAB: the labelled plans' bundle kernel, whose
// bundles marked kRecLab read and write their own label scores.
template <bool REV, bool SPILL, bool LAB = false, bool TEAM = false>
__global__ __launch_bounds__(kThreadsMax) void inside_kernel(KernelPlan p, const float *__restrict__ scores,
                                                             const float *__restrict__ grad,
                                                             float *__restrict__ logZ,
                                                             float *__restrict__ marg) {
    extern __shared__ __align__(16) char smem_raw[];
    if constexpr (SPILL && !TEAM) {
        inside_block<REV, true, false, LAB>(p, blockIdx.x, nullptr, smem_raw, scores, grad, logZ, marg);
    } else if constexpr (SPILL) {
        Team tm;
        int job, stride;
        if (!spill_jobs(p, tm, job, stride)) return;
        for (; job < p.inside.n_spill; job += stride, ++tm.job) {
            inside_block<REV, true, false, LAB>(p, job, nullptr, smem_raw, scores, grad, logZ, marg, nullptr, nullptr,
                                                tm);
            __syncthreads();
        }
    } else
        inside_block<REV, false, false, LAB>(p, blockIdx.x, p.inside.recs + (size_t)blockIdx.x * p.rec_stride,
                                             smem_raw, scores, grad, logZ, marg);
}

// Labelled scores [B][N1][N1][L] of the sentences whose bundles leave their
// label work to these passes (longer than kLabInBundleMaxN words, or with
// their chart in the workspace), spread over the whole chip.
// label_reduce_kernel writes each valid cell's label log-sum-exp
// s'(i,j) = log sum_l exp s(i,j,l) (Sec. 4.2, Eq. tree-label-score: the
// one-stage Z sums exp of the labelled score over labels per span) into sp
// [B][N1][N1]; the unlabelled kernels then run on sp; label_expand_kernel
// writes the per-label marginals mu(i,j) exp(s(i,j,l) - s'(i,j)) from their
// marginals mu [B][N1][N1].  Only valid cells are read or written.
// Both passes run over the contiguous label blocks of the rows: row i of
// sentence b holds the labels of cells (i, i+1..n) back to back, and a
// wavefront takes a chunk of at most kLabelRowChunk consecutive floats of one
// row (p.lab_rows: sentence, row, first float), its lanes on consecutive
// floats, so that every global access is a whole cache line, and every load
// of a chunk is issued before the first use (a chunk is a few hundred floats:
// serial round trips to memory, not bandwidth, would bound it otherwise).
constexpr int kLabelWaves = kLabelChunk / 64;          // chunks per workgroup, a wavefront each
constexpr int kLabelPer = kLabelRowChunk / 64;         // floats of a chunk per lane
struct Label_row {
    size_t cell0;   // the row's first cell (i, i+1)
    int f0, len;    // the chunk's first float, the row block's floats
};
__device__ __forceinline__ bool label_row(const KernelPlan &p, int r, Label_row *o) {
    if (r >= p.n_lab_rows) return false;
    const int4 rc = reinterpret_cast<const int4 *>(p.lab_rows)[r];   // (sentence, row, first float)
    const int N1 = p.n1, n = p.len[rc.x], i = rc.y;
    o->cell0 = ((size_t)rc.x * N1 + i) * N1 + i + 1;
    o->f0 = rc.z;
    o->len = (n - i) * p.L;
    return true;
}

// The reduction stages the cells that start in its chunk (their labels run
// up to L - 1 floats past it) in LDS, then folds a cell per lane from there:
// the max, then the sum of exp2 of the shifted terms, label by label.
__global__ __launch_bounds__(kLabelChunk) void label_reduce_kernel(KernelPlan p, const float *__restrict__ s4,
                                                                   float *__restrict__ sp) {
    extern __shared__ float lab_stage[];   // kLabelWaves x (kLabelRowChunk + L) floats
    const int wave = (int)threadIdx.x >> 6, lane = (int)threadIdx.x & 63, L = p.L;
    float *stage = lab_stage + wave * (kLabelRowChunk + L);
    Label_row rw{};
    int c0 = 0, c1 = 0;
    if (label_row(p, (int)blockIdx.x * kLabelWaves + wave, &rw)) {
        c0 = (rw.f0 + L - 1) / L;                                     // first cell starting in the chunk
        c1 = min((rw.f0 + kLabelRowChunk - 1) / L + 1, rw.len / L);   // one past the last
        const int a = c0 * L, e = c1 * L;                             // its floats, e - a < kLabelRowChunk + L
        const float *src = s4 + rw.cell0 * L;
        for (int base = a; base < e; base += 64 * kLabelPer) {
            float v[kLabelPer];
#pragma unroll
            for (int k = 0; k < kLabelPer; ++k) v[k] = src[min(base + 64 * k + lane, e - 1)];
#pragma unroll
            for (int k = 0; k < kLabelPer; ++k)
                if (base + 64 * k + lane < e) stage[base + 64 * k + lane - a] = v[k];
        }
    }
    __syncthreads();
    for (int c = c0 + lane; c < c1; c += 64) {
        const float *row = stage + (c - c0) * L;
        float m = -INFINITY;
        for (int k = 0; k < L; ++k) m = fmax_nn(m, row[k]);
        const float m2 = m * LOG2E_F;
        float acc = 0.f;
        for (int k = 0; k < L; ++k) acc += fast_exp2(row[k] * LOG2E_F - m2);
        sp[rw.cell0 + c] = (m2 + fast_log2(acc)) * (float)LN2_D;
    }
}

// The expansion: the chunk's cells' marginals and log-sum-exps (log2 units)
// are staged in LDS, a cell per lane, and each float of the chunk takes its
// cell's pair from there.
__global__ __launch_bounds__(kLabelChunk) void label_expand_kernel(KernelPlan p, const float *__restrict__ s4,
                                                                   const float *__restrict__ sp,
                                                                   const float *__restrict__ mu,
                                                                   float *__restrict__ marg) {
    extern __shared__ float lab_cells[];   // kLabelWaves x 2 x (kLabelRowChunk / 2 + 2) floats
    constexpr int kCells = kLabelRowChunk / 2 + 2;   // cells a chunk can touch (L >= 2)
    const int wave = (int)threadIdx.x >> 6, lane = (int)threadIdx.x & 63, L = p.L;
    float *cm = lab_cells + wave * 2 * kCells, *co = cm + kCells;
    Label_row rw{};
    const bool have = label_row(p, (int)blockIdx.x * kLabelWaves + wave, &rw);
    const int end = have ? min(rw.f0 + kLabelRowChunk, rw.len) : 0;   // the chunk's floats [f0, end)
    const int c0 = have ? rw.f0 / L : 0, nc = have ? (end - 1) / L + 1 - c0 : 0;
    const float *src = s4 + rw.cell0 * L;
    float x[kLabelPer];
    if (have) {
#pragma unroll
        for (int k = 0; k < kLabelPer; ++k) x[k] = src[min(rw.f0 + 64 * k + lane, end - 1)];
        for (int c = lane; c < nc; c += 64) {
            cm[c] = mu[rw.cell0 + c0 + c];
            co[c] = sp[rw.cell0 + c0 + c] * LOG2E_F;
        }
    }
    __syncthreads();
    if (!have) return;
    float *dst = marg + rw.cell0 * L;
    const float invL = 1.0f / (float)L;
#pragma unroll
    for (int k = 0; k < kLabelPer; ++k) {
        const int f = rw.f0 + 64 * k + lane;
        if (f < end) {
            const int c = div_small(f, L, invL) - c0;   // cell (i, i+1+c0+c)
            dst[f] = cm[c] * fast_exp2(x[k] * LOG2E_F - co[c]);
        }
    }
}

// The gold-tree loss: the inside kernel with marginals, minus the gold
// indicator (inside_block, GOLD).
template <bool SPILL, bool TEAM = false>
__global__ __launch_bounds__(kThreadsMax) void loss_kernel(KernelPlan p, const float *__restrict__ scores,
                                                           const int32_t *__restrict__ gold,
                                                           const float *__restrict__ grad,
                                                           float *__restrict__ loss,
                                                           float *__restrict__ marg) {
    extern __shared__ __align__(16) char smem_raw[];
    if constexpr (SPILL && !TEAM) {
        inside_block<true, true, true>(p, blockIdx.x, nullptr, smem_raw, scores, grad, nullptr, marg, gold, loss);
    } else if constexpr (SPILL) {
        Team tm;
        int job, stride;
        if (!spill_jobs(p, tm, job, stride)) return;
        for (; job < p.inside.n_spill; job += stride, ++tm.job) {
            inside_block<true, true, true>(p, job, nullptr, smem_raw, scores, grad, nullptr, marg, gold, loss, tm);
            __syncthreads();
        }
    } else
        inside_block<true, false, true>(p, blockIdx.x, p.inside.recs + (size_t)blockIdx.x * p.rec_stride, smem_raw,
                                        scores, grad, nullptr, marg, gold, loss);
}

template <bool SPILL, bool LAB, bool TEAM = false>
__global__ __launch_bounds__(kThreadsMax) void cky_kernel(KernelPlan p, const float *__restrict__ scores,
                                                          int32_t *__restrict__ spans,
                                                          float *__restrict__ best,
                                                          int32_t *__restrict__ labels) {
    extern __shared__ __align__(16) char smem_raw[];
    if constexpr (SPILL && !TEAM) {
        cky_block<true, LAB>(p, blockIdx.x, nullptr, smem_raw, scores, spans, best, labels);
    } else if constexpr (SPILL) {
        Team tm;
        int job, stride;
        if (!spill_jobs(p, tm, job, stride)) return;
        for (; job < p.cky.n_spill; job += stride, ++tm.job) {
            cky_block<true, LAB>(p, job, nullptr, smem_raw, scores, spans, best, labels, false, tm);
            __syncthreads();
        }
    } else
        cky_block<false, LAB>(p, blockIdx.x, p.cky.recs + (size_t)blockIdx.x * p.rec_stride, smem_raw, scores, spans,
                              best, labels);
}

// Claim the next bundle of a persistent launch over n_rec records (see
// parse_kernel): returns its index, n_rec or more when none is left.
__device__ __forceinline__ int claim_next(int32_t *counter, int n_rec, int *slot) {
    if (threadIdx.x == 0) {
        const int ticket = atomicAdd(counter, 1);
        if (ticket == n_rec - 1) atomicExch(counter, 0);
        *slot = (int)gridDim.x + ticket;
    }
    __syncthreads();   // the claim is published and the bundle's LDS is free
    const int cur = *slot;
    __syncthreads();   // every thread has read the slot
    return cur;
}

// The workspace-chart sentences of the fused pass in one launch: job
// b < inside.n_spill runs the inside sweep with the marginals of the b-th
// such sentence, the others run CKY, so that a long sentence's two passes
// run side by side on different CUs (their workspace charts are disjoint:
// the CKY schedule's follow the inside schedule's).
template <bool TEAM>
__global__ __launch_bounds__(kThreadsMax) void spill_parse_kernel(KernelPlan p, const float *__restrict__ scores,
                                                                  const float *__restrict__ grad,
                                                                  float *__restrict__ logZ, float *__restrict__ marg,
                                                                  int32_t *__restrict__ spans,
                                                                  float *__restrict__ best) {
    extern __shared__ __align__(16) char smem_raw[];
    if constexpr (!TEAM) {   // a workgroup per job
        const int b = (int)blockIdx.x;
        if (b < p.inside.n_spill) inside_block<true, true>(p, b, nullptr, smem_raw, scores, grad, logZ, marg);
        else cky_block<true>(p, b - p.inside.n_spill, nullptr, smem_raw, scores, spans, best);
        return;
    }
    Team tm;
    int job, stride;
    if (!spill_jobs(p, tm, job, stride)) return;
    for (; job < p.inside.n_spill + p.cky.n_spill; job += stride, ++tm.job) {
        if (job < p.inside.n_spill)
            inside_block<true, true>(p, job, nullptr, smem_raw, scores, grad, logZ, marg, nullptr, nullptr, tm);
        else
            cky_block<true>(p, job - p.inside.n_spill, nullptr, smem_raw, scores, spans, best, nullptr, false, tm);
        __syncthreads();
    }
}

// MBR decoding (Sec. 3.3) in one launch: each bundle runs the inside sweep
// with the outside and writes the marginals, then CKY with the marginals in
// place of the scores, in the same workgroup.  The CKY prologue reads back
// exactly the cells this thread wrote (the same cell walk over the same
// bundle), so the marginals come from this CU's cache, and the LDS charts are
// reused.  Persistent, bundles claimed as in parse_kernel.
__global__ __launch_bounds__(kThreadsMax) void mbr_kernel(KernelPlan p, const float *__restrict__ scores,
                                                          float *__restrict__ logZ, float *marg,
                                                          int32_t *__restrict__ spans,
                                                          float *__restrict__ best) {
    extern __shared__ __align__(16) char smem_raw[];
    __shared__ int slot;
    int cur = blockIdx.x;
    for (;;) {
        const int32_t *rec = p.mbr + (size_t)cur * p.rec_stride;
        inside_block<true, false>(p, 0, rec, smem_raw, scores, nullptr, logZ, marg);
        __syncthreads();   // the marginals are written and the inside charts are free
        cky_block<false>(p, 0, rec, smem_raw, marg, spans, best, nullptr, true);
        if ((int)gridDim.x >= p.n_mbr) break;
        cur = claim_next(p.counter, p.n_mbr, &slot);
        if (cur >= p.n_mbr) break;
    }
}

// Labelling stage (Sec. 2.1, Eq. label-argmax): row r of sentence b's span
// list gets the lowest label attaining max_l s(i,j,l) when it is a span of
// sentence b, else -1.  A group of kLabelLanes lanes per row: lane q reads
// labels q, q + kLabelLanes, ... of the row's contiguous label scores (keeping
// its first maximum), then the group takes the max and the lowest label at it.
constexpr int kLabelLanes = 16;
__global__ __launch_bounds__(256) void label_spans_kernel(const int32_t *__restrict__ len,
                                                          const float *__restrict__ s4, int n1, int L, int B,
                                                          const int32_t *__restrict__ spans,
                                                          int32_t *__restrict__ labels) {
    const int R = 2 * (n1 - 1) - 1;
    const int64_t rows = (int64_t)B * R;
    const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kLabelLanes;
    const int q = threadIdx.x & (kLabelLanes - 1);
    const bool ok = row < rows;          // the same for every lane of a group
    const int64_t rr = ok ? row : rows - 1;
    const int b = (int)(rr / R);
    const int i = spans[2 * rr], j = spans[2 * rr + 1], n = len[b];
    const bool valid = ok && 0 <= i && i < j && j <= n;
    float m = -INFINITY;
    int bl = 0x7fffffff;
    if (valid) {
        const float *v = s4 + (((size_t)b * n1 + i) * n1 + j) * L;
        for (int l = q; l < L; l += kLabelLanes) {
            const float x = v[l];
            if (x > m) {
                m = x;
                bl = l;
            }
        }
    }
    const float mg = grp_max<kLabelLanes>(m);
    const int k = grp_min_i<kLabelLanes>(m == mg ? bl : 0x7fffffff);
    if (ok && q == 0) labels[rr] = valid ? k : -1;
}

// The whole pass -- inside, marginals and CKY -- in one launch of at most
// one workgroup per workgroup slot, each running a chain of bundles from the
// plan's merged list (inside and CKY bundles by decreasing predicted
// duration): workgroup b starts with bundle b and, as each bundle ends,
// claims the next from a counter (ticket t is bundle grid + t), so that
// workgroups take the next bundles in the order they free up, whatever their
// XCD.  (Claiming any earlier -- at the end of the sweep, to fetch ahead --
// measured slower: the order then strays from the order of freeing.)  Every
// processed bundle claims once, so the n_mix claims end on ticket n_mix - 1,
// whose holder zeroes the counter for the next launch; with as many
// workgroups as bundles nobody claims.
__global__ __launch_bounds__(kThreadsMax) void parse_kernel(KernelPlan p, const float *__restrict__ scores,
                                                            const float *__restrict__ grad,
                                                            float *__restrict__ logZ,
                                                            float *__restrict__ marg,
                                                            int32_t *__restrict__ spans,
                                                            float *__restrict__ best) {
    extern __shared__ __align__(16) char smem_raw[];
    __shared__ int slot;
    int cur = blockIdx.x;
    for (;;) {
        const int32_t *rec = p.mix + (size_t)cur * p.rec_stride;
        if (rec[kRecKind] == kKindInside)
            inside_block<true, false>(p, 0, rec, smem_raw, scores, grad, logZ, marg);
        else
            cky_block<false>(p, 0, rec, smem_raw, scores, spans, best);
        if ((int)gridDim.x >= p.n_mix) break;   // one bundle per workgroup: no claims at all
        cur = claim_next(p.counter, p.n_mix, &slot);
        if (cur >= p.n_mix) break;
    }
}

// Zeroes n words (the no-allocation entry point's claim counter): a kernel,
// not hipMemsetAsync, so that the call stays a plain kernel node when a
// caller captures it into a graph.
__global__ void zero_words(int32_t *p, int n) {
    for (int t = threadIdx.x; t < n; t += blockDim.x) p[t] = 0;
}

// Scratch of the no-allocation entry point, one per GPU for the life of the
// process.  In host code `scratch` names a host-side stand-in, not device
// memory: host code only ever uses the address scratch_address() resolved.
__device__ __align__(256) char scratch[kScratchBytes];

}  // namespace

// ---------------------------------------------------------------------------
// Launchers.

hipError_t scratch_address(int device, char **out) {
    static std::mutex mu;
    static char *addr[kMaxDevices] = {};
    *out = nullptr;
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (addr[device] == nullptr) {
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[device] = static_cast<char *>(ptr);
    }
    *out = addr[device];
    return hipSuccess;
}

hipError_t launch_parse_scratch(const KernelPlan &p, char *scr, const float *scores, const float *grad,
                                float *logZ, float *marg, int32_t *spans, float *best, hipStream_t stream) {
    KernelPlan q = p;
    q.counter = reinterpret_cast<int32_t *>(scr);
    q.ws = scr + kScratchCounterBytes;
    q.team_area = nullptr;   // workspace sentences on lone workgroups: no memory beyond the scratch
    hipLaunchKernelGGL(zero_words, dim3(1), dim3(64), 0, stream, q.counter, (int)(kScratchCounterBytes / 4));
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_parse(q, scores, grad, logZ, marg, spans, best, stream);
}

int spill_blocks_per_cu() {
    const void *fns[] = {
        (const void *)inside_kernel<false, true, false, true>, (const void *)inside_kernel<true, true, false, true>,
        (const void *)cky_kernel<true, false, true>,           (const void *)cky_kernel<true, true, true>,
        (const void *)loss_kernel<true, true>,                 (const void *)spill_parse_kernel<true>,
    };
    int least = 1 << 30;
    for (const void *f : fns) {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, f, kThreadsMax, 0) != hipSuccess) {
            (void)hipGetLastError();
            return 0;
        }
        least = nb < least ? nb : least;
    }
    return least;
}

hipError_t set_kernel_attributes(int max_lds_bytes) {
    const void *fns[] = {
        (const void *)inside_kernel<false, false>,        (const void *)inside_kernel<true, false>,
        (const void *)inside_kernel<false, false, true>,  (const void *)inside_kernel<true, false, true>,
        (const void *)cky_kernel<false, false>,           (const void *)cky_kernel<false, true>,
        (const void *)loss_kernel<false>,                 (const void *)parse_kernel,
        (const void *)mbr_kernel,
    };
    for (const void *f : fns) {
        hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, max_lds_bytes);
        if (e != hipSuccess) return e;
    }
    // the label reduction's staging at the most labels a plan accepts
    return hipFuncSetAttribute((const void *)label_reduce_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)(kLabelWaves * (kLabelRowChunk + CRF_MAX_LABELS) * sizeof(float)));
}

template <bool SPILL, bool LAB = false, bool TEAM = false>
static void launch_inside_k(const KernelPlan &p, dim3 grid, int threads, size_t lds, hipStream_t s,
                            const float *scores, const float *grad, float *logZ, float *marg) {
    const dim3 block(threads);
    if (marg != nullptr)
        hipLaunchKernelGGL((inside_kernel<true, SPILL, LAB, TEAM>), grid, block, lds, s, p, scores, grad, logZ, marg);
    else
        hipLaunchKernelGGL((inside_kernel<false, SPILL, LAB, TEAM>), grid, block, lds, s, p, scores, grad, logZ, marg);
}

// Sets the team size of a workspace launch (team_shape) and its grid; a
// team launch gets its team area cleared by a kernel first.
static hipError_t spill_launch_shape(KernelPlan &q, int jobs, hipStream_t stream, dim3 *grid) {
    const TeamShape ts = team_shape(jobs, q.team_cap, q.team_area != nullptr);
    q.team_k = ts.k;
    *grid = dim3(ts.grid);
    if (ts.k < 2) return hipSuccess;
    hipLaunchKernelGGL(zero_words, dim3(1), dim3(256), 0, stream, q.team_area,
                       kTeamHeaderWords + kTeamLineWords * (ts.grid / ts.k));
    return hipGetLastError();
}

// The bundles' launch and the workspace sentences' launch of one inside pass.
template <bool LAB>
static hipError_t launch_inside_sweeps(const KernelPlan &p, const float *scores, const float *grad, float *logZ,
                                       float *marg, hipStream_t stream) {
    const Schedule &q = p.inside;
    hipError_t e;
    if (q.n_bundles > 0) {
        launch_inside_k<false, LAB>(p, dim3(q.n_bundles), q.threads, q.lds_bytes, stream, scores, grad, logZ, marg);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (q.n_spill > 0) {
        KernelPlan t = p;
        dim3 grid;
        if ((e = spill_launch_shape(t, q.n_spill, stream, &grid)) != hipSuccess) return e;
        if (t.team_k > 1) launch_inside_k<true, false, true>(t, grid, kThreadsMax, 0, stream, scores, grad, logZ, marg);
        else launch_inside_k<true>(t, grid, kThreadsMax, 0, stream, scores, grad, logZ, marg);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_inside(const KernelPlan &p, const float *scores, const float *grad, float *logZ,
                         float *marg, hipStream_t stream) {
    hipError_t e;
    if (p.L > 1) {
        // labelled: the label log-sum-exps of the sentences whose label
        // passes run chip-wide into the workspace, the sweeps (on those, and
        // on their own label scores for the bundles marked kRecLab; the
        // former's marginals into the workspace too), then those sentences'
        // per-label marginals
        float *sp = reinterpret_cast<float *>(p.ws + p.lab_sp_off);
        float *mu = reinterpret_cast<float *>(p.ws + p.lab_mu_off);
        const dim3 lab_grid((p.n_lab_rows + kLabelWaves - 1) / kLabelWaves);
        if (p.n_lab_rows > 0) {
            hipLaunchKernelGGL(label_reduce_kernel, lab_grid, dim3(kLabelChunk),
                               (size_t)kLabelWaves * (kLabelRowChunk + p.L) * sizeof(float), stream, p, scores, sp);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        KernelPlan u = p;
        u.L = 1;
        u.lab_s4 = scores;
        u.lab_out = marg;
        u.lab_L = p.L;
        if ((e = launch_inside_sweeps<true>(u, sp, grad, logZ, marg != nullptr ? mu : nullptr, stream)) != hipSuccess)
            return e;
        if (marg == nullptr || p.n_lab_rows < 1) return hipSuccess;
        hipLaunchKernelGGL(label_expand_kernel, lab_grid, dim3(kLabelChunk),
                           (size_t)kLabelWaves * 2 * (kLabelRowChunk / 2 + 2) * sizeof(float), stream, p, scores, sp,
                           mu, marg);
        return hipGetLastError();
    }
    return launch_inside_sweeps<false>(p, scores, grad, logZ, marg, stream);
}

template <bool LAB>
static hipError_t launch_cky_k(const KernelPlan &p, const float *scores, int32_t *spans, float *best,
                               hipStream_t stream, int32_t *labels) {
    const Schedule &q = p.cky;
    hipError_t e;
    if (q.n_bundles > 0) {
        hipLaunchKernelGGL((cky_kernel<false, LAB>), dim3(q.n_bundles), dim3(q.threads), (size_t)q.lds_bytes, stream, p,
                           scores, spans, best, labels);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (q.n_spill > 0) {
        KernelPlan t = p;
        dim3 grid;
        if ((e = spill_launch_shape(t, q.n_spill, stream, &grid)) != hipSuccess) return e;
        if (t.team_k > 1)
            hipLaunchKernelGGL((cky_kernel<true, LAB, true>), grid, dim3(kThreadsMax), 0, stream, t, scores, spans, best,
                               labels);
        else
            hipLaunchKernelGGL((cky_kernel<true, LAB>), grid, dim3(kThreadsMax), 0, stream, t, scores, spans, best, labels);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_cky(const KernelPlan &p, const float *scores, int32_t *spans, float *best,
                      hipStream_t stream, int32_t *labels) {
    return labels != nullptr ? launch_cky_k<true>(p, scores, spans, best, stream, labels)
                             : launch_cky_k<false>(p, scores, spans, best, stream, nullptr);
}

hipError_t launch_mbr(const KernelPlan &p, const float *scores, float *logZ, float *marg, int32_t *spans,
                      float *best, hipStream_t stream) {
    if (p.mbr == nullptr || p.counter == nullptr || p.mbr_grid < 1) {
        // separate launches, in stream order: inside + marginals, then CKY
        // over the marginals
        hipError_t e = launch_inside(p, scores, nullptr, logZ, marg, stream);
        if (e != hipSuccess) return e;
        return launch_cky(p, marg, spans, best, stream);
    }
    hipLaunchKernelGGL(mbr_kernel, dim3(p.mbr_grid), dim3(p.inside.threads), (size_t)p.mbr_lds, stream, p, scores,
                       logZ, marg, spans, best);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // sentences too long for LDS (the plan has checked that the inside and
    // CKY workspace lists hold the same sentences): their marginals, then
    // CKY over them
    if (p.inside.n_spill > 0) {
        KernelPlan t = p;
        dim3 grid;
        if ((e = spill_launch_shape(t, p.inside.n_spill, stream, &grid)) != hipSuccess) return e;
        if (t.team_k > 1) launch_inside_k<true, false, true>(t, grid, kThreadsMax, 0, stream, scores, nullptr, logZ, marg);
        else launch_inside_k<true>(t, grid, kThreadsMax, 0, stream, scores, nullptr, logZ, marg);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = spill_launch_shape(t, p.cky.n_spill, stream, &grid)) != hipSuccess) return e;
        if (t.team_k > 1)
            hipLaunchKernelGGL((cky_kernel<true, false, true>), grid, dim3(kThreadsMax), 0, stream, t, marg, spans, best,
                               nullptr);
        else
            hipLaunchKernelGGL((cky_kernel<true, false>), grid, dim3(kThreadsMax), 0, stream, t, marg, spans, best, nullptr);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_loss(const KernelPlan &p, const float *scores, const int32_t *gold, const float *grad,
                       float *loss, float *grad_scores, hipStream_t stream) {
    const Schedule &q = p.inside;
    hipError_t e;
    if (q.n_bundles > 0) {
        hipLaunchKernelGGL((loss_kernel<false>), dim3(q.n_bundles), dim3(q.threads), (size_t)q.lds_bytes, stream, p,
                           scores, gold, grad, loss, grad_scores);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (q.n_spill > 0) {
        KernelPlan t = p;
        dim3 grid;
        if ((e = spill_launch_shape(t, q.n_spill, stream, &grid)) != hipSuccess) return e;
        if (t.team_k > 1)
            hipLaunchKernelGGL((loss_kernel<true, true>), grid, dim3(kThreadsMax), 0, stream, t, scores, gold, grad, loss,
                               grad_scores);
        else
            hipLaunchKernelGGL((loss_kernel<true>), grid, dim3(kThreadsMax), 0, stream, t, scores, gold, grad, loss,
                               grad_scores);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_label_spans(const KernelPlan &p, const float *label_scores, int L, const int32_t *spans,
                              int32_t *labels, hipStream_t stream) {
    const int64_t rows = (int64_t)p.B * (2 * (p.n1 - 1) - 1);
    const int64_t blocks = (rows * kLabelLanes + 255) / 256;
    hipLaunchKernelGGL(label_spans_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, p.len, label_scores, p.n1, L,
                       p.B, spans, labels);
    return hipGetLastError();
}

hipError_t launch_parse(const KernelPlan &p, const float *scores, const float *grad, float *logZ,
                        float *marg, int32_t *spans, float *best, hipStream_t stream) {
    const Schedule &qi = p.inside, &qc = p.cky;
    hipError_t e;
    if (p.mix != nullptr && p.counter != nullptr && p.fused_grid >= 1 && p.n_mix == qi.n_bundles + qc.n_bundles) {
        const size_t lds = (size_t)(qi.lds_bytes > qc.lds_bytes ? qi.lds_bytes : qc.lds_bytes);
        hipLaunchKernelGGL(parse_kernel, dim3(p.fused_grid), dim3(qi.threads), lds, stream, p,
                           scores, grad, logZ, marg, spans, best);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    } else {
        // the LDS bundles of each pass as its own launch
        if (qi.n_bundles > 0) {
            launch_inside_k<false>(p, dim3(qi.n_bundles), qi.threads, qi.lds_bytes, stream, scores, grad, logZ, marg);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        if (qc.n_bundles > 0) {
            hipLaunchKernelGGL((cky_kernel<false, false>), dim3(qc.n_bundles), dim3(qc.threads), (size_t)qc.lds_bytes,
                               stream, p, scores, spans, best, nullptr);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
    }
    if (qi.n_spill + qc.n_spill > 0) {
        KernelPlan t = p;
        dim3 grid;
        if ((e = spill_launch_shape(t, qi.n_spill + qc.n_spill, stream, &grid)) != hipSuccess) return e;
        if (t.team_k > 1)
            hipLaunchKernelGGL(spill_parse_kernel<true>, grid, dim3(kThreadsMax), 0, stream, t, scores, grad, logZ, marg,
                               spans, best);
        else
            hipLaunchKernelGGL(spill_parse_kernel<false>, grid, dim3(kThreadsMax), 0, stream, t, scores, grad, logZ, marg,
                               spans, best);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace crf
