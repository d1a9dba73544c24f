// crf_plan.cpp -- host side of the C ABI: argument checks, the per-batch
// schedule and the plan's device memory.
//
// Scheduling.  Sentences are independent (Algorithm 1 parallelises over the
// batch), and a sentence's cost grows as its number of split points,
// T(n) = (n+1) n (n-1) / 6, plus a latency term per width step.  Workgroups
// are dispatched in blockIdx order, so bundles are launched longest first:
// the longest dependency chains start first and short bundles fill the tail
// (longest-processing-time-first); the fused launch's order and the split of
// its last bundles come from a replay of the dispatch (plan_fused_launch).
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <numeric>
#include <vector>

#include "../../include/crf_inside.h"
#include "crf_internal.h"

namespace {

thread_local char g_last_error[256] = "";

int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return code;
}

int ok() {
    g_last_error[0] = '\0';
    return CRF_OK;
}

int hip_fail(hipError_t e, const char *where) {
    return fail(CRF_EHIP, "%s: %s", where, hipGetErrorString(e));
}

}  // namespace

struct crf_plan {
    int device = -1;
    int32_t B = 0, n1 = 0, L = 1, max_len = 0;
    uint32_t flags = 0;
    std::vector<void *> allocations;
    crf::KernelPlan kp{};
    int64_t ws_bytes = 0;
    int32_t split_ws_count = 0;    // sentences with CKY split tables in the workspace
    int32_t workspace_users = 0;   // sentences using the workspace in some call
};

namespace {

void release(crf_plan *p) {
    for (void *a : p->allocations) (void)hipFree(a);
    p->allocations.clear();
}

template <typename T>
hipError_t upload(crf_plan *p, const std::vector<T> &v, const T **dst) {
    *dst = nullptr;
    if (v.empty()) return hipSuccess;
    void *d = nullptr;
    hipError_t e = hipMalloc(&d, v.size() * sizeof(T));
    if (e != hipSuccess) return e;
    p->allocations.push_back(d);
    e = hipMemcpy(d, v.data(), v.size() * sizeof(T), hipMemcpyHostToDevice);
    *dst = static_cast<const T *>(d);
    return e;
}

// One kind of chart's schedule on the host: equal-length bundles for the LDS
// kernel, single sentences for the workspace kernel.
struct HostSchedule {
    std::vector<crf::Bundle> bundles;
    std::vector<int32_t> order;      // sentence ids grouped by bundle
    std::vector<int32_t> spill;      // sentence ids on the workspace kernel
    std::vector<int64_t> off;        // their chart offsets in the workspace
    int32_t lds_bytes = 0;
    int32_t threads = crf::kThreadsDefault;
    int64_t ws_bytes = 0;
};

// Cost model of one sentence for sizing bundles: split points plus a latency
// term per width step.  (Labelled scores are reduced over their labels
// before the bundles run, so the bundles' work is the same.)
inline double sentence_cost(int n) {
    const double T = (double)(n + 1) * n * (n - 1) / 6.0;
    return T + 200.0 * (n - 1);
}

// Predicted duration (microseconds on MI355X, two workgroups per CU) of a
// bundle of `count` sentences of n words, fitted to per-workgroup timings of
// the fused launch: a latency per width step, a per-cell term for the global
// loads and stores around the sweep (inside) or the tree walk (CKY), and the
// split points themselves.
inline double split_points(int n) { return (double)(n + 1) * n * (n - 1) / 6.0; }
inline double predict_inside(int n, int count) {
    return 0.86 * (n - 1) + 0.0037 * count * (double)n * n + 1.0e-4 * count * split_points(n) + 3.6;
}
inline double predict_cky(int n, int count) {
    return 0.94 * (n - 1) + 0.045 * count * (double)n + 7.0e-5 * count * split_points(n) + 4.7;
}

// Predicted end of a launch whose workgroups (durations `dur`, in launch
// order) are dealt round-robin to n_part partitions (XCDs) of `slots`
// workgroup slots each, a workgroup starting when a slot of its partition
// frees up.  ends[b] receives each workgroup's predicted end.
double simulate_launch(const std::vector<double> &dur, int n_part, int slots, std::vector<double> &ends,
                       std::vector<double> &heap) {
    heap.assign((size_t)n_part * slots, 0.0);
    ends.resize(dur.size());
    double end = 0.0;
    auto later = [](double a, double b) { return a > b; };   // min-heap
    for (size_t b = 0; b < dur.size(); ++b) {
        double *h = heap.data() + (b % n_part) * (size_t)slots;
        std::pop_heap(h, h + slots, later);
        const double e = h[slots - 1] + dur[b];
        h[slots - 1] = e;
        std::push_heap(h, h + slots, later);
        ends[b] = e;
        end = std::max(end, e);
    }
    return end;
}

// Launch order of the fused kernel (mix: e >= 0 inside bundle e, e < 0 CKY
// bundle ~e), longest predicted first.  Then the tail: while it helps the
// predicted makespan, the multi-sentence bundle that ends last is split in
// two (the halves keep their sentences' slots of the order array), which
// trades a little more total work for a shorter end of the launch.  Both
// bundle lists come back in launch order.  fits(inside, n, count) says
// whether a bundle of that shape fits the launch's LDS; a split takes the
// count nearest to half whose two parts both fit, and a bundle with no such
// count stays whole.
template <typename FIT>
void plan_fused_launch(std::vector<crf::Bundle> &in, std::vector<crf::Bundle> &ck, int n_part, int slots,
                       std::vector<int32_t> &mix, FIT &&fits) {
    struct Item {
        double d;
        bool inside;
        bool whole;   // no split of it fits
        crf::Bundle bd;
    };
    auto predict = [](const Item &x) {
        return x.inside ? predict_inside(x.bd.n, x.bd.count) : predict_cky(x.bd.n, x.bd.count);
    };
    std::vector<Item> items;
    items.reserve(2 * (in.size() + ck.size()));
    for (const crf::Bundle &b : in) items.push_back({0.0, true, false, b});
    for (const crf::Bundle &b : ck) items.push_back({0.0, false, false, b});
    for (Item &x : items) x.d = predict(x);
    auto longer = [](const Item &a, const Item &b) { return a.d > b.d; };
    std::stable_sort(items.begin(), items.end(), longer);

    std::vector<double> dur, ends, heap;
    auto simulate = [&]() {
        dur.resize(items.size());
        for (size_t i = 0; i < items.size(); ++i) dur[i] = items[i].d;
        return simulate_launch(dur, n_part, slots, ends, heap);
    };
    double best = simulate();
    std::vector<Item> best_items = items;
    const int max_iter = (int)items.size() / 2;
    for (int it = 0, stale = 0; it < max_iter && stale < 64; ++it) {
        int j = -1;
        for (int i = 0; i < (int)items.size(); ++i)
            if (items[i].bd.count >= 2 && !items[i].whole && (j < 0 || ends[i] > ends[j])) j = i;
        if (j < 0) break;
        const int c = items[j].bd.count, n = items[j].bd.n;
        const bool kind = items[j].inside;
        int half = 0;
        for (int d = 0; d <= 3 && half == 0; ++d)
            for (int h : {c / 2 - d, c / 2 + d})
                if (half == 0 && h >= 1 && h < c && fits(kind, n, h) && fits(kind, n, c - h)) half = h;
        if (half == 0) {
            items[j].whole = true;
            continue;
        }
        Item a = items[j], b = items[j];
        a.bd.count = half;
        b.bd.first += a.bd.count;
        b.bd.count -= a.bd.count;
        a.d = predict(a);
        b.d = predict(b);
        items.erase(items.begin() + j);
        for (const Item &x : {a, b}) items.insert(std::upper_bound(items.begin(), items.end(), x, longer), x);
        const double m = simulate();
        if (m < best - 1e-6) {
            best = m;
            best_items = items;
            stale = 0;
        } else {
            ++stale;
        }
    }
    in.clear();
    ck.clear();
    mix.clear();
    for (const Item &x : best_items) {
        if (x.inside) {
            mix.push_back((int32_t)in.size());
            in.push_back(x.bd);
        } else {
            mix.push_back(~(int32_t)ck.size());
            ck.push_back(x.bd);
        }
    }
}

// Bundle sizing.  A bundle's split points are aimed at target_scale times the
// batch's share per workgroup slot.  Inside bundles aim at twice the share:
// their width steps are latency bound, so more sentences per step cost
// little, and fewer, fuller bundles measured 3-5% faster on the 5,000-sentence
// mixed batch than an even share; CKY bundles take the share.
constexpr double kInsideTargetScale = 2.0, kCkyTargetScale = 1.0;

// `order` is sorted by decreasing length.  `bundle_bytes(n, count)` is the
// LDS of a bundle of `count` sentences of n words, `spill_chart(n)` a
// sentence's workspace chart.  A bundle's LDS need not grow with its count
// (the inside chart stride depends on the count's factors of two), so a
// length's bundles hold at most the largest count below which every count
// fits.
template <typename BB, typename FS>
HostSchedule make_schedule(const std::vector<int32_t> &order, const int32_t *len, int lds_cap,
                           bool force_spill, int64_t ws_base, BB &&bundle_bytes, FS &&spill_chart,
                           double target_scale) {
    HostSchedule s;
    s.threads = crf::kThreadsDefault;
    // Workgroup LDS budget: half the CU when every eligible sentence fits in
    // half (two workgroups per CU), else all of it (one).
    const int64_t half = lds_cap / 2 - crf::kReservedLds, full = lds_cap - crf::kReservedLds;
    int64_t biggest = 0;
    std::vector<int32_t> eligible;
    int64_t cursor = ws_base;
    for (int32_t b : order) {
        const int n = len[b];
        const int64_t need = bundle_bytes(n, 1);
        if (!force_spill && need <= full && n <= crf::kMaxLenInLds) {
            eligible.push_back(b);
            biggest = std::max(biggest, need);
        } else {
            s.spill.push_back(b);
            s.off.push_back(cursor);
            // The kernels' masked tail loads may read up to 511 elements
            // past a chart; an 8 KiB guard band keeps them inside the workspace.
            cursor += (spill_chart(n) + 8192 + 255) / 256 * 256;
        }
    }
    s.ws_bytes = cursor - ws_base;
    const bool small = biggest <= half;
    const int64_t budget = small ? half : full;
    const int slots = 256 * (small ? 2 : 1);

    // Target cost per bundle: spread the total over the workgroup slots, but
    // never split below one sentence.
    double total = 0.0;
    for (int32_t b : eligible) total += sentence_cost(len[b]);
    const double target = std::max(total / slots, 1.0) * target_scale;

    struct Tmp { crf::Bundle bd; double cost; };
    std::vector<Tmp> tmp;
    size_t a = 0;
    while (a < eligible.size()) {
        const int n = len[eligible[a]];
        size_t e = a;
        while (e < eligible.size() && len[eligible[e]] == n) ++e;
        const int count = (int)(e - a);
        int by_lds = 1;
        while (by_lds < crf::kMaxBundle && bundle_bytes(n, by_lds + 1) <= budget) ++by_lds;
        const int by_cost = std::max(1, (int)(target / sentence_cost(n)));
        const int per = std::min(by_lds, std::max(1, by_cost));
        const int nbund = (count + per - 1) / per;
        for (int q = 0; q < nbund; ++q) {
            const int lo = (int)((int64_t)count * q / nbund), hi = (int)((int64_t)count * (q + 1) / nbund);
            Tmp t;
            t.bd.first = (int32_t)(a + lo);
            t.bd.count = hi - lo;
            t.bd.n = n;
            t.bd.split_ws = -1;
            t.cost = (hi - lo) * (sentence_cost(n) - 200.0 * (n - 1)) + 200.0 * (n - 1);
            tmp.push_back(t);
            s.lds_bytes = std::max<int32_t>(s.lds_bytes, (int32_t)bundle_bytes(n, hi - lo));
        }
        a = e;
    }
// Most expensive bundles first: workgroups are dispatched in order.
    std::stable_sort(tmp.begin(), tmp.end(), [](const Tmp &x, const Tmp &y) { return x.cost > y.cost; });
    for (const Tmp &t : tmp) {
        crf::Bundle bd = t.bd;
        const int first = (int)s.order.size();
        for (int q = 0; q < bd.count; ++q) s.order.push_back(eligible[bd.first + q]);
        bd.first = first;
        s.bundles.push_back(bd);
    }
    return s;
}

}  // namespace

extern "C" {

const char *crf_status_string(int status) {
    switch (status) {
        case CRF_OK: return "success";
        case CRF_EINVAL: return "invalid argument";
        case CRF_ENOMEM: return "out of memory";
        case CRF_EHIP: return "HIP runtime error";
        case CRF_EUNSUPPORTED: return "unsupported";
        default: return "unknown status";
    }
}

const char *crf_last_error(void) { return g_last_error; }

int crf_plan_create(crf_plan **out, const int32_t *lengths_host, int32_t batch, int32_t n1,
                    int32_t num_labels, uint32_t flags) {
    if (out == nullptr) return fail(CRF_EINVAL, "out is NULL");
    *out = nullptr;
    if (lengths_host == nullptr) return fail(CRF_EINVAL, "lengths_host is NULL");
    if (batch < 1) return fail(CRF_EINVAL, "batch %d < 1", batch);
    if (n1 < 2 || n1 > CRF_MAX_LEN + 1)
        return fail(CRF_EINVAL, "n1 %d outside [2, %d]", n1, CRF_MAX_LEN + 1);
    if (num_labels < 1 || num_labels > CRF_MAX_LABELS)
        return fail(CRF_EINVAL, "num_labels %d outside [1, %d]", num_labels, CRF_MAX_LABELS);
    if (flags & ~(CRF_FORCE_SPILL | CRF_NO_TEAMS)) return fail(CRF_EINVAL, "unknown flags 0x%x", flags);
    int32_t max_len = 0;
    for (int32_t b = 0; b < batch; ++b) {
        const int32_t n = lengths_host[b];
        if (n < 1 || n > n1 - 1)
            return fail(CRF_EINVAL, "lengths[%d] = %d outside [1, n1-1 = %d]", b, n, n1 - 1);
        max_len = std::max(max_len, n);
    }

    // Arguments are valid: from here on HIP calls are made.
    crf_plan *p = new (std::nothrow) crf_plan();
    if (p == nullptr) return fail(CRF_ENOMEM, "host allocation of the plan failed");
    p->B = batch;
    p->n1 = n1;
    p->L = num_labels;
    p->max_len = max_len;
    p->flags = flags;

    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) { delete p; return hip_fail(e, "hipGetDevice"); }
    int lds_cap = 0;
    e = hipDeviceGetAttribute(&lds_cap, hipDeviceAttributeMaxSharedMemoryPerBlock, p->device);
    if (e != hipSuccess) { delete p; return hip_fail(e, "hipDeviceGetAttribute"); }

    // Longest first; ties keep batch order.
    std::vector<int32_t> order(batch);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(),
                     [&](int32_t a, int32_t b) { return lengths_host[a] > lengths_host[b]; });

    const bool force = (flags & CRF_FORCE_SPILL) != 0;
    // Bundles take the strict chart layout when it fits in half a CU, or,
    // for a bundle that needs a whole CU in either layout, in the whole CU;
    // else the loose one (inside_layout, cky_layout).
    const int64_t half_cu = lds_cap / 2 - crf::kReservedLds, full_cu = lds_cap - crf::kReservedLds;
    auto strict_fits = [=](int64_t strict_bytes, int64_t loose_bytes) {
        return strict_bytes <= half_cu || (loose_bytes > half_cu && strict_bytes <= full_cu);
    };
    auto inside_strict = [=](int n, int64_t count) {
        return strict_fits(crf::inside_bundle_bytes(n, (int)count, true), crf::inside_bundle_bytes(n, (int)count, false));
    };
    auto inside_bundle_bytes = [=](int n, int64_t count) {
        return crf::inside_bundle_bytes(n, (int)count, inside_strict(n, count));
    };
    auto inside_spill_bytes = [](int n) { return 4 * (int64_t)crf::inside_layout(n, 1, true).cs; };
    auto cky_spill_bytes = [](int n) { return crf::cky_chart_bytes(n, 2); };
    // The CKY bundle's tail: padding so that the last chart's masked reads
    // (into the ids and the room behind it) stay inside the bundle.
    auto cky_tail = [](int n, int64_t count) {
        const int64_t tables = 4 * count + crf::bundle_extra_bytes(n);
        return std::max<int64_t>(0, 8 * (int64_t)crf::masked_reach(n) - tables);
    };
    // A sentence's split table sits in LDS after its chart when a bundle of
    // one such sentence still fits in half the CU; longer sentences keep it
    // in the workspace.
    auto split_in_lds = [=](int n) {
        return crf::cky_chart_bytes(n, 1) + 4 + crf::bundle_extra_bytes(n) + cky_tail(n, 1) <= half_cu;
    };
    // CKY bundle: the charts (with their split tables when they fit), the
    // ids (i32), the room of bundle_extra_bytes, the tail; the strict chart layout when it
    // fits in half a CU, else the loose one (cky_layout).
    auto cky_bytes_with = [=](int n, int64_t count, bool strict) {
        const int cs = crf::cky_layout(n, (int)count, split_in_lds(n) ? 1 : 0, strict).cs;
        return count * (cs + 4) + crf::bundle_extra_bytes(n) + cky_tail(n, count);
    };
    auto cky_strict = [=](int n, int64_t count) {
        return strict_fits(cky_bytes_with(n, count, true), cky_bytes_with(n, count, false));
    };
    auto cky_bundle_bytes = [=](int n, int64_t count) { return cky_bytes_with(n, count, cky_strict(n, count)); };
    HostSchedule si = make_schedule(order, lengths_host, lds_cap, force, 0, inside_bundle_bytes,
                                    inside_spill_bytes, kInsideTargetScale);
    HostSchedule sc = make_schedule(order, lengths_host, lds_cap, force, si.ws_bytes, cky_bundle_bytes,
                                    cky_spill_bytes, kCkyTargetScale);
    int64_t split_cursor = si.ws_bytes + sc.ws_bytes;
    std::vector<char> uses_ws(batch, 0);
    for (int32_t b : si.spill) uses_ws[b] = 1;
    for (int32_t b : sc.spill) uses_ws[b] = 1;
    for (crf::Bundle &bd : sc.bundles) {
        if (split_in_lds(bd.n)) continue;
        bd.split_ws = (int32_t)(split_cursor / 256);
        split_cursor += (bd.count * crf::cky_split_count(bd.n) + 255) / 256 * 256;
        p->split_ws_count += bd.count;
        for (int q = 0; q < bd.count; ++q) uses_ws[sc.order[bd.first + q]] = 1;
    }
    sc.ws_bytes = split_cursor - si.ws_bytes;

    // MBR decoding (unlabelled plans): bundles whose workgroup holds the
    // inside chart and then, in the same LDS, the CKY chart over the
    // marginals, so a bundle's LDS is the larger of the two.  Sentences past
    // LDS run on the inside and CKY workspace kernels, which must then list
    // the same sentences; if they do not, or no bundle is left, MBR decoding
    // runs as separate launches.
    HostSchedule sm;
    bool mbr_fused = num_labels == 1;
    if (mbr_fused) {
        auto mbr_bytes = [=](int n, int64_t count) {
            return std::max(inside_bundle_bytes(n, count), cky_bundle_bytes(n, count));
        };
        sm = make_schedule(order, lengths_host, lds_cap, force, 0, mbr_bytes, [](int) { return (int64_t)0; },
                           kCkyTargetScale);
        auto sorted = [](std::vector<int32_t> v) {
            std::sort(v.begin(), v.end());
            return v;
        };
        const std::vector<int32_t> ms = sorted(sm.spill);
        mbr_fused = !sm.bundles.empty() && ms == sorted(si.spill) && ms == sorted(sc.spill);
        if (mbr_fused)
            for (crf::Bundle &bd : sm.bundles) {
                if (split_in_lds(bd.n)) continue;
                bd.split_ws = (int32_t)(split_cursor / 256);
                split_cursor += (bd.count * crf::cky_split_count(bd.n) + 255) / 256 * 256;
            }
    }
    // Labelled plans: the label log-sum-exps and their marginals, [B][N1][N1]
    // float32 each, and the chunks of the label passes.
    std::vector<int32_t> lab_rows;
    int64_t lab_sp_off = 0, lab_mu_off = 0;
    if (num_labels > 1) {
        std::vector<char> in_ws(batch, 0);   // inside charts in the workspace: never in a bundle
        for (int32_t b : si.spill) in_ws[b] = 1;
        const int64_t plane = (int64_t)batch * n1 * n1 * 4;
        lab_sp_off = (split_cursor + 255) / 256 * 256;
        lab_mu_off = (lab_sp_off + plane + 255) / 256 * 256;
        split_cursor = lab_mu_off + plane;
        for (int32_t b = 0; b < batch; ++b) {
            const int n = lengths_host[b];
            if (n <= crf::kLabInBundleMaxN && !in_ws[b]) continue;   // its bundle does its own label I/O
            for (int i = 0; i < n; ++i)
                for (int64_t f0 = 0; f0 < (int64_t)(n - i) * num_labels; f0 += crf::kLabelRowChunk) {
                    lab_rows.push_back(b);
                    lab_rows.push_back(i);
                    lab_rows.push_back((int32_t)f0);
                    lab_rows.push_back(0);
                }
        }
        std::fill(uses_ws.begin(), uses_ws.end(), 1);
    }
    p->ws_bytes = split_cursor;
    p->workspace_users = (int32_t)std::count(uses_ws.begin(), uses_ws.end(), 1);

    // Biaffine scorer tiles: sentences of up to kBiaRows - 1 words packed
    // whole into tiles of kBiaRows fence posts (their scores are the tile's
    // diagonal blocks; longest first, each into the open tile with the least
    // room that still holds it, found through lists of open tiles by free
    // rows), longer ones cut into blocks of fence posts with a tile per pair
    // of row block <= column block.
    std::vector<int32_t> bia;
    {
        std::vector<std::vector<int32_t>> packed;
        std::vector<std::vector<int32_t>> by_free(crf::kBiaRows + 1);
        for (int32_t b : order) {
            const int n = lengths_host[b];
            if (n + 1 <= crf::kBiaRows) {
                int t = -1;
                for (int f = n + 1; f <= crf::kBiaRows && t < 0; ++f)
                    if (!by_free[f].empty()) {
                        t = by_free[f].back();
                        by_free[f].pop_back();
                    }
                if (t < 0) {
                    t = (int)packed.size();
                    packed.emplace_back();
                }
                for (int i = 0; i <= n; ++i) packed[t].push_back(b * n1 + i);
                const int room = crf::kBiaRows - (int)packed[t].size();
                if (room > 0) by_free[room].push_back(t);
                continue;
            }
            const int nblk = (n + 1 + crf::kBiaRows - 1) / crf::kBiaRows;
            for (int rb = 0; rb < nblk; ++rb)
                for (int cb = rb; cb < nblk; ++cb) {
                    for (int r = 0; r < crf::kBiaRows; ++r) {
                        const int i = rb * crf::kBiaRows + r;
                        bia.push_back(i <= n ? b * n1 + i : -1);
                    }
                    for (int c = 0; c < crf::kBiaCols; ++c) {
                        const int j = cb * crf::kBiaCols + c;
                        bia.push_back(j <= n ? b * n1 + j : -1);
                    }
                }
        }
        for (const auto &ids : packed)
            for (int h = 0; h < 2; ++h)
                for (int r = 0; r < crf::kBiaRows; ++r) bia.push_back(r < (int)ids.size() ? ids[r] : -1);
    }

    std::vector<int32_t> len(lengths_host, lengths_host + batch);
    crf::KernelPlan &kp = p->kp;
    kp.B = batch;
    kp.n1 = n1;
    kp.L = num_labels;
    std::vector<int32_t> mix;
    int32_t fused_slots = 0;
    if (num_labels == 1 && !si.bundles.empty() && !sc.bundles.empty() && si.threads == sc.threads) {
        // One workgroup slot per CU per half of the LDS; the fused kernel's
        // workgroups fill every slot and take bundles from one queue, in the
        // order they free up.
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, p->device) != hipSuccess || cus < 1)
            cus = 256;
        const int per_cu = std::min(4, std::max(1, (int)(lds_cap / std::max(si.lds_bytes, sc.lds_bytes))));
        fused_slots = cus * per_cu;
        auto fits = [&](bool inside, int n, int count) {
            return inside ? inside_bundle_bytes(n, count) <= si.lds_bytes : cky_bundle_bytes(n, count) <= sc.lds_bytes;
        };
        plan_fused_launch(si.bundles, sc.bundles, 1, fused_slots, mix, fits);
    }
    kp.n_mix = (int32_t)mix.size();
    kp.fused_grid = std::min<int32_t>(kp.n_mix, fused_slots);
    // Workgroup records: the bundle's shape and its sentence ids.
    int max_count = 1;
    for (const crf::Bundle &bd : si.bundles) max_count = std::max(max_count, (int)bd.count);
    for (const crf::Bundle &bd : sc.bundles) max_count = std::max(max_count, (int)bd.count);
    if (mbr_fused)
        for (const crf::Bundle &bd : sm.bundles) max_count = std::max(max_count, (int)bd.count);
    const int stride = crf::kRecHeader + max_count;
    kp.rec_stride = stride;
    auto put_inside_layout = [&](int32_t *q, int n, int count, int off) {
        const crf::InsideLayout l = crf::inside_layout(n, count, inside_strict(n, count));
        q[crf::kRecE + off] = l.e;
        q[crf::kRecLd + off] = l.ld;
        q[crf::kRecCs + off] = l.cs;
    };
    auto put_cky_layout = [&](int32_t *q, int n, int count, int off) {
        const crf::CkyLayout l = crf::cky_layout(n, count, split_in_lds(n) ? 1 : 0, cky_strict(n, count));
        q[crf::kRecE + off] = l.e;
        q[crf::kRecLd + off] = l.ld;
        q[crf::kRecCs + off] = l.cs;
    };
    constexpr int kSecond = crf::kRecE2 - crf::kRecE;   // offset of the second layout's fields
    auto records = [&](const HostSchedule &h, int kind) {
        std::vector<int32_t> r((size_t)h.bundles.size() * stride, 0);
        for (size_t b = 0; b < h.bundles.size(); ++b) {
            const crf::Bundle &bd = h.bundles[b];
            int32_t *q = r.data() + b * stride;
            q[crf::kRecN] = bd.n;
            q[crf::kRecCount] = bd.count;
            q[crf::kRecSplitWs] = kind == crf::kKindInside ? -1 : bd.split_ws;
            q[crf::kRecKind] = kind;
            q[crf::kRecLab] = kind == crf::kKindInside && num_labels > 1 && bd.n <= crf::kLabInBundleMaxN;
            if (kind == crf::kKindCky) {
                put_cky_layout(q, bd.n, bd.count, 0);
            } else {
                put_inside_layout(q, bd.n, bd.count, 0);
                if (kind == crf::kKindMbr) put_cky_layout(q, bd.n, bd.count, kSecond);
            }
            q[crf::kRecMagic] = (int32_t)crf::div_magic(bd.count);
            for (int t = 0; t < bd.count; ++t) q[crf::kRecHeader + t] = h.order[bd.first + t];
        }
        return r;
    };
    const std::vector<int32_t> rec_in = records(si, crf::kKindInside), rec_ck = records(sc, crf::kKindCky);
    const std::vector<int32_t> rec_mbr = mbr_fused ? records(sm, crf::kKindMbr) : std::vector<int32_t>();
    kp.n_lab_rows = (int32_t)(lab_rows.size() / 4);
    kp.n_bia_tiles = (int32_t)(bia.size() / (crf::kBiaRows + crf::kBiaCols));
    kp.lab_sp_off = lab_sp_off;
    kp.lab_mu_off = lab_mu_off;
    kp.n_mbr = mbr_fused ? (int32_t)sm.bundles.size() : 0;
    kp.mbr_lds = mbr_fused ? sm.lds_bytes : 0;
    kp.mbr_grid = 0;
    if (mbr_fused) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, p->device) != hipSuccess || cus < 1)
            cus = 256;
        const int per_cu = std::min(4, std::max(1, (int)(lds_cap / std::max(1, sm.lds_bytes))));
        kp.mbr_grid = std::min<int32_t>(kp.n_mbr, cus * per_cu);
    }
    std::vector<int32_t> rec_mix;
    rec_mix.reserve(mix.size() * stride);
    for (int32_t e : mix) {
        const int32_t *q = e >= 0 ? rec_in.data() + (size_t)e * stride : rec_ck.data() + (size_t)(~e) * stride;
        rec_mix.insert(rec_mix.end(), q, q + stride);
    }
    auto fill = [](crf::Schedule &q, const HostSchedule &h) {
        q.n_bundles = (int32_t)h.bundles.size();
        q.n_spill = (int32_t)h.spill.size();
        q.lds_bytes = h.lds_bytes;
        q.threads = h.threads;
    };
    fill(kp.inside, si);
    fill(kp.cky, sc);

    if ((e = upload(p, len, &kp.len)) != hipSuccess ||
        (e = upload(p, rec_in, &kp.inside.recs)) != hipSuccess ||
        (e = upload(p, si.spill, &kp.inside.order_spill)) != hipSuccess ||
        (e = upload(p, si.off, &kp.inside.ws_off)) != hipSuccess ||
        (e = upload(p, rec_ck, &kp.cky.recs)) != hipSuccess ||
        (e = upload(p, sc.spill, &kp.cky.order_spill)) != hipSuccess ||
        (e = upload(p, sc.off, &kp.cky.ws_off)) != hipSuccess ||
        (e = upload(p, rec_mix, &kp.mix)) != hipSuccess ||
        (e = upload(p, rec_mbr, &kp.mbr)) != hipSuccess ||
        (e = upload(p, lab_rows, &kp.lab_rows)) != hipSuccess ||
        (e = upload(p, bia, &kp.bia_tiles)) != hipSuccess) {
        const int code = (e == hipErrorOutOfMemory) ? CRF_ENOMEM : CRF_EHIP;
        release(p);
        delete p;
        return code == CRF_ENOMEM ? fail(code, "device allocation of the schedule failed")
                                  : hip_fail(e, "schedule upload");
    }
    kp.counter = nullptr;
    if (kp.fused_grid > 0 || kp.mbr_grid > 0) {
        void *c = nullptr;
        if ((e = hipMalloc(&c, 256)) != hipSuccess || (p->allocations.push_back(c), false) ||
            (e = hipMemset(c, 0, 256)) != hipSuccess) {
            release(p);
            delete p;
            return hip_fail(e, "claim counter");
        }
        kp.counter = static_cast<int32_t *>(c);
    }
    // Teams for the workspace sentences: the workgroups the device holds at
    // once, and the team area (none when no team of two fits).
    kp.team_area = nullptr;
    kp.team_cap = 0;
    kp.team_k = 1;
    if ((!si.spill.empty() || !sc.spill.empty()) && !(flags & CRF_NO_TEAMS)) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, p->device) != hipSuccess)
            (void)hipGetLastError(), cus = 0;
        kp.team_cap = std::max(0, cus) * crf::spill_blocks_per_cu();
        if (kp.team_cap >= 16) {
            void *a = nullptr;
            if ((e = hipMalloc(&a, (size_t)crf::kTeamAreaBytes)) != hipSuccess || (p->allocations.push_back(a), false)) {
                release(p);
                delete p;
                return hip_fail(e, "team area");
            }
            kp.team_area = static_cast<int32_t *>(a);
        }
    }
    kp.ws = nullptr;
    if (p->ws_bytes > 0) {
        void *ws = nullptr;
        e = hipMalloc(&ws, (size_t)p->ws_bytes);
        if (e != hipSuccess) {
            release(p);
            delete p;
            return fail(CRF_ENOMEM, "workspace of %lld bytes: %s", (long long)p->ws_bytes,
                        hipGetErrorString(e));
        }
        p->allocations.push_back(ws);
        kp.ws = static_cast<char *>(ws);
    }
    // Best effort: ROCm launches with any dynamic LDS up to the per-block
    // limit without this attribute; a real shortfall surfaces as a launch error.
    if (crf::set_kernel_attributes(std::max(std::max(si.lds_bytes, sc.lds_bytes), kp.mbr_lds)) != hipSuccess)
        (void)hipGetLastError();
    if (crf::set_biaffine_attributes() != hipSuccess) (void)hipGetLastError();
    // Resolve this device's scratch address for the no-allocation entry
    // point now (it retries, and reports a failure, on its first call).
    char *scr = nullptr;
    if (crf::scratch_address(p->device, &scr) != hipSuccess) (void)hipGetLastError();
    *out = p;
    return ok();
}

int crf_plan_destroy(crf_plan *plan) {
    if (plan == nullptr) return ok();
    int dev = -1;
    (void)hipGetDevice(&dev);
    if (dev != plan->device) (void)hipSetDevice(plan->device);
    hipError_t e = hipDeviceSynchronize();
    release(plan);
    if (dev >= 0 && dev != plan->device) (void)hipSetDevice(dev);
    delete plan;
    if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
    return ok();
}

int crf_plan_info(const crf_plan *plan, crf_plan_stats *out) {
    if (plan == nullptr || out == nullptr) return fail(CRF_EINVAL, "NULL argument");
    out->batch = plan->B;
    out->n1 = plan->n1;
    out->num_labels = plan->L;
    out->max_len = plan->max_len;
    out->lds_count = plan->B - plan->kp.inside.n_spill;
    out->spill_count = plan->kp.inside.n_spill;
    out->workspace_bytes = plan->ws_bytes;
    out->lds_bytes_inside = plan->kp.inside.lds_bytes;
    out->lds_bytes_cky = plan->kp.cky.lds_bytes;
    out->cky_spill_count = plan->kp.cky.n_spill;
    out->split_ws_count = plan->split_ws_count;
    out->workspace_users = plan->workspace_users;
    out->fused_queue = plan->kp.counter != nullptr ? 1 : 0;
    out->mbr_fused = plan->kp.mbr != nullptr ? 1 : 0;
    return ok();
}

static int check_device(const crf_plan *plan) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != plan->device)
        return fail(CRF_EINVAL, "plan was created on device %d, current device is %d",
                    plan->device, dev);
    return CRF_OK;
}

int crf_inside_fwd(const crf_plan *plan, const float *scores, float *logZ, void *stream) {
    if (plan == nullptr) return fail(CRF_EINVAL, "plan is NULL");
    if (scores == nullptr || logZ == nullptr) return fail(CRF_EINVAL, "scores/logZ is NULL");
    int rc = check_device(plan);
    if (rc != CRF_OK) return rc;
    hipError_t e = crf::launch_inside(plan->kp, scores, nullptr, logZ, nullptr,
                                      static_cast<hipStream_t>(stream));
    return e == hipSuccess ? ok() : hip_fail(e, "crf_inside_fwd launch");
}

int crf_inside_fwd_bwd(const crf_plan *plan, const float *scores, const float *grad_logZ,
                       float *logZ, float *marginals, void *stream) {
    if (plan == nullptr) return fail(CRF_EINVAL, "plan is NULL");
    if (scores == nullptr || marginals == nullptr)
        return fail(CRF_EINVAL, "scores/marginals is NULL");
    int rc = check_device(plan);
    if (rc != CRF_OK) return rc;
    hipError_t e = crf::launch_inside(plan->kp, scores, grad_logZ, logZ, marginals,
                                      static_cast<hipStream_t>(stream));
    return e == hipSuccess ? ok() : hip_fail(e, "crf_inside_fwd_bwd launch");
}

int crf_inside_bwd(const crf_plan *plan, const float *scores, const float *grad_logZ,
                   float *marginals, void *stream) {
    return crf_inside_fwd_bwd(plan, scores, grad_logZ, nullptr, marginals, stream);
}

int crf_inside_fwd_bwd_cky(const crf_plan *plan, const float *scores, const float *grad_logZ,
                           float *logZ, float *marginals, int32_t *spans, float *best,
                           void *stream) {
    if (plan == nullptr) return fail(CRF_EINVAL, "plan is NULL");
    if (scores == nullptr || marginals == nullptr || spans == nullptr)
        return fail(CRF_EINVAL, "scores/marginals/spans is NULL");
    if (plan->L != 1)
        return fail(CRF_EUNSUPPORTED, "CKY decode of labelled scores (L = %d)", plan->L);
    int rc = check_device(plan);
    if (rc != CRF_OK) return rc;
    hipError_t e = crf::launch_parse(plan->kp, scores, grad_logZ, logZ, marginals, spans, best,
                                     static_cast<hipStream_t>(stream));
    return e == hipSuccess ? ok() : hip_fail(e, "crf_inside_fwd_bwd_cky launch");
}

int crf_inside_fwd_bwd_cky_noalloc(const crf_plan *plan, const float *scores, const float *grad_logZ,
                                   float *logZ, float *marginals, int32_t *spans, float *best,
                                   void *stream) {
    if (plan == nullptr) return fail(CRF_EINVAL, "plan is NULL");
    if (scores == nullptr || marginals == nullptr || spans == nullptr)
        return fail(CRF_EINVAL, "scores/marginals/spans is NULL");
    if (plan->L != 1)
        return fail(CRF_EUNSUPPORTED, "CKY decode of labelled scores (L = %d)", plan->L);
    if (plan->ws_bytes > crf::kScratchBytes - crf::kScratchCounterBytes)
        return fail(CRF_EINVAL,
                    "the plan needs %lld bytes of workspace, more than the %lld bytes of static scratch "
                    "(use crf_inside_fwd_bwd_cky)",
                    (long long)plan->ws_bytes, (long long)(crf::kScratchBytes - crf::kScratchCounterBytes));
    int rc = check_device(plan);
    if (rc != CRF_OK) return rc;
    char *scr = nullptr;
    hipError_t e = crf::scratch_address(plan->device, &scr);
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    e = crf::launch_parse_scratch(plan->kp, scr, scores, grad_logZ, logZ, marginals, spans, best,
                                  static_cast<hipStream_t>(stream));
    return e == hipSuccess ? ok() : hip_fail(e, "crf_inside_fwd_bwd_cky_noalloc launch");
}

int crf_mbr_decode(const crf_plan *plan, const float *scores, float *logZ, float *marginals, int32_t *spans,
                   float *best, void *stream) {
    if (plan == nullptr) return fail(CRF_EINVAL, "plan is NULL");
    if (scores == nullptr || marginals == nullptr || spans == nullptr)
        return fail(CRF_EINVAL, "scores/marginals/spans is NULL");
    if (scores == marginals) return fail(CRF_EINVAL, "marginals must not alias scores");
    if (plan->L != 1) return fail(CRF_EUNSUPPORTED, "MBR decoding of labelled scores (L = %d)", plan->L);
    int rc = check_device(plan);
    if (rc != CRF_OK) return rc;
    hipError_t e = crf::launch_mbr(plan->kp, scores, logZ, marginals, spans, best, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? ok() : hip_fail(e, "crf_mbr_decode launch");
}

int crf_gold_loss(const crf_plan *plan, const float *scores, const int32_t *gold_spans, const float *grad_loss,
                  float *loss, float *grad_scores, void *stream) {
    if (plan == nullptr) return fail(CRF_EINVAL, "plan is NULL");
    if (scores == nullptr || gold_spans == nullptr || loss == nullptr || grad_scores == nullptr)
        return fail(CRF_EINVAL, "scores/gold_spans/loss/grad_scores is NULL");
    if (scores == grad_scores) return fail(CRF_EINVAL, "grad_scores must not alias scores");
    if (plan->L != 1) return fail(CRF_EUNSUPPORTED, "gold-tree loss of labelled scores (L = %d)", plan->L);
    int rc = check_device(plan);
    if (rc != CRF_OK) return rc;
    hipError_t e = crf::launch_loss(plan->kp, scores, gold_spans, grad_loss, loss, grad_scores,
                                    static_cast<hipStream_t>(stream));
    return e == hipSuccess ? ok() : hip_fail(e, "crf_gold_loss launch");
}

int crf_cky_decode_labeled(const crf_plan *plan, const float *scores, int32_t *spans, int32_t *labels, float *best,
                           void *stream) {
    if (plan == nullptr) return fail(CRF_EINVAL, "plan is NULL");
    if (scores == nullptr || spans == nullptr || labels == nullptr)
        return fail(CRF_EINVAL, "scores/spans/labels is NULL");
    int rc = check_device(plan);
    if (rc != CRF_OK) return rc;
    hipError_t e = crf::launch_cky(plan->kp, scores, spans, best, static_cast<hipStream_t>(stream), labels);
    return e == hipSuccess ? ok() : hip_fail(e, "crf_cky_decode_labeled launch");
}

int crf_label_spans(const crf_plan *plan, const float *label_scores, int32_t num_labels, const int32_t *spans,
                    int32_t *labels, void *stream) {
    if (plan == nullptr) return fail(CRF_EINVAL, "plan is NULL");
    if (label_scores == nullptr || spans == nullptr || labels == nullptr)
        return fail(CRF_EINVAL, "label_scores/spans/labels is NULL");
    if (num_labels < 1 || num_labels > CRF_MAX_LABELS)
        return fail(CRF_EINVAL, "num_labels %d outside [1, %d]", num_labels, CRF_MAX_LABELS);
    int rc = check_device(plan);
    if (rc != CRF_OK) return rc;
    hipError_t e = crf::launch_label_spans(plan->kp, label_scores, num_labels, spans, labels,
                                           static_cast<hipStream_t>(stream));
    return e == hipSuccess ? ok() : hip_fail(e, "crf_label_spans launch");
}

int crf_biaffine_scores(const crf_plan *plan, const uint16_t *rl, const uint16_t *rr, const uint16_t *w,
                        int32_t d, int32_t ldw, int32_t num_labels, float *scores, void *stream) {
    if (plan == nullptr) return fail(CRF_EINVAL, "plan is NULL");
    if (rl == nullptr || rr == nullptr || w == nullptr || scores == nullptr)
        return fail(CRF_EINVAL, "rl/rr/w/scores is NULL");
    if (d < 4 || d > crf::kBiaMaxD || d % 4 != 0)
        return fail(CRF_EINVAL, "d %d is not a multiple of 4 in [4, %d]", d, crf::kBiaMaxD);
    if (ldw < d + 1 || ldw % 4 != 0) return fail(CRF_EINVAL, "ldw %d < d+1 or not a multiple of 4", ldw);
    if (num_labels < 1 || num_labels > CRF_MAX_LABELS)
        return fail(CRF_EINVAL, "num_labels %d outside [1, %d]", num_labels, CRF_MAX_LABELS);
    if (((uintptr_t)rl | (uintptr_t)rr | (uintptr_t)w) & 7)
        return fail(CRF_EINVAL, "rl/rr/w must be 8-byte aligned");
    int rc = check_device(plan);
    if (rc != CRF_OK) return rc;
    hipError_t e = crf::launch_biaffine(plan->kp, rl, rr, w, d, ldw, num_labels, scores,
                                        static_cast<hipStream_t>(stream));
    return e == hipSuccess ? ok() : hip_fail(e, "crf_biaffine_scores launch");
}

int crf_cky_decode(const crf_plan *plan, const float *scores, int32_t *spans, float *best,
                   void *stream) {
    if (plan == nullptr) return fail(CRF_EINVAL, "plan is NULL");
    if (scores == nullptr || spans == nullptr) return fail(CRF_EINVAL, "scores/spans is NULL");
    if (plan->L != 1)
        return fail(CRF_EUNSUPPORTED, "CKY decode of labelled scores (L = %d)", plan->L);
    int rc = check_device(plan);
    if (rc != CRF_OK) return rc;
    hipError_t e = crf::launch_cky(plan->kp, scores, spans, best, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? ok() : hip_fail(e, "crf_cky_decode launch");
}

}  // extern "C"
