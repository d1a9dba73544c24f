// Host-only build of the plan code for the CPU tests: the HIP runtime calls
// the plan makes are served from host memory (no device is touched), and
// the launch entry points are never called.  Prints the plan's records:
//   P n_mix fused_grid lds_inside lds_cky half_cu
//   W spill cky_spill split_ws workspace_users workspace_bytes fused_queue
//   R kind n count split_ws strict ld cs e bytes id...
// one R line per record of the fused queue, in queue order; M lines for the
// MBR bundles, I lines for labelled plans' inside bundles, T lines for the
// biaffine scorer's tiles.  Arguments: a file
// of sentence lengths, and optionally the number of labels.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "../paper_2008_03736_amd/csrc/crf_plan.cpp"

extern "C" {
hipError_t hipGetDevice(int *d) {
    *d = 0;
    return hipSuccess;
}
hipError_t hipSetDevice(int) { return hipSuccess; }
hipError_t hipDeviceGetAttribute(int *v, hipDeviceAttribute_t a, int) {
    *v = a == hipDeviceAttributeMaxSharedMemoryPerBlock ? 163840 : 256;   // MI355X: 160 KiB, 256 CUs
    return hipSuccess;
}
hipError_t hipMalloc(void **p, size_t n) {
    *p = std::malloc(n ? n : 1);
    return *p ? hipSuccess : hipErrorOutOfMemory;
}
hipError_t hipFree(void *p) {
    std::free(p);
    return hipSuccess;
}
hipError_t hipMemcpy(void *d, const void *s, size_t n, hipMemcpyKind) {
    std::memcpy(d, s, n);
    return hipSuccess;
}
hipError_t hipMemset(void *d, int v, size_t n) {
    std::memset(d, v, n);
    return hipSuccess;
}
hipError_t hipDeviceSynchronize() { return hipSuccess; }
hipError_t hipGetLastError() { return hipSuccess; }
const char *hipGetErrorString(hipError_t) { return "host stub"; }
}

namespace crf {
hipError_t launch_inside(const KernelPlan &, const float *, const float *, float *, float *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_cky(const KernelPlan &, const float *, int32_t *, float *, hipStream_t, int32_t *) {
    return hipErrorNotSupported;
}
hipError_t launch_mbr(const KernelPlan &, const float *, float *, float *, int32_t *, float *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_loss(const KernelPlan &, const float *, const int32_t *, const float *, float *, float *,
                       hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_label_spans(const KernelPlan &, const float *, int, const int32_t *, int32_t *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_parse(const KernelPlan &, const float *, const float *, float *, float *, int32_t *, float *,
                        hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t set_kernel_attributes(int) { return hipSuccess; }
int spill_blocks_per_cu() { return 1; }
int64_t biaffine_lds_bytes(int) { return 0; }
hipError_t set_biaffine_attributes() { return hipSuccess; }
hipError_t launch_biaffine(const KernelPlan &, const uint16_t *, const uint16_t *, const uint16_t *, int, int, int,
                           float *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t scratch_address(int, char **out) {
    *out = nullptr;
    return hipErrorNotSupported;
}
hipError_t launch_parse_scratch(const KernelPlan &, char *, const float *, const float *, float *, float *, int32_t *,
                                float *, hipStream_t) {
    return hipErrorNotSupported;
}
}  // namespace crf

int main(int argc, char **argv) {
    if (argc < 2) return 2;
    if (std::strcmp(argv[1], "runs") == 0) {   // shape_run_end against step_shape_k, K = 1 .. 5000
        const int top = 5000;
        for (int K = 1; K <= top; ++K) {
            const crf::StepShape s = crf::step_shape_k(K);
            const int e = crf::shape_run_end(K);
            if (e <= K) { std::printf("BAD %d end %d\n", K, e); return 1; }
            for (int k = K; k < std::min(e, top + 1); ++k) {
                const crf::StepShape t = crf::step_shape_k(k);
                if (t.G != s.G || t.C != s.C || t.MF != s.MF) { std::printf("BAD %d end %d at %d\n", K, e, k); return 1; }
            }
            if (e <= top) {
                const crf::StepShape t = crf::step_shape_k(e);
                if (t.G == s.G && t.C == s.C) { std::printf("BAD %d end %d same shape\n", K, e); return 1; }
            }
        }
        std::printf("RUNS OK\n");
        return 0;
    }
    if (std::strcmp(argv[1], "teams") == 0) {   // S jobs cap k grid: the workspace launch shapes
        for (int cap : {0, 8, 16, 32, 64, 256, 512, 1024})
            for (int jobs = 0; jobs <= 300; ++jobs) {
                const crf::TeamShape t = crf::team_shape(jobs, cap, true);
                std::printf("S %d %d %d %d\n", jobs, cap, t.k, t.grid);
            }
        const crf::TeamShape t = crf::team_shape(5, 256, false);
        std::printf("N %d %d\n", t.k, t.grid);
        return 0;
    }
    std::vector<int32_t> len;
    FILE *f = std::fopen(argv[1], "r");
    if (!f) return 2;
    int x;
    while (std::fscanf(f, "%d", &x) == 1) len.push_back(x);
    std::fclose(f);
    int n1 = 2;
    for (int v : len) n1 = std::max(n1, v + 1);
    crf_plan *p = nullptr;
    const int labels = argc > 2 ? std::atoi(argv[2]) : 1;
    const uint32_t flags = argc > 3 ? (uint32_t)std::atoi(argv[3]) : 0u;
    const int rc = crf_plan_create(&p, len.data(), (int32_t)len.size(), n1, labels, flags);
    if (rc != CRF_OK) {
        std::printf("E %d\n", rc);
        return 1;
    }
    const crf::KernelPlan &kp = p->kp;
    const int half_cu = 163840 / 2 - crf::kReservedLds;
    std::printf("P %d %d %d %d %d\n", kp.n_mix, kp.fused_grid, kp.inside.lds_bytes, kp.cky.lds_bytes, half_cu);
    crf_plan_stats st;
    if (crf_plan_info(p, &st) != CRF_OK) {
        std::printf("E info\n");
        return 1;
    }
    std::printf("W %d %d %d %d %lld %d\n", st.spill_count, st.cky_spill_count, st.split_ws_count, st.workspace_users,
                (long long)st.workspace_bytes, st.fused_queue);
    std::printf("Q %d %d\n", kp.team_cap, kp.team_area != nullptr ? 1 : 0);
    for (int b = 0; b < kp.n_mix; ++b) {
        const int32_t *r = kp.mix + (size_t)b * kp.rec_stride;
        const int n = r[crf::kRecN], count = r[crf::kRecCount], split_ws = r[crf::kRecSplitWs];
        const int kind = r[crf::kRecKind], e = r[crf::kRecE], ld = r[crf::kRecLd], cs = r[crf::kRecCs];
        if ((uint32_t)r[crf::kRecMagic] != crf::div_magic(count)) {
            std::printf("E magic\n");
            return 1;
        }
        // which layout the plan chose: the strict one if the record holds it
        int strict;
        long long bytes = -1;   // (the CKY tail is the plan's; the test checks the strides)
        if (kind == 1) {
            const crf::InsideLayout l = crf::inside_layout(n, count, true);
            strict = l.ld == ld && l.cs == cs && l.e == e;
            bytes = crf::inside_bundle_bytes(n, count, strict != 0);
        } else {
            const crf::CkyLayout l = crf::cky_layout(n, count, split_ws < 0 ? 1 : 0, true);
            strict = l.ld == ld && l.cs == cs && l.e == e;
        }
        std::printf("R %d %d %d %d %d %d %d %d %lld", kind, n, count, split_ws, strict, ld, cs, e, bytes);
        for (int t = 0; t < count; ++t) std::printf(" %d", r[crf::kRecHeader + t]);
        std::printf("\n");
    }
    // MBR bundles, as
    //   M n count split_ws inside_strict cky_strict mbr_grid mbr_lds id...
    for (int b = 0; b < kp.n_mbr; ++b) {
        const int32_t *r = kp.mbr + (size_t)b * kp.rec_stride;
        const int n = r[crf::kRecN], count = r[crf::kRecCount];
        const crf::InsideLayout li = crf::inside_layout(n, count, true);
        const crf::CkyLayout lc = crf::cky_layout(n, count, r[crf::kRecSplitWs] < 0 ? 1 : 0, true);
        const int si = li.ld == r[crf::kRecLd] && li.cs == r[crf::kRecCs] && li.e == r[crf::kRecE];
        const int sc = lc.ld == r[crf::kRecLd2] && lc.cs == r[crf::kRecCs2] && lc.e == r[crf::kRecE2];
        if (r[crf::kRecKind] != crf::kKindMbr) {
            std::printf("E kind\n");
            return 1;
        }
        const long long ib = crf::inside_bundle_bytes(n, count, si != 0);
        std::printf("M %d %d %d %d %d %d %d %lld", n, count, r[crf::kRecSplitWs], si, sc, kp.mbr_grid, kp.mbr_lds, ib);
        for (int t = 0; t < count; ++t) std::printf(" %d", r[crf::kRecHeader + t]);
        std::printf("\n");
    }
    // Labelled plans have no fused queue: their inside bundles, as
    //   I n count id...
    for (int b = 0; kp.n_mix == 0 && b < kp.inside.n_bundles; ++b) {
        const int32_t *r = kp.inside.recs + (size_t)b * kp.rec_stride;
        std::printf("I %d %d", r[crf::kRecN], r[crf::kRecCount]);
        for (int t = 0; t < r[crf::kRecCount]; ++t) std::printf(" %d", r[crf::kRecHeader + t]);
        std::printf("\n");
    }
    // Biaffine scorer tiles, as
    //   T n1 row_id x kBiaRows col_id x kBiaCols   (b n1 + fence post, or -1)
    for (int t = 0; t < kp.n_bia_tiles; ++t) {
        const int32_t *r = kp.bia_tiles + (size_t)t * (crf::kBiaRows + crf::kBiaCols);
        std::printf("T %d", n1);
        for (int k = 0; k < crf::kBiaRows + crf::kBiaCols; ++k) std::printf(" %d", r[k]);
        std::printf("\n");
    }
    crf_plan_destroy(p);
    return 0;
}
