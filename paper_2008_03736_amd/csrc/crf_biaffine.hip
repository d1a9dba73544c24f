// crf_biaffine.hip -- the biaffine span scorer on gfx950 matrix cores.
//
// Sec. 2.2, Eq. biaffine: a span (i,j) of a sentence is scored from the left
// boundary representation of fence post i and the right one of fence post j,
//     s(i,j) = [r^l_i ; 1]^T W r^r_j,   W of (d+1) x d entries,
// one W per label for label scores (Sec. 2.2, label scoring): s(i,j,l).
// This is the producer of the CRF's span scores and the one dense
// contraction of the parser, so it runs on MFMA (bf16 inputs, fp32
// accumulation).
//
// Design.  A workgroup (four wavefronts, sixteen rows each) takes a tile of
// kBiaRows rows (left fence posts) and kBiaCols columns (right fence posts)
// -- short sentences packed whole into one tile (their scores are the tile's
// diagonal blocks), longer ones cut into row and column blocks -- and one
// label.  For each chunk of kBiaChunk of the d output dimensions of W it
// computes U = [R^l ; 1] W[:, chunk] (MFMA over K = d+1; each wavefront
// keeps its rows, with the 1 and the zero padding of K, as fragments in
// registers for the whole tile, and W's chunk is staged in LDS while the
// next one is loaded into registers), keeps U on chip as bf16 hi + lo parts
// (a 16-bit mantissa in all), and accumulates S += U R^r[:, chunk]^T (MFMA,
// two products for hi and lo).  U never leaves the CU; W is read once per
// tile from L2.  The chunk is narrow so that two workgroups share a CU and
// one's barriers and load latencies hide behind the other's products.  Only
// the valid cells 0 <= i < j <= n_b of S are written.
//
// MFMA v_mfma_f32_16x16x32_bf16 (gfx950): A 16 x 32, B 32 x 16, D 16 x 16;
// lane l supplies A row l%16 and B column l%16 at K offsets 8(l/16)..+7, and
// holds D rows 4(l/16)..+3 of column l%16.  The first product is taken as
// U^T = W^T [R^l ; 1]^T, so that a lane holds four consecutive columns of
// one row of U and stores them with one 8-byte write.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "crf_internal.h"

namespace crf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kPad = 8;                       // bf16 of padding per staged row (keeps 16-byte reads conflict-free)
constexpr int kUStride = kBiaChunk + kPad;    // row stride of the staged U and R^r chunks
constexpr int kWRows = kBiaChunk / 4;         // rows of a W chunk each wavefront stages

// Eight consecutive bf16 of a staged row as an MFMA operand.
__device__ __forceinline__ bf16x8 frag(const uint16_t *p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(p));
}

// K of the first product: d + 1 padded to 128, 256 or 512.
__host__ __device__ inline int bia_kp(int d) { return d + 1 <= 128 ? 128 : d + 1 <= 256 ? 256 : 512; }

// One chunk of W[:, c0 .. c0 + kBiaChunk)^T as this thread's share of the
// staged rows (wave w: rows kWRows w .. +kWRows; lane: pieces of four at
// lane, lane + 64): row c holds W[k][c0 + c] for k <= d (k = d: the bias),
// zeros after.  Loaded into registers, stored to LDS separately, so that the
// next chunk's loads fly while the current one is multiplied.  The loads are
// unconditional, from addresses clamped into the weights (row min(c, d-1),
// column min(k, d): at k = d the bias and three entries of the row's
// padding, ldw >= d + 4), and the masks are applied when the chunk is
// stored: a load whose result were used at once would wait out its whole L2
// latency there.  Rows are wave-uniform (scalar addresses).
// P = 4 or 8: bf16 per piece (8-byte or 16-byte loads; 16-byte pieces need
// 16-byte aligned rows, ldw a multiple of 8).
template <int KS, int P>
struct WChunk {
    static constexpr int H = (32 * KS / P + 63) / 64;   // pieces per lane and row
    using V = typename std::conditional<P == 8, uint4, uint2>::type;
    V v[kWRows][H];
};
template <int KS, int P>
__device__ __forceinline__ void load_w(WChunk<KS, P> &r, const uint16_t *wl, int c0, int d, int ldw, int wv,
                                       int lane) {
    using V = typename WChunk<KS, P>::V;
    // scalar row base + one 32-bit lane offset per piece (saddr form); the
    // last piece is the one holding k = d (the bias), inside the row since
    // ldw >= d + 1 is a multiple of P
    const int dp = d - d % P;
    uint32_t ko[WChunk<KS, P>::H];
#pragma unroll
    for (int h = 0; h < WChunk<KS, P>::H; ++h) ko[h] = 2u * (uint32_t)min(P * (lane + 64 * h), dp);   // bytes
#pragma unroll
    for (int rr_ = 0; rr_ < kWRows; ++rr_) {
        const char *row = reinterpret_cast<const char *>(wl + (size_t)min(c0 + kWRows * wv + rr_, d - 1) * ldw);
#pragma unroll
        for (int h = 0; h < WChunk<KS, P>::H; ++h) r.v[rr_][h] = *reinterpret_cast<const V *>(row + ko[h]);
    }
}
// Keep the bf16 at k .. k+1 of a 32-bit word when each is <= d (k = d: the bias).
__device__ __forceinline__ uint32_t keep2(uint32_t x, int k, int d) {
    return x & ((k <= d ? 0x0000FFFFu : 0u) | (k + 1 <= d ? 0xFFFF0000u : 0u));
}
template <int KS, int P>
__device__ __forceinline__ void store_w(const WChunk<KS, P> &r, uint16_t *Ws, int lda, int c0, int d, int wv,
                                        int lane) {
    using V = typename WChunk<KS, P>::V;
#pragma unroll
    for (int h = 0; h < WChunk<KS, P>::H; ++h) {
        const int k = P * (lane + 64 * h);
        if (k >= 32 * KS) continue;
#pragma unroll
        for (int rr_ = 0; rr_ < kWRows; ++rr_) {
            const bool row = c0 + kWRows * wv + rr_ < d;
            V v = r.v[rr_][h];
            v.x = row ? keep2(v.x, k, d) : 0u;
            v.y = row ? keep2(v.y, k + 2, d) : 0u;
            if constexpr (P == 8) {
                v.z = row ? keep2(v.z, k + 4, d) : 0u;
                v.w = row ? keep2(v.w, k + 6, d) : 0u;
            }
            *reinterpret_cast<V *>(Ws + (kWRows * wv + rr_) * lda + k) = v;
        }
    }
}

// Tile record: kBiaRows row ids then kBiaCols column ids, each b * N1 + i
// (sentence b, fence post i) or -1.  KS = K / 32 steps of the first product
// (K = d + 1 padded to 128, 256 or 512), taken in groups of kGrp steps whose
// fragments are read from LDS while the previous group is multiplied.
constexpr int kGrp = 2;
constexpr int kRAhead = 3;   // chunks of r^r in flight
template <int KS, int P>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void biaffine_kernel(
    const int32_t *__restrict__ tiles, const int32_t *__restrict__ len, int N1, int d, int ldw, int L,
    const uint16_t *__restrict__ rl, const uint16_t *__restrict__ rr, const uint16_t *__restrict__ w,
    float *__restrict__ scores) {
    extern __shared__ __align__(16) char smem_raw[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    constexpr int Kp = 32 * KS;              // K of the first product
    constexpr int NC = kBiaChunk / 16;       // 16-column blocks of a chunk
    constexpr int NG = KS / kGrp < 1 ? 1 : KS / kGrp;
    constexpr int GS = KS / NG;              // steps per group
    const int lda = Kp + kPad;
    uint16_t *Ws = reinterpret_cast<uint16_t *>(smem_raw);   // [kBiaChunk][lda]: W[:, chunk]^T
    uint16_t *Rs = Ws + kBiaChunk * lda;                     // [kBiaCols][kUStride]: r^r[:, chunk]
    uint16_t *Uh = Rs + kBiaCols * kUStride;                 // [kBiaRows][kUStride]: U hi
    uint16_t *Ul = Uh + kBiaRows * kUStride;                 // [kBiaRows][kUStride]: U lo
    int32_t *Ob = reinterpret_cast<int32_t *>(Ul + kBiaRows * kUStride);   // [kBiaRows + kBiaCols]
    int32_t *Oi = Ob + kBiaRows + kBiaCols;                                // [kBiaRows + kBiaCols]
    int32_t *On = Oi + kBiaRows + kBiaCols;                                // [kBiaRows]
    const int32_t *rec = tiles + (size_t)blockIdx.x * (kBiaRows + kBiaCols);
    const int l = blockIdx.y;
    const uint16_t *wl = w + (size_t)l * d * ldw;

    // Issue the first W chunk's loads before anything waits.
    WChunk<KS, P> wn;
    load_w<KS, P>(wn, wl, 0, d, ldw, wv, lane);

    // r^r of the tile's columns: thread t stages column t/4, dimensions
    // 8 (t%4) .. +7 of each chunk (two loads of four: rows are 8-byte
    // aligned).  These are scattered pieces of rows in HBM, whose latency is
    // longer than a chunk's products: they are loaded kRAhead chunks ahead
    // (rn[c % kRAhead] holds chunk c's pieces).
    const int sj = tid >> 2, sk = 8 * (tid & 3);
    const int cid = rec[kBiaRows + sj];
    const uint16_t *crow = rr + (size_t)(cid >= 0 ? cid : 0) * d;
    uint2 rn[kRAhead][2];
#pragma unroll
    for (int a = 0; a < kRAhead; ++a)
#pragma unroll
        for (int h = 0; h < 2; ++h)
            rn[a][h] = *reinterpret_cast<const uint2 *>(crow + min(kBiaChunk * a + sk + 4 * h, d - 4));

    // This wave's rows [r^l_i ; 1 ; 0 ...] as MFMA fragments, in registers
    // for the whole tile: row 16 wave + lane%16, K offsets k0 + 8 (lane/16).
    uint2 afr[KS][2];
    {
        const int id = rec[16 * wave + (lane & 15)];
        const uint16_t *row = rl + (size_t)(id >= 0 ? id : 0) * d;
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
            for (int h = 0; h < 2; ++h)
                afr[s][h] = *reinterpret_cast<const uint2 *>(row + min(32 * s + 8 * (lane >> 4) + 4 * h, d - 4));
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int k = 32 * s + 8 * (lane >> 4) + 4 * h;
                uint2 v = id >= 0 && k < d ? afr[s][h] : make_uint2(0u, 0u);
                if (k == d) v.x = 0x3F80u;                   // the appended 1 (k = d, a multiple of 4)
                afr[s][h] = v;
            }
    }

    // Where the tile's cells of S go, decoded once into LDS (read back by the
    // final writes, so that they wait on no memory): per row and column its
    // sentence (-1 / -2: none) and fence post, per row the sentence length.
    if (tid < kBiaRows + kBiaCols) {
        const int id = rec[tid];
        const int b = id >= 0 ? id / N1 : tid < kBiaRows ? -1 : -2;
        Ob[tid] = b;
        Oi[tid] = id - b * N1;
        if (tid < kBiaRows) On[tid] = len[b >= 0 ? b : 0];
    }

    f32x4 acc[kBiaCols / 16];   // S rows 16 wave + 4 (lane/16) + t, columns 16 c + lane%16
#pragma unroll
    for (int c = 0; c < kBiaCols / 16; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};

    // (the chunk loop runs in steps of kRAhead chunks so that the slot of
    // rn each chunk uses is a compile-time index)
    for (int cb = 0; cb < d; cb += kRAhead * kBiaChunk) {
#pragma unroll
    for (int a = 0; a < kRAhead; ++a) {
        const int c0 = cb + a * kBiaChunk;
        if (c0 >= d) break;
        __syncthreads();   // the previous chunk's readers are done
        store_w<KS, P>(wn, Ws, lda, c0, d, wv, lane);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const uint2 v = cid >= 0 && c0 + sk + 4 * h < d ? rn[a][h] : make_uint2(0u, 0u);
            *reinterpret_cast<uint2 *>(Rs + sj * kUStride + sk + 4 * h) = v;
        }
        if (c0 + kBiaChunk < d)   // the next chunk's W flies during this one's products
            load_w<KS, P>(wn, wl, c0 + kBiaChunk, d, ldw, wv, lane);
        if (c0 + kRAhead * kBiaChunk < d) {   // and r^r kRAhead chunks ahead
#pragma unroll
            for (int h = 0; h < 2; ++h)
                rn[a][h] = *reinterpret_cast<const uint2 *>(crow + min(c0 + kRAhead * kBiaChunk + sk + 4 * h, d - 4));
        }
        __syncthreads();

        // U^T[chunk][16 wave .. +16] = W[:, chunk]^T [r^l ; 1]^T
        f32x4 u[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) u[c] = f32x4{0.f, 0.f, 0.f, 0.f};
        const uint16_t *wrow = Ws + (lane & 15) * lda + 8 * (lane >> 4);
        bf16x8 bw[2][GS][NC];
#pragma unroll
        for (int s = 0; s < GS; ++s)
#pragma unroll
            for (int c = 0; c < NC; ++c) bw[0][s][c] = frag(wrow + 16 * c * lda + 32 * s);
#pragma unroll
        for (int g = 0; g < NG; ++g) {
            if (g + 1 < NG) {
#pragma unroll
                for (int s = 0; s < GS; ++s)
#pragma unroll
                    for (int c = 0; c < NC; ++c)
                        bw[(g + 1) & 1][s][c] = frag(wrow + 16 * c * lda + 32 * ((g + 1) * GS + s));
            }
            // keep the next group's reads ahead of this group's products (the
            // scheduler would otherwise pair each read with its product and
            // wait out the LDS latency at every one)
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int s = 0; s < GS; ++s) {
                const int ks = g * GS + s;
                const bf16x8 a =
                    __builtin_bit_cast(bf16x8, make_uint4(afr[ks][0].x, afr[ks][0].y, afr[ks][1].x, afr[ks][1].y));
#pragma unroll
                for (int c = 0; c < NC; ++c)
                    u[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bw[g & 1][s][c], a, u[c], 0, 0, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        // U to LDS as bf16 hi + lo: row 16 wave + lane%16, columns
        // 16 c + 4 (lane/16) .. +3
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const bf16x4 hi = __builtin_convertvector(u[c], bf16x4);
            const f32x4 rest = u[c] - __builtin_convertvector(hi, f32x4);
            const bf16x4 lo = __builtin_convertvector(rest, bf16x4);
            const int o = (16 * wave + (lane & 15)) * kUStride + 16 * c + 4 * (lane >> 4);
            *reinterpret_cast<bf16x4 *>(Uh + o) = hi;
            *reinterpret_cast<bf16x4 *>(Ul + o) = lo;
        }
        __syncthreads();

        // S[16 wave .. +16][columns] += U R^r[:, chunk]^T, hi and lo parts
        const int urow = (16 * wave + (lane & 15)) * kUStride + 8 * (lane >> 4);
        bf16x8 ah[kBiaChunk / 32], al[kBiaChunk / 32], br[kBiaChunk / 32][kBiaCols / 16];
#pragma unroll
        for (int k = 0; k < kBiaChunk / 32; ++k) {
            ah[k] = frag(Uh + urow + 32 * k);
            al[k] = frag(Ul + urow + 32 * k);
#pragma unroll
            for (int c = 0; c < kBiaCols / 16; ++c)
                br[k][c] = frag(Rs + (16 * c + (lane & 15)) * kUStride + 32 * k + 8 * (lane >> 4));
        }
#pragma unroll
        for (int k = 0; k < kBiaChunk / 32; ++k)
#pragma unroll
            for (int c = 0; c < kBiaCols / 16; ++c) {
                acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[k], br[k][c], acc[c], 0, 0, 0);
                acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[k], br[k][c], acc[c], 0, 0, 0);
            }
    }
    }

    // The valid cells: row and column of one sentence, i < j <= n_b.
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const int r = 16 * wave + 4 * (lane >> 4) + t;
        const int b = Ob[r], i = Oi[r], n = On[r];
#pragma unroll
        for (int c = 0; c < kBiaCols / 16; ++c) {
            const int q = kBiaRows + 16 * c + (lane & 15), j = Oi[q];
            if (b == Ob[q] && i < j && j <= n) scores[(((size_t)b * N1 + i) * N1 + j) * L + l] = acc[c][t];
        }
    }
}

}  // namespace

hipError_t set_biaffine_attributes() {
    const void *fns[] = {(const void *)biaffine_kernel<4, 4>,  (const void *)biaffine_kernel<8, 4>,
                         (const void *)biaffine_kernel<16, 4>, (const void *)biaffine_kernel<4, 8>,
                         (const void *)biaffine_kernel<8, 8>,  (const void *)biaffine_kernel<16, 8>};
    const int lds[] = {(int)biaffine_lds_bytes(127), (int)biaffine_lds_bytes(255), (int)biaffine_lds_bytes(kBiaMaxD)};
    for (int k = 0; k < 6; ++k) {
        const hipError_t e = hipFuncSetAttribute(fns[k], hipFuncAttributeMaxDynamicSharedMemorySize, lds[k % 3]);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

int64_t biaffine_lds_bytes(int d) {
    const int64_t lda = bia_kp(d) + kPad;
    return 2 * (kBiaChunk * lda + (kBiaCols + 2 * kBiaRows) * (int64_t)kUStride) +
           4 * (2 * (kBiaRows + kBiaCols) + kBiaRows);
}

template <int P>
static void launch_biaffine_p(const KernelPlan &p, dim3 grid, size_t lds, hipStream_t stream, const uint16_t *rl,
                              const uint16_t *rr, const uint16_t *w, int d, int ldw, int L, float *scores) {
    const dim3 block(256);
    const int kp = bia_kp(d);
    if (kp == 128)
        hipLaunchKernelGGL((biaffine_kernel<4, P>), grid, block, lds, stream, p.bia_tiles, p.len, p.n1, d, ldw, L, rl,
                           rr, w, scores);
    else if (kp == 256)
        hipLaunchKernelGGL((biaffine_kernel<8, P>), grid, block, lds, stream, p.bia_tiles, p.len, p.n1, d, ldw, L, rl,
                           rr, w, scores);
    else
        hipLaunchKernelGGL((biaffine_kernel<16, P>), grid, block, lds, stream, p.bia_tiles, p.len, p.n1, d, ldw, L, rl,
                           rr, w, scores);
}

hipError_t launch_biaffine(const KernelPlan &p, const uint16_t *rl, const uint16_t *rr, const uint16_t *w, int d,
                           int ldw, int L, float *scores, hipStream_t stream) {
    if (p.n_bia_tiles < 1) return hipSuccess;
    const size_t lds = (size_t)biaffine_lds_bytes(d);
    const dim3 grid(p.n_bia_tiles, L);
    // 16-byte W pieces when every row starts 16-byte aligned
    if (ldw % 8 == 0 && ((uintptr_t)w & 15) == 0)
        launch_biaffine_p<8>(p, grid, lds, stream, rl, rr, w, d, ldw, L, scores);
    else
        launch_biaffine_p<4>(p, grid, lds, stream, rl, rr, w, d, ldw, L, scores);
    return hipGetLastError();
}

}  // namespace crf
