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
// Design.  A workgroup (four wavefronts) takes a tile of kBiaRows rows (left
// fence posts) and kBiaCols columns (right fence posts) -- short sentences
// packed whole into one tile (their scores are the tile's diagonal blocks),
// longer ones cut into row and column blocks -- and one label.  For each
// chunk of kBiaChunk of the d output dimensions of W it computes
// U = [R^l ; 1] W[:, chunk] on MFMA with K = d+1 split four ways: wavefront w
// keeps the tile's 64 rows over its quarter of K (with the 1 and the zero
// padding) as fragments in registers for the whole tile, loads its quarter of
// W's chunk straight from L2 into registers (each W fragment feeds four
// products, and W never passes through LDS), and the four partial sums meet
// in LDS.  U stays on chip as bf16 hi + lo parts (a 16-bit mantissa in all),
// and S += U R^r[:, chunk]^T (MFMA, two products for hi and lo) accumulates
// sixteen rows per wavefront.  Only the valid cells 0 <= i < j <= n_b of S
// are written.
//
// MFMA v_mfma_f32_16x16x32_bf16 (gfx950): A 16 x 32, B 32 x 16, D 16 x 16;
// lane l supplies A row l%16 and B column l%16 at K offsets 8(l/16)..+7, and
// holds D rows 4(l/16)..+3 of column l%16.  The first product is taken as
// U^T = W^T [R^l ; 1]^T: W is stored transposed, so an A fragment is eight
// consecutive entries of one stored row, and a lane's D holds four
// consecutive columns of one row of U.
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
constexpr int kPStride = kBiaChunk + 4;       // row stride (floats) of the staged partial sums of U
constexpr int kNM = kBiaChunk / 16;           // 16-column blocks of U in a chunk
constexpr int kNN = kBiaRows / 16;            // 16-row blocks of the tile

// Eight consecutive bf16 of a staged row as an MFMA operand.
__device__ __forceinline__ bf16x8 frag(const uint16_t *p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(p));
}
__device__ __forceinline__ bf16x8 frag(const uint4 &v) { return __builtin_bit_cast(bf16x8, v); }

// K of the first product: d + 1 padded to 128, 256 or 512.
__host__ __device__ inline int bia_kp(int d) { return d + 1 <= 128 ? 128 : d + 1 <= 256 ? 256 : 512; }

// This wavefront's A fragments of one chunk: W^T rows c0 + 16 m + lane%16
// (clamped to row d-1: the columns of U past d meet zero r^r entries), K
// offsets kq0 + 32 s + 8 (lane/16) .. +7.  P = 8 or 4: one 16-byte load or
// two 8-byte loads (16-byte pieces need 16-byte aligned rows, ldw a multiple
// of 8).  Offsets are clamped to the piece that holds k = d (the bias), which
// lies inside the row since ldw >= d + 1 is a multiple of P; what a clamped
// or partial piece brings past k = d is masked off at use (wmask).
template <int KQ, int P>
__device__ __forceinline__ void load_wq(uint4 (&f)[kNM][KQ], const uint16_t *wl, int c0, int d, int ldw, int kq0,
                                        int lane) {
    const int dp = d - d % P;
#pragma unroll
    for (int m = 0; m < kNM; ++m) {
        const uint16_t *row = wl + (size_t)min(c0 + 16 * m + (lane & 15), d - 1) * ldw;
#pragma unroll
        for (int s = 0; s < KQ; ++s) {
            const int k = kq0 + 32 * s + 8 * (lane >> 4);
            if constexpr (P == 8) {
                f[m][s] = *reinterpret_cast<const uint4 *>(row + min(k, dp));
            } else {
                const uint2 a = *reinterpret_cast<const uint2 *>(row + min(k, dp));
                const uint2 b = *reinterpret_cast<const uint2 *>(row + min(k + 4, dp));
                f[m][s] = make_uint4(a.x, a.y, b.x, b.y);
            }
        }
    }
}
// Bits of a fragment's four words that hold entries k <= d (k: its first entry).
__device__ __forceinline__ uint32_t keep_word(int k, int d) {
    return (k <= d ? 0x0000FFFFu : 0u) | (k + 1 <= d ? 0xFFFF0000u : 0u);
}

// Tile record: kBiaRows row ids then kBiaCols column ids, each b * N1 + i
// (sentence b, fence post i) or -1.  KS = K / 32 steps of the first product
// (K = d + 1 padded to 128, 256 or 512); each wavefront takes KS / 4 of them.
constexpr int kRAhead = 3;   // chunks of r^r in flight
template <int KS, int P>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void biaffine_kernel(
    const int32_t *__restrict__ tiles, const int32_t *__restrict__ len, int N1, int d, int ldw, int L,
    const uint16_t *__restrict__ rl, const uint16_t *__restrict__ rr, const uint16_t *__restrict__ w,
    float *__restrict__ scores) {
    static_assert(KS % 4 == 0, "K splits four ways");
    constexpr int KQ = KS / 4;               // steps of this wavefront's quarter of K
    extern __shared__ __align__(16) char smem_raw[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int kq0 = 32 * KQ * __builtin_amdgcn_readfirstlane(wave);   // first K of this wavefront
    float *Ps = reinterpret_cast<float *>(smem_raw);                   // [4][kBiaRows][kPStride]: partial U
    uint16_t *Rs = reinterpret_cast<uint16_t *>(Ps + 4 * kBiaRows * kPStride);   // [kBiaCols][kUStride]: r^r[:, chunk]
    uint16_t *Uh = Rs + kBiaCols * kUStride;                 // [kBiaRows][kUStride]: U hi
    uint16_t *Ul = Uh + kBiaRows * kUStride;                 // [kBiaRows][kUStride]: U lo
    int32_t *Ob = reinterpret_cast<int32_t *>(Ul + kBiaRows * kUStride);   // [kBiaRows + kBiaCols]
    int32_t *Oi = Ob + kBiaRows + kBiaCols;                                // [kBiaRows + kBiaCols]
    int32_t *On = Oi + kBiaRows + kBiaCols;                                // [kBiaRows]
    const int32_t *rec = tiles + (size_t)blockIdx.x * (kBiaRows + kBiaCols);
    const int l = blockIdx.y;
    const uint16_t *wl = w + (size_t)l * d * ldw;

    // Issue the first W chunk's loads before anything waits.
    uint4 wf[kNM][KQ];
    load_wq<KQ, P>(wf, wl, 0, d, ldw, kq0, lane);
    uint4 wmask[KQ];
#pragma unroll
    for (int s = 0; s < KQ; ++s) {
        const int k = kq0 + 32 * s + 8 * (lane >> 4);
        wmask[s] = make_uint4(keep_word(k, d), keep_word(k + 2, d), keep_word(k + 4, d), keep_word(k + 6, d));
    }

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

    // The tile's rows [r^l_i ; 1 ; 0 ...] over this wavefront's quarter of K
    // as MFMA fragments, in registers for the whole tile: row 16 n + lane%16,
    // K offsets kq0 + 32 s + 8 (lane/16) .. +7 (two pieces of four).
    uint4 rf[kNN][KQ];
#pragma unroll
    for (int n = 0; n < kNN; ++n) {
        const int id = rec[16 * n + (lane & 15)];
        const uint16_t *row = rl + (size_t)(id >= 0 ? id : 0) * d;
        uint2 v[KQ][2];
#pragma unroll
        for (int s = 0; s < KQ; ++s)
#pragma unroll
            for (int h = 0; h < 2; ++h)
                v[s][h] = *reinterpret_cast<const uint2 *>(row + min(kq0 + 32 * s + 8 * (lane >> 4) + 4 * h, d - 4));
#pragma unroll
        for (int s = 0; s < KQ; ++s) {
            uint2 q[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int k = kq0 + 32 * s + 8 * (lane >> 4) + 4 * h;   // a multiple of 4, as d is
                q[h] = id >= 0 && k < d ? v[s][h] : make_uint2(0u, 0u);
                if (k == d) q[h].x = 0x3F80u;                            // the appended 1
            }
            rf[n][s] = make_uint4(q[0].x, q[0].y, q[1].x, q[1].y);
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
        __syncthreads();   // the previous chunk's readers of Ps, Rs, Uh and Ul are done
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const uint2 v = cid >= 0 && c0 + sk + 4 * h < d ? rn[a][h] : make_uint2(0u, 0u);
            *reinterpret_cast<uint2 *>(Rs + sj * kUStride + sk + 4 * h) = v;
        }
        if (c0 + kRAhead * kBiaChunk < d) {   // r^r kRAhead chunks ahead
#pragma unroll
            for (int h = 0; h < 2; ++h)
                rn[a][h] = *reinterpret_cast<const uint2 *>(crow + min(c0 + kRAhead * kBiaChunk + sk + 4 * h, d - 4));
        }

        // U^T[chunk][tile rows], this wavefront's quarter of K
        f32x4 u[kNM][kNN];
#pragma unroll
        for (int m = 0; m < kNM; ++m)
#pragma unroll
            for (int n = 0; n < kNN; ++n) u[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KQ; ++s)
#pragma unroll
            for (int m = 0; m < kNM; ++m) {
                const uint4 wv = wf[m][s];
                const bf16x8 af = frag(make_uint4(wv.x & wmask[s].x, wv.y & wmask[s].y, wv.z & wmask[s].z,
                                                  wv.w & wmask[s].w));
#pragma unroll
                for (int n = 0; n < kNN; ++n)
                    u[m][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, frag(rf[n][s]), u[m][n], 0, 0, 0);
            }
        // the next chunk's W flies while this one's sums meet and its second
        // product runs
        if (c0 + kBiaChunk < d) load_wq<KQ, P>(wf, wl, c0 + kBiaChunk, d, ldw, kq0, lane);
        // partial sums to LDS: row 16 n + lane%16, columns 16 m + 4 (lane/16) .. +3
#pragma unroll
        for (int m = 0; m < kNM; ++m)
#pragma unroll
            for (int n = 0; n < kNN; ++n)
                *reinterpret_cast<f32x4 *>(Ps + (wave * kBiaRows + 16 * n + (lane & 15)) * kPStride + 16 * m +
                                           4 * (lane >> 4)) = u[m][n];
        __syncthreads();
        // the four quarters summed, to bf16 hi + lo: thread t takes row t/4,
        // columns 8 (t%4) .. +7
        {
            const int r = tid >> 2, c = 8 * (tid & 3);
            f32x4 s0 = f32x4{0.f, 0.f, 0.f, 0.f}, s1 = s0;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float *src = Ps + (q * kBiaRows + r) * kPStride + c;
                s0 += *reinterpret_cast<const f32x4 *>(src);
                s1 += *reinterpret_cast<const f32x4 *>(src + 4);
            }
            const bf16x4 h0 = __builtin_convertvector(s0, bf16x4), h1 = __builtin_convertvector(s1, bf16x4);
            const bf16x4 l0 = __builtin_convertvector(s0 - __builtin_convertvector(h0, f32x4), bf16x4);
            const bf16x4 l1 = __builtin_convertvector(s1 - __builtin_convertvector(h1, f32x4), bf16x4);
            *reinterpret_cast<bf16x4 *>(Uh + r * kUStride + c) = h0;
            *reinterpret_cast<bf16x4 *>(Uh + r * kUStride + c + 4) = h1;
            *reinterpret_cast<bf16x4 *>(Ul + r * kUStride + c) = l0;
            *reinterpret_cast<bf16x4 *>(Ul + r * kUStride + c + 4) = l1;
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

int64_t biaffine_lds_bytes(int) {
    return 4 * (4 * kBiaRows * (int64_t)kPStride) + 2 * ((kBiaCols + 2 * kBiaRows) * (int64_t)kUStride) +
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
