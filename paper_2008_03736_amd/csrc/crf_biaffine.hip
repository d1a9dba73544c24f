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
// kBiaRows rows (left fence posts) and
// kBiaCols columns (right fence posts) -- short sentences packed whole into
// one tile (their scores are the tile's diagonal blocks), longer ones cut
// into row and column blocks -- and one label.  For each chunk of kBiaChunk
// of the d output dimensions of W it computes U = [R^l ; 1] W[:, chunk]
// (MFMA over K = d+1; each wavefront keeps its rows, with the 1 and the zero
// padding of K, as A fragments in registers for the whole tile, and W's
// chunk is staged in LDS while the next one is loaded into registers), keeps
// U on chip as bf16 hi + lo parts (a 16-bit mantissa in all), and
// accumulates S += U R^r[:, chunk]^T (MFMA, two products for hi and lo).  U
// never leaves the CU; W is read once per tile from L2.  Only the valid
// cells 0 <= i < j <= n_b of S are written.
//
// MFMA v_mfma_f32_16x16x32_bf16 (gfx950): A 16 x 32, B 32 x 16, D 16 x 16;
// lane l supplies A row l%16 and B column l%16 at K offsets 8(l/16)..+7, and
// holds D rows 4(l/16)..+3 of column l%16.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "crf_internal.h"

namespace crf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kPad = 8;                       // bf16 of padding per staged row (keeps 16-byte reads conflict-free)
constexpr int kUStride = kBiaChunk + kPad;    // row stride of the staged U and R^r chunks

__device__ __forceinline__ uint16_t bf16_bits(float x) {   // round to nearest even (finite x)
    const uint32_t u = __builtin_bit_cast(uint32_t, x);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}
__device__ __forceinline__ float bf16_float(uint16_t h) { return __builtin_bit_cast(float, (uint32_t)h << 16); }

// Eight consecutive bf16 of a staged row as an MFMA operand.
__device__ __forceinline__ bf16x8 frag(const uint16_t *p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(p));
}

// Four bf16 of a representation row, k .. k+3 (d is a multiple of 4, so all
// four are in the row or none is).
__device__ __forceinline__ uint2 rep4(const uint16_t *row, int k, int d) {
    return k < d ? *reinterpret_cast<const uint2 *>(row + k) : make_uint2(0u, 0u);
}

// K of the first product: d + 1 padded to 128, 256 or 512.
__host__ __device__ inline int bia_kp(int d) { return d + 1 <= 128 ? 128 : d + 1 <= 256 ? 256 : 512; }

// One chunk of W[:, c0 .. c0 + kBiaChunk)^T as this thread's share of the
// staged rows (wave w: rows 16 w .. 16 w + 15; lane: pieces lane, lane + 64):
// row c holds W[k][c0 + c] for k <= d (k = d: the bias), zeros after.  Loaded
// into registers, stored to LDS separately, so that the next chunk's loads
// fly while the current one is multiplied.
template <int KS>
struct WChunk {
    static constexpr int H = (8 * KS + 63) / 64;   // pieces of 4 per lane and row
    uint2 v[16][H];
};
template <int KS>
__device__ __forceinline__ void load_w(WChunk<KS> &r, const uint16_t *wl, int c0, int d, int ldw, int wave, int lane) {
#pragma unroll
    for (int rr_ = 0; rr_ < 16; ++rr_)
#pragma unroll
        for (int h = 0; h < WChunk<KS>::H; ++h) {
            const int c = 16 * wave + rr_, k = 4 * (lane + 64 * h);
            uint2 v = make_uint2(0u, 0u);
            if (k < 32 * KS && c0 + c < d && k <= d) {
                // ldw >= d+1, and ldw and d are multiples of 4: k .. k+3 lie in
                // the row; at k = d only the bias entry is kept
                v = *reinterpret_cast<const uint2 *>(wl + (size_t)(c0 + c) * ldw + k);
                if (k == d) {
                    v.x &= 0x0000FFFFu;
                    v.y = 0u;
                }
            }
            r.v[rr_][h] = v;
        }
}
template <int KS>
__device__ __forceinline__ void store_w(const WChunk<KS> &r, uint16_t *Ws, int lda, int wave, int lane) {
#pragma unroll
    for (int rr_ = 0; rr_ < 16; ++rr_)
#pragma unroll
        for (int h = 0; h < WChunk<KS>::H; ++h) {
            const int k = 4 * (lane + 64 * h);
            if (k < 32 * KS) *reinterpret_cast<uint2 *>(Ws + (16 * wave + rr_) * lda + k) = r.v[rr_][h];
        }
}

// Tile record: kBiaRows row ids then kBiaCols column ids, each b * N1 + i
// (sentence b, fence post i) or -1.  KS = K / 32 steps of the first product
// (K = d + 1 padded to 128, 256 or 512): all of a chunk's fragments are read
// before its products, so one LDS latency is paid per chunk, not per MFMA.
// (One workgroup per CU is all the LDS allows, one wavefront per SIMD: the
// whole register file is this wavefront's.)
template <int KS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void biaffine_kernel(
    const int32_t *__restrict__ tiles,
                                                       const int32_t *__restrict__ len, int N1, int d, int ldw,
                                                       int L, const uint16_t *__restrict__ rl,
                                                       const uint16_t *__restrict__ rr,
                                                       const uint16_t *__restrict__ w,
                                                       float *__restrict__ scores) {
    extern __shared__ __align__(16) char smem_raw[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    constexpr int Kp = 32 * KS;              // K of the first product
    const int lda = Kp + kPad;
    uint16_t *Ws = reinterpret_cast<uint16_t *>(smem_raw);   // [kBiaChunk][lda]: W[:, chunk]^T
    uint16_t *Rs = Ws + kBiaChunk * lda;                     // [kBiaCols][kUStride]: r^r[:, chunk]
    uint16_t *Uh = Rs + kBiaCols * kUStride;                 // [kBiaRows][kUStride]: U hi
    uint16_t *Ul = Uh + kBiaRows * kUStride;                 // [kBiaRows][kUStride]: U lo
    const int32_t *rec = tiles + (size_t)blockIdx.x * (kBiaRows + kBiaCols);
    const int l = blockIdx.y;
    const uint16_t *wl = w + (size_t)l * d * ldw;

    // This wave's rows [r^l_i ; 1 ; 0 ...] as MFMA A fragments, in registers
    // for the whole tile: row 16 wave + lane%16, K offsets k0 + 8 (lane/16).
    uint2 afr[KS][2];
    {
        const int id = rec[16 * wave + (lane & 15)];
        const uint16_t *row = rl + (size_t)(id >= 0 ? id : 0) * d;
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int k = 32 * s + 8 * (lane >> 4) + 4 * h;
                uint2 v = make_uint2(0u, 0u);
                if (id >= 0) v = rep4(row, k, d);
                if (k == d) v.x = 0x3F80u;                   // the appended 1 (k = d, a multiple of 4)
                afr[s][h] = v;
            }
    }

    f32x4 acc[kBiaCols / 16];   // S rows 16 wave + 4 (lane/16) + t, columns 16 c + lane%16
#pragma unroll
    for (int c = 0; c < kBiaCols / 16; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};

    WChunk<KS> wn;
    load_w<KS>(wn, wl, 0, d, ldw, wave, lane);
    for (int c0 = 0; c0 < d; c0 += kBiaChunk) {
        __syncthreads();   // the previous chunk's readers are done
        store_w<KS>(wn, Ws, lda, wave, lane);
        // r^r[:, c0 .. c0+chunk) of the tile's columns: wave w stages columns
        // 16 w .. +15, four per pass of 16 lanes
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int j = 16 * wave + 4 * q + (lane >> 4), k = 4 * (lane & 15);
            const int id = rec[kBiaRows + j];
            uint2 v = make_uint2(0u, 0u);
            if (id >= 0) v = rep4(rr + (size_t)id * d, c0 + k, d);
            *reinterpret_cast<uint2 *>(Rs + j * kUStride + k) = v;
        }
        if (c0 + kBiaChunk < d) load_w<KS>(wn, wl, c0 + kBiaChunk, d, ldw, wave, lane);   // in flight meanwhile
        __syncthreads();

        // U[16 wave .. +16][chunk] = [r^l ; 1] W[:, chunk]
        f32x4 u[kBiaChunk / 16];
#pragma unroll
        for (int c = 0; c < kBiaChunk / 16; ++c) u[c] = f32x4{0.f, 0.f, 0.f, 0.f};
        const uint16_t *wrow = Ws + (lane & 15) * lda + 8 * (lane >> 4);
        bf16x8 bw[KS][kBiaChunk / 16];
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
            for (int c = 0; c < kBiaChunk / 16; ++c) bw[s][c] = frag(wrow + 16 * c * lda + 32 * s);
        __builtin_amdgcn_sched_barrier(0);   // every fragment read in flight before the first product
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            const bf16x8 a = __builtin_bit_cast(bf16x8, make_uint4(afr[s][0].x, afr[s][0].y, afr[s][1].x, afr[s][1].y));
#pragma unroll
            for (int c = 0; c < kBiaChunk / 16; ++c)
                u[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bw[s][c], u[c], 0, 0, 0);
        }
        // U to LDS as bf16 hi + lo (row 16 wave + 4 (lane/16) + t, column 16 c + lane%16)
#pragma unroll
        for (int c = 0; c < kBiaChunk / 16; ++c)
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int r = 16 * wave + 4 * (lane >> 4) + t, col = 16 * c + (lane & 15);
                const uint16_t hi = bf16_bits(u[c][t]);
                Uh[r * kUStride + col] = hi;
                Ul[r * kUStride + col] = bf16_bits(u[c][t] - bf16_float(hi));
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
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int k = 0; k < kBiaChunk / 32; ++k)
#pragma unroll
            for (int c = 0; c < kBiaCols / 16; ++c) {
                acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[k], br[k][c], acc[c], 0, 0, 0);
                acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[k], br[k][c], acc[c], 0, 0, 0);
            }
    }

    // The valid cells: row and column of one sentence, i < j <= n_b.
#pragma unroll
    for (int c = 0; c < kBiaCols / 16; ++c)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int ri = rec[16 * wave + 4 * (lane >> 4) + t], cj = rec[kBiaRows + 16 * c + (lane & 15)];
            if (ri < 0 || cj < 0) continue;
            const int b = ri / N1, i = ri - b * N1, b2 = cj / N1, j = cj - b2 * N1;
            if (b == b2 && i < j && j <= len[b]) scores[((size_t)ri * N1 + j) * L + l] = acc[c][t];
        }
}

}  // namespace

hipError_t set_biaffine_attributes() {
    const void *fns[] = {(const void *)biaffine_kernel<4>, (const void *)biaffine_kernel<8>,
                         (const void *)biaffine_kernel<16>};
    const int lds[] = {(int)biaffine_lds_bytes(127), (int)biaffine_lds_bytes(255), (int)biaffine_lds_bytes(kBiaMaxD)};
    for (int k = 0; k < 3; ++k) {
        const hipError_t e = hipFuncSetAttribute(fns[k], hipFuncAttributeMaxDynamicSharedMemorySize, lds[k]);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

int64_t biaffine_lds_bytes(int d) {
    const int64_t lda = bia_kp(d) + kPad;
    return 2 * (kBiaChunk * lda + (kBiaCols + 2 * kBiaRows) * (int64_t)kUStride);
}

hipError_t launch_biaffine(const KernelPlan &p, const uint16_t *rl, const uint16_t *rr, const uint16_t *w, int d,
                           int ldw, int L, float *scores, hipStream_t stream) {
    if (p.n_bia_tiles < 1) return hipSuccess;
    const size_t lds = (size_t)biaffine_lds_bytes(d);
    const dim3 grid(p.n_bia_tiles, L), block(256);
    const int kp = bia_kp(d);
    if (kp == 128)
        hipLaunchKernelGGL(biaffine_kernel<4>, grid, block, lds, stream, p.bia_tiles, p.len, p.n1, d, ldw, L, rl, rr, w, scores);
    else if (kp == 256)
        hipLaunchKernelGGL(biaffine_kernel<8>, grid, block, lds, stream, p.bia_tiles, p.len, p.n1, d, ldw, L, rl, rr, w, scores);
    else
        hipLaunchKernelGGL(biaffine_kernel<16>, grid, block, lds, stream, p.bia_tiles, p.len, p.n1, d, ldw, L, rl, rr, w, scores);
    return hipGetLastError();
}

}  // namespace crf
