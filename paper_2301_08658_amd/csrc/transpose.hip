// bf16 matrix transpose through LDS (HBM-bound).
//
// Turns an operand that is contiguous along its M/N side into one contiguous
// along the contraction, so that every product of a shard linear (Sec. 3.2
// forward, Sec. 4.2 backward) can run in the GEMM's NT layout: W -> W^T for
// the forward, X -> X^T and dY -> dY^T for dW = X^T dY.
//
// One workgroup moves a 64 x 64 tile: 16-byte loads along the source rows,
// a transposed write into LDS, 16-byte stores along the destination rows.
// Partial tiles at the edges go element by element.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace atp {
namespace {

constexpr int TILE = 64;
constexpr int PAD = 8;                 // LDS row pitch 72 elements (144 B)
constexpr int THREADS = 256;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(THREADS) void transpose_kernel(const uint16_t* __restrict__ src,
                                                            int64_t lds, int64_t rows,
                                                            int64_t cols, uint16_t* __restrict__ dst,
                                                            int64_t ldd, int tiles_c) {
    __shared__ __attribute__((aligned(16))) uint16_t tile[TILE][TILE + PAD];
    const int tid = threadIdx.x;
    const int64_t r0 = (int64_t)(blockIdx.x / tiles_c) * TILE;
    const int64_t c0 = (int64_t)(blockIdx.x % tiles_c) * TILE;
    // load: 64 rows x 8 chunks of 8 elements; tile[c][r] = src[r0 + r][c0 + c]
#pragma unroll
    for (int j = 0; j < TILE * TILE / 8 / THREADS; ++j) {
        const int q = tid + j * THREADS;
        const int r = q >> 3, c = (q & 7) * 8;
        const int64_t gr = r0 + r, gc = c0 + c;
        uint16_t v[8];
        if (gr < rows && gc + 8 <= cols) {
            const u32x4 w = *reinterpret_cast<const u32x4*>(src + gr * lds + gc);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[2 * e] = (uint16_t)(w[e] & 0xffffu);
                v[2 * e + 1] = (uint16_t)(w[e] >> 16);
            }
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
                v[e] = (gr < rows && gc + e < cols) ? src[gr * lds + gc + e] : (uint16_t)0;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) tile[c + e][r] = v[e];
    }
    __syncthreads();
    // store: dst[c0 + c][r0 + r .. +8] = tile[c][r .. r+8]
#pragma unroll
    for (int j = 0; j < TILE * TILE / 8 / THREADS; ++j) {
        const int q = tid + j * THREADS;
        const int c = q >> 3, r = (q & 7) * 8;
        const int64_t gc = c0 + c, gr = r0 + r;
        if (gc >= cols) continue;
        if (gr + 8 <= rows) {
            *reinterpret_cast<u32x4*>(dst + gc * ldd + gr) =
                *reinterpret_cast<const u32x4*>(&tile[c][r]);
        } else {
            for (int e = 0; e < 8 && gr + e < rows; ++e) dst[gc * ldd + gr + e] = tile[c][r + e];
        }
    }
}

// Shapes whose rows and columns are multiples of 8 (every operand the block
// transposes): no LDS.  A lane moves one 8 x 8 block: eight 16-byte loads
// (source rows r..r+7, columns c..c+7), a register transpose (one byte
// permute per output word), eight 16-byte stores (destination rows c..c+7).
// A wave holds 8 row blocks x 8 column blocks (lane = 8 cb + rb), so every
// load and every store instruction covers 8 rows x 128 contiguous bytes.
// A workgroup of four waves spans 64 source rows x 256 source columns.
//
// With part, the lanes also form the column sums of the 64-row block in the
// column-sum order (8-row group of each lane, then the groups in ascending
// row order through LDS) and write them to part[(r0 / 64) * ldpart + c].
__global__ __launch_bounds__(THREADS) void transpose8_kernel(const uint16_t* __restrict__ src,
                                                             int64_t lds, int64_t rows,
                                                             int64_t cols,
                                                             uint16_t* __restrict__ dst,
                                                             int64_t ldd, int tiles_c,
                                                             float* __restrict__ part,
                                                             int64_t ldpart) {
    __shared__ float gsum[4][8][64 + 1];   // [wave][row group][column of the wave]
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int rb = lane & 7, cb = lane >> 3;
    const int64_t r0 = (int64_t)(blockIdx.x / tiles_c) * 64;
    const int64_t c0 = (int64_t)(blockIdx.x % tiles_c) * 256 + wave * 64;
    const int64_t r = r0 + 8 * rb, c = c0 + 8 * cb;
    const bool live = r < rows && c < cols;
    if (part) {
        float gs[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) gs[e] = 0.0f;
        if (live) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const u32x4 w = *reinterpret_cast<const u32x4*>(src + (r + i) * lds + c);
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    gs[2 * k] += __uint_as_float(w[k] << 16);
                    gs[2 * k + 1] += __uint_as_float(w[k] & 0xffff0000u);
                }
            }
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) gsum[wave][rb][8 * cb + e] = gs[e];
        __syncthreads();
        if (rb == 0 && c < cols) {
            const int ng = (int)((rows - r0 + 7) / 8 < 8 ? (rows - r0 + 7) / 8 : 8);
            float sb[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) sb[e] = 0.0f;
            for (int g = 0; g < ng; ++g)
#pragma unroll
                for (int e = 0; e < 8; ++e) sb[e] += gsum[wave][g][8 * cb + e];
            float* pp = part + (r0 / 64) * ldpart + c;
            *reinterpret_cast<f32x4*>(pp) = f32x4{sb[0], sb[1], sb[2], sb[3]};
            *reinterpret_cast<f32x4*>(pp + 4) = f32x4{sb[4], sb[5], sb[6], sb[7]};
        }
    }
    if (!live || !dst) return;
    u32x4 in[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) in[i] = *reinterpret_cast<const u32x4*>(src + (r + i) * lds + c);
    // out row j (source column c + j), word k = (in[2k] element j, in[2k+1] element j):
    // element j of a row sits in word j / 2, low half for even j
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
        u32x4 o;
#pragma unroll
        for (int k = 0; k < 4; ++k)
            o[k] = __builtin_amdgcn_perm(in[2 * k + 1][j >> 1], in[2 * k][j >> 1], sel);
        *reinterpret_cast<u32x4*>(dst + (c + j) * ldd + r) = o;
    }
}

}  // namespace

hipError_t launch_transpose(const void* src, int64_t lds, int64_t rows, int64_t cols, void* dst,
                            int64_t ldd, hipStream_t s, float* part, int64_t ldpart) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    const bool by8 = rows % 8 == 0 && cols % 8 == 0 && lds % 8 == 0 && ldd % 8 == 0;
    if (part && (!by8 || ldpart < cols || ldpart % 4)) return hipErrorInvalidValue;
    if (by8) {
        const int64_t tr = (rows + 63) / 64, tc = (cols + 255) / 256;
        if (tr * tc > 0x7fffffff) return hipErrorInvalidValue;
        hipLaunchKernelGGL(transpose8_kernel, dim3((unsigned)(tr * tc)), dim3(THREADS), 0, s,
                           static_cast<const uint16_t*>(src), lds, rows, cols,
                           static_cast<uint16_t*>(dst), ldd, (int)tc, part, ldpart);
        return hipGetLastError();
    }
    const int64_t tr = (rows + TILE - 1) / TILE, tc = (cols + TILE - 1) / TILE;
    if (tr * tc > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL(transpose_kernel, dim3((unsigned)(tr * tc)), dim3(THREADS), 0, s,
                       static_cast<const uint16_t*>(src), lds, rows, cols,
                       static_cast<uint16_t*>(dst), ldd, (int)tc);
    return hipGetLastError();
}

}  // namespace atp
