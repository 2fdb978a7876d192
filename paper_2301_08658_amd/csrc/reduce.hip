// Partial-sum reduction (the arithmetic of the grouped all-reduce of a
// Partial(SUM) output, Sec. 3.1 / 3.2) with fused bias, GeLU and GeLU'
// epilogues, and the bias-gradient column sum (Sec. 4.2).
//
// The reduction is HBM-bound: per output element it streams nparts fp32
// (or bf16: the 16-bit partials variant, Sec. 5) values in and one
// bf16/fp32 value out.  Each thread owns 8 consecutive columns of one row:
// two 16-byte non-temporal loads per fp32 part (one per bf16 part), all
// parts of a group of 8 issued before the first add so up to 16 loads are
// in flight per thread; parts are then summed in fp32 in group order
// 0..d-1, so the result is bit-identical on every member of the group.
// Rows of a chunk are contiguous, so a launch is one linear sweep of
// [rows x ncols].
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "epilogue_math.h"
#include "kernels.h"

namespace atp {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int RT = 256;        // threads per block
constexpr int PGROUP = 8;      // parts loaded before summing

using epi::bf16_to_f32;
using epi::f32_to_bf16_rne;
using epi::gelu_f;
using epi::gelu_grad_f;

__device__ __forceinline__ void unpack8(const u32x4& w, float* f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[2 * i] = bf16_to_f32(w[i] & 0xffffu);
        f[2 * i + 1] = bf16_to_f32(w[i] >> 16);
    }
}

__device__ __forceinline__ u32x4 pack8(const float* f) {
    u32x4 w;
#pragma unroll
    for (int i = 0; i < 4; ++i)
        w[i] = f32_to_bf16_rne(f[2 * i]) | (f32_to_bf16_rne(f[2 * i + 1]) << 16);
    return w;
}

template <int EPI, bool OUT_BF16, bool PART_BF16>
__global__ __launch_bounds__(RT) void reduce_kernel(ReduceProblem p) {
    const int64_t cols8 = p.ncols >> 3;
    const int64_t total = p.rows * cols8;
    const int64_t g = (int64_t)blockIdx.x * RT + threadIdx.x;
    if (g >= total) return;
    const int64_t r = g / cols8;
    const int64_t c = (g - r * cols8) << 3;
    const int64_t row = p.row0 + r;
    const int64_t off = row * p.ldp + c;

    float s[8];
    for (int j0 = 0; j0 < p.nparts; j0 += PGROUP) {
        f32x4 lo[PGROUP], hi[PGROUP];
        u32x4 hw[PGROUP];   // eight bf16 parts
#pragma unroll
        for (int u = 0; u < PGROUP; ++u) {
            if (j0 + u < p.nparts) {
                if constexpr (PART_BF16) {
                    hw[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(
                        static_cast<const uint16_t*>(p.parts[j0 + u]) + off));
                } else {
                    const f32x4* q = reinterpret_cast<const f32x4*>(
                        static_cast<const float*>(p.parts[j0 + u]) + off);
                    lo[u] = __builtin_nontemporal_load(q);
                    hi[u] = __builtin_nontemporal_load(q + 1);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < PGROUP; ++u) {
            if (j0 + u < p.nparts) {
                if constexpr (PART_BF16) {
                    float f[8];
                    unpack8(hw[u], f);
#pragma unroll
                    for (int e = 0; e < 4; ++e) { lo[u][e] = f[e]; hi[u][e] = f[4 + e]; }
                }
                if (j0 + u == 0) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) { s[e] = lo[u][e]; s[4 + e] = hi[u][e]; }
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) { s[e] += lo[u][e]; s[4 + e] += hi[u][e]; }
                }
            }
        }
    }

    const int64_t oo = row * p.ldo + c;
    if constexpr (EPI == EPI_BIAS || EPI == EPI_BIAS_GELU) {
        float b[8];
        unpack8(*reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(p.bias) + c), b);
#pragma unroll
        for (int e = 0; e < 8; ++e) s[e] += b[e];
    }
    if constexpr (EPI == EPI_BIAS_GELU) {
        if (p.pre_out) {
            const u32x4 w = pack8(s);
            __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(
                                               static_cast<uint16_t*>(p.pre_out) + oo));
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) s[e] = gelu_f(s[e]);
    }
    if constexpr (EPI == EPI_GELU_BWD) {
        float x[8];
        unpack8(*reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(p.pre_in) + oo), x);
#pragma unroll
        for (int e = 0; e < 8; ++e) s[e] *= gelu_grad_f(x[e]);
    }
    if constexpr (OUT_BF16) {
        __builtin_nontemporal_store(pack8(s),
                                    reinterpret_cast<u32x4*>(static_cast<uint16_t*>(p.out) + oo));
    } else {
        f32x4* q = reinterpret_cast<f32x4*>(static_cast<float*>(p.out) + oo);
        __builtin_nontemporal_store(f32x4{s[0], s[1], s[2], s[3]}, q);
        __builtin_nontemporal_store(f32x4{s[4], s[5], s[6], s[7]}, q + 1);
    }
}

template <int EPI, bool OUT_BF16, bool PART_BF16>
hipError_t launch_r(const ReduceProblem& p, hipStream_t s) {
    const int64_t total = p.rows * (p.ncols >> 3);
    if (total == 0) return hipSuccess;
    const int64_t blocks = (total + RT - 1) / RT;
    hipLaunchKernelGGL((reduce_kernel<EPI, OUT_BF16, PART_BF16>), dim3((unsigned)blocks), dim3(RT),
                       0, s, p);
    return hipGetLastError();
}

// Column sums in one fixed order, the same on every path (so db has the
// same bits whether or not it is formed during dY's transpose):
//   db[c] = (((0 + S_0) + S_1) + ...),  S_b over the 64-row block b,
//   S_b = (((0 + G_b0) + G_b1) + ...)   over its 8-row groups inside [0, T),
//   G_bg = (((0 + x_r) + x_r+1) + ...)  over the group's rows inside [0, T).
// A block owns 64 columns: 8 column lanes (8 columns, one 16-byte load per
// row) x 128 row lanes; row lane ty forms S_b for b = ty, ty + 128, ... one
// round of 128 blocks at a time, and 64 threads fold each round's S_b into
// their column's sum in ascending b.  Blocks are renumbered so neighbouring
// column groups run on the same XCD.
constexpr int CS_CL = 8;                 // column lanes
constexpr int CS_COLS = CS_CL * 8;       // columns per block
constexpr int CS_ROWL = 128;             // row lanes (row blocks per round)
constexpr int CS_T = CS_CL * CS_ROWL;    // threads per block

__global__ __launch_bounds__(CS_T) void colsum_kernel(const uint16_t* __restrict__ dy, int64_t ld,
                                                      int64_t T, int64_t N, float* __restrict__ db) {
    __shared__ float part[CS_ROWL][CS_COLS + 1];
    const int tx = threadIdx.x % CS_CL;
    const int ty = threadIdx.x / CS_CL;
    const int G = gridDim.x, xcd = blockIdx.x % 8, idx = blockIdx.x / 8;
    const int per = G / 8, rem = G % 8;
    const int64_t blk = (xcd < rem) ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
    const int64_t c = blk * CS_COLS + tx * 8;
    const int64_t nb = (T + 63) / 64;
    float acc = 0.0f;                      // column blk * 64 + threadIdx.x (first 64 threads)
    for (int64_t b0 = 0; b0 < nb; b0 += CS_ROWL) {
        const int64_t b = b0 + ty;
        float sb[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) sb[e] = 0.0f;
        if (c < N && b < nb) {
            for (int g = 0; g < 8; ++g) {
                const int64_t r0 = b * 64 + g * 8;
                if (r0 >= T) break;
                float gs[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) gs[e] = 0.0f;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    if (r0 + i < T) {
                        float f[8];
                        unpack8(*reinterpret_cast<const u32x4*>(dy + (r0 + i) * ld + c), f);
#pragma unroll
                        for (int e = 0; e < 8; ++e) gs[e] += f[e];
                    }
                }
#pragma unroll
                for (int e = 0; e < 8; ++e) sb[e] += gs[e];
            }
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) part[ty][tx * 8 + e] = sb[e];
        __syncthreads();
        if (threadIdx.x < CS_COLS) {
            const int64_t nr = nb - b0 < CS_ROWL ? nb - b0 : CS_ROWL;
            for (int r = 0; r < nr; ++r) acc += part[r][threadIdx.x];
        }
        __syncthreads();
    }
    if (threadIdx.x < CS_COLS) {
        const int64_t col = blk * CS_COLS + threadIdx.x;
        if (col < N) db[col] = acc;
    }
}

// db[c] = (((0 + part_0[c]) + part_1[c]) + ...) over nb row-block partials.
// The loads of 32 partials are issued before their sums, so a thread waits
// for memory once per 32 blocks instead of once per block; the additions
// keep the block order.
__global__ __launch_bounds__(256) void colsum_finish_kernel(const float* __restrict__ part,
                                                            int64_t ldp, int64_t nb, int64_t N,
                                                            float* __restrict__ db) {
    constexpr int U = 32;
    const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (c >= N) return;
    float acc = 0.0f;
    int64_t b = 0;
    for (; b + U <= nb; b += U) {
        float v[U];
#pragma unroll
        for (int i = 0; i < U; ++i) v[i] = part[(b + i) * ldp + c];
#pragma unroll
        for (int i = 0; i < U; ++i) acc += v[i];
    }
    for (; b < nb; ++b) acc += part[b * ldp + c];
    db[c] = acc;
}

template <bool PART_BF16>
hipError_t launch_reduce_parts(const ReduceProblem& p, hipStream_t s) {
    const bool b = p.out_bf16;
    switch (p.epi) {
    case EPI_NONE:
        return b ? launch_r<EPI_NONE, true, PART_BF16>(p, s)
                 : launch_r<EPI_NONE, false, PART_BF16>(p, s);
    case EPI_BIAS:
        return b ? launch_r<EPI_BIAS, true, PART_BF16>(p, s)
                 : launch_r<EPI_BIAS, false, PART_BF16>(p, s);
    case EPI_BIAS_GELU:
        return b ? launch_r<EPI_BIAS_GELU, true, PART_BF16>(p, s)
                 : launch_r<EPI_BIAS_GELU, false, PART_BF16>(p, s);
    case EPI_GELU_BWD:
        return b ? launch_r<EPI_GELU_BWD, true, PART_BF16>(p, s)
                 : launch_r<EPI_GELU_BWD, false, PART_BF16>(p, s);
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_reduce(const ReduceProblem& p, hipStream_t s) {
    return p.parts_bf16 ? launch_reduce_parts<true>(p, s) : launch_reduce_parts<false>(p, s);
}

hipError_t launch_split_sum(const float* ws, int S, int64_t stride, int64_t ld, int64_t rows,
                            int64_t cols, void* out, int64_t ldo, bool out_bf16, hipStream_t s) {
    if (S < 1 || S > kMaxParts || (cols & 7) || (ld & 3) || (ldo & (out_bf16 ? 7 : 3)))
        return hipErrorInvalidValue;
    ReduceProblem p{};
    p.nparts = S;
    for (int i = 0; i < S; ++i) p.parts[i] = ws + i * stride;
    p.ldp = ld;
    p.row0 = 0;
    p.rows = rows;
    p.ncols = cols;
    p.epi = EPI_NONE;
    p.out = out;
    p.ldo = ldo;
    p.out_bf16 = out_bf16;
    return launch_reduce(p, s);
}

hipError_t launch_colsum_finish(const float* part, int64_t ldp, int64_t nb, int64_t N, float* db,
                                hipStream_t s) {
    if (N <= 0) return hipSuccess;
    hipLaunchKernelGGL(colsum_finish_kernel, dim3((unsigned)((N + 255) / 256)), dim3(256), 0, s,
                       part, ldp, nb, N, db);
    return hipGetLastError();
}

hipError_t launch_colsum(const void* dy, int64_t ld, int64_t T, int64_t N, float* db,
                         hipStream_t s) {
    if (N <= 0) return hipSuccess;
    const int64_t blocks = (N + CS_COLS - 1) / CS_COLS;
    hipLaunchKernelGGL(colsum_kernel, dim3((unsigned)blocks), dim3(CS_T), 0, s,
                       static_cast<const uint16_t*>(dy), ld, T, N, db);
    return hipGetLastError();
}

}  // namespace atp
