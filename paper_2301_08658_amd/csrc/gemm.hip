// bf16 x bf16 -> fp32 MFMA GEMM for gfx950 (CDNA4) with fused epilogues.
//
// One kernel template serves the three products of a shard linear
// (Sec. 3.2 forward Y = X W; Sec. 4.2 backward dX = dY W^T, dW = X^T dY):
//
//   * Workgroup tile 256 x 256, K step 64, 256 threads = 4 wave64s in a
//     2 x 2 arrangement; each wave owns a 128 x 128 sub-tile held as 4 x 4
//     v_mfma_f32_32x32x16_bf16 accumulators (256 fp32 per lane).
//   * Both operands live in LDS as [row][k] with k contiguous, so every
//     MFMA fragment is one 16-byte LDS read.  Rows are padded to 72
//     elements (144 B): consecutive rows then start 16 B apart modulo the
//     bank width and a wave's fragment reads are conflict free.
//   * An operand that is contiguous along k in memory (X, dY, W for dX) is
//     copied in 16-byte chunks.  An operand contiguous along its M/N side
//     (W in the forward, X and dY in dW) is fetched as 8 x 8 element blocks
//     (eight coalesced 16-byte row loads) and transposed in registers
//     before the 16-byte LDS stores.
//   * Two LDS stages: global loads of step k+1 are in flight while step k
//     is multiplied; one barrier per K step.
//   * The MFMA is issued with the N-side fragment as its first operand, so
//     each lane's 16 results are 4 runs of 4 consecutive output columns:
//     the epilogue writes 16 B (fp32) or 8 B (bf16) per lane.
//   * Every output element accumulates its K products in the same order
//     (64-wide steps, MFMA k order inside) whatever M, so token chunking
//     never changes a value.
//   * Workgroups are renumbered so that consecutive tiles land on the same
//     XCD (the dispatcher deals workgroups round-robin over the 8 XCDs),
//     and tiles are visited in groups of 8 M-tiles so the tiles that
//     share a weight panel run together and hit that XCD's L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace atp {
namespace {

constexpr int BM = 256;
constexpr int BN = 256;
constexpr int BK = 64;
constexpr int LDK = BK + 8;       // padded LDS row length (elements)
constexpr int NT = 256;           // threads per workgroup
constexpr int WM = 128;           // wave sub-tile
constexpr int WN = 128;
constexpr int FM = WM / 32;       // MFMA blocks per wave along M
constexpr int FN = WN / 32;       // ... along N
constexpr int GROUP_M = 8;
constexpr int NUM_XCD = 8;
constexpr int STAGE_ELEMS = (BM + BN) * LDK;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return 0x7fc0u;  // NaN
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ float gelu_f(float x) {
    return 0.5f * x * (1.0f + erff(x * 0.70710678118654752440f));
}

__device__ __forceinline__ float gelu_grad_f(float x) {
    const float cdf = 0.5f * (1.0f + erff(x * 0.70710678118654752440f));
    const float pdf = 0.39894228040143267794f * expf(-0.5f * x * x);
    return cdf + x * pdf;
}

// ---------------------------------------------------------------------------
// Global -> register -> LDS copy of one operand tile (rows = M or N side).
// ---------------------------------------------------------------------------
template <bool KCONTIG>
struct TileCopy;

// Operand stored as [row][k] with k contiguous: 256 rows x 8 chunks of 16 B.
template <>
struct TileCopy<true> {
    u32x4 r[8];
    __device__ __forceinline__ void load(const uint16_t* __restrict__ base, int64_t ld,
                                         int64_t row0, int64_t rows, int64_t k0, int64_t K,
                                         int tid) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int id = tid + NT * i;
            const int row = id >> 3;
            const int cc = id & 7;
            const int64_t gr = row0 + row;
            const int64_t gk = k0 + cc * 8;
            const bool ok = (gr < rows) && (gk < K);
            const uint16_t* p = base + (ok ? gr * ld + gk : 0);
            const u32x4 v = *reinterpret_cast<const u32x4*>(p);
            r[i] = ok ? v : u32x4{0u, 0u, 0u, 0u};
        }
    }
    __device__ __forceinline__ void store(uint16_t* __restrict__ lds, int tid) const {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int id = tid + NT * i;
            const int row = id >> 3;
            const int cc = id & 7;
            *reinterpret_cast<u32x4*>(lds + row * LDK + cc * 8) = r[i];
        }
    }
};

// Operand stored as [k][row] with the row index contiguous: each thread
// fetches an 8 (k) x 8 (row) block and transposes it.
template <>
struct TileCopy<false> {
    u32x4 r[8];
    __device__ __forceinline__ void load(const uint16_t* __restrict__ base, int64_t ld,
                                         int64_t row0, int64_t rows, int64_t k0, int64_t K,
                                         int tid) {
        const int kb = tid >> 5;     // 0..7  : k block of 8
        const int rb = tid & 31;     // 0..31 : row block of 8
        const int64_t gr = row0 + rb * 8;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int64_t gk = k0 + kb * 8 + i;
            const bool ok = (gr < rows) && (gk < K);
            const uint16_t* p = base + (ok ? gk * ld + gr : 0);
            const u32x4 v = *reinterpret_cast<const u32x4*>(p);
            r[i] = ok ? v : u32x4{0u, 0u, 0u, 0u};
        }
    }
    __device__ __forceinline__ void store(uint16_t* __restrict__ lds, int tid) const {
        const int kb = tid >> 5;
        const int rb = tid & 31;
        // r[e] holds k = kb*8+e, rows rb*8+0..7 (two per dword).  Output row
        // j holds k = kb*8+0..7: dword p = (k 2p low half, k 2p+1 high half).
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int q = j >> 1;
            u32x4 o;
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                const uint32_t lo = r[2 * p][q];
                const uint32_t hi = r[2 * p + 1][q];
                o[p] = (j & 1) ? ((lo >> 16) | (hi & 0xffff0000u))
                               : ((lo & 0xffffu) | (hi << 16));
            }
            *reinterpret_cast<u32x4*>(lds + (rb * 8 + j) * LDK + kb * 8) = o;
        }
    }
};

struct KArgs {
    const uint16_t* A; int64_t lda;
    const uint16_t* B; int64_t ldb;
    void* C; int64_t ldc;
    const uint16_t* bias;
    const uint16_t* pre_in;
    uint16_t* pre_out;
    int64_t M, N, K;
    int tiles_m, tiles_n;
};

__device__ __forceinline__ void tile_coords(const KArgs& a, int& tm, int& tn) {
    const int G = gridDim.x;
    const int pid = blockIdx.x;
    // renumber: workgroups dealt to XCD x become one contiguous range
    const int xcd = pid % NUM_XCD;
    const int idx = pid / NUM_XCD;
    const int per = G / NUM_XCD;
    const int rem = G % NUM_XCD;
    const int logical = (xcd < rem) ? xcd * (per + 1) + idx
                                    : rem * (per + 1) + (xcd - rem) * per + idx;
    // grouped order: GROUP_M row tiles per column sweep
    const int in_group = GROUP_M * a.tiles_n;
    const int group = logical / in_group;
    const int first_m = group * GROUP_M;
    const int gsize = min(a.tiles_m - first_m, GROUP_M);
    const int r = logical % in_group;
    tm = first_m + r % gsize;
    tn = r / gsize;
}

template <bool A_K, bool B_K, int EPI, bool OUT_BF16>
__global__ __launch_bounds__(NT, 1) void gemm_kernel(KArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t smem[2 * STAGE_ELEMS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1;
    const int wn = wave & 1;

    int tm, tn;
    tile_coords(a, tm, tn);
    const int64_t m0 = (int64_t)tm * BM;
    const int64_t n0 = (int64_t)tn * BN;

    TileCopy<A_K> ca;
    TileCopy<B_K> cb;

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    const int nk = (int)((a.K + BK - 1) / BK);

    if (nk > 0) {   // K == 0 (no tokens in a dW product) reads nothing and writes zeros
        ca.load(a.A, a.lda, m0, a.M, 0, a.K, tid);
        cb.load(a.B, a.ldb, n0, a.N, 0, a.K, tid);
        ca.store(smem, tid);
        cb.store(smem + BM * LDK, tid);
    }
    __syncthreads();

    const int frag_row = lane & 31;
    const int frag_k = (lane >> 5) * 8;

    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        const bool more = (kt + 1) < nk;
        if (more) {
            const int64_t k0 = (int64_t)(kt + 1) * BK;
            ca.load(a.A, a.lda, m0, a.M, k0, a.K, tid);
            cb.load(a.B, a.ldb, n0, a.N, k0, a.K, tid);
        }
        const uint16_t* sa = smem + cur * STAGE_ELEMS;
        const uint16_t* sb = sa + BM * LDK;
#pragma unroll
        for (int s = 0; s < BK / 16; ++s) {
            bf16x8 fa[FM], fb[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i)
                fa[i] = *reinterpret_cast<const bf16x8*>(
                    sa + (wm * WM + i * 32 + frag_row) * LDK + s * 16 + frag_k);
#pragma unroll
            for (int j = 0; j < FN; ++j)
                fb[j] = *reinterpret_cast<const bf16x8*>(
                    sb + (wn * WN + j * 32 + frag_row) * LDK + s * 16 + frag_k);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[j], fa[i], acc[i][j],
                                                                        0, 0, 0);
        }
        if (more) {
            uint16_t* nxt = smem + (cur ^ 1) * STAGE_ELEMS;
            ca.store(nxt, tid);
            cb.store(nxt + BM * LDK, tid);
        }
        __syncthreads();
    }

    // Epilogue.  Lane holds C(m = base_m + lane%32, n = base_n + 8g + 4*(lane/32) + 0..3)
    // in acc[..][..][4g .. 4g+3].
    const int lrow = lane & 31;
    const int lcol = (lane >> 5) * 4;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int64_t m = m0 + wm * WM + i * 32 + lrow;
        if (m >= a.M) continue;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int64_t n = n0 + wn * WN + j * 32 + g * 8 + lcol;
                if (n >= a.N) continue;
                float v[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = acc[i][j][4 * g + r];
                if constexpr (EPI == EPI_BIAS || EPI == EPI_BIAS_GELU) {
                    const u32x2 bb = *reinterpret_cast<const u32x2*>(a.bias + n);
                    v[0] += bf16_to_f32(bb[0] & 0xffffu);
                    v[1] += bf16_to_f32(bb[0] >> 16);
                    v[2] += bf16_to_f32(bb[1] & 0xffffu);
                    v[3] += bf16_to_f32(bb[1] >> 16);
                }
                if constexpr (EPI == EPI_BIAS_GELU) {
                    if (a.pre_out) {
                        u32x2 pp;
                        pp[0] = f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16);
                        pp[1] = f32_to_bf16_rne(v[2]) | (f32_to_bf16_rne(v[3]) << 16);
                        *reinterpret_cast<u32x2*>(a.pre_out + m * a.ldc + n) = pp;
                    }
#pragma unroll
                    for (int r = 0; r < 4; ++r) v[r] = gelu_f(v[r]);
                }
                if constexpr (EPI == EPI_GELU_BWD) {
                    const u32x2 pp = *reinterpret_cast<const u32x2*>(a.pre_in + m * a.ldc + n);
                    v[0] *= gelu_grad_f(bf16_to_f32(pp[0] & 0xffffu));
                    v[1] *= gelu_grad_f(bf16_to_f32(pp[0] >> 16));
                    v[2] *= gelu_grad_f(bf16_to_f32(pp[1] & 0xffffu));
                    v[3] *= gelu_grad_f(bf16_to_f32(pp[1] >> 16));
                }
                if constexpr (OUT_BF16) {
                    u32x2 o;
                    o[0] = f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16);
                    o[1] = f32_to_bf16_rne(v[2]) | (f32_to_bf16_rne(v[3]) << 16);
                    *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(a.C) + m * a.ldc + n) = o;
                } else {
                    *reinterpret_cast<f32x4*>(static_cast<float*>(a.C) + m * a.ldc + n) =
                        f32x4{v[0], v[1], v[2], v[3]};
                }
            }
        }
    }
}

template <bool A_K, bool B_K, int EPI, bool OUT_BF16>
hipError_t launch_t(const GemmProblem& p, hipStream_t s) {
    KArgs a;
    a.A = static_cast<const uint16_t*>(p.A);
    a.lda = p.lda;
    a.B = static_cast<const uint16_t*>(p.B);
    a.ldb = p.ldb;
    a.C = p.C;
    a.ldc = p.ldc;
    a.bias = static_cast<const uint16_t*>(p.bias);
    a.pre_in = static_cast<const uint16_t*>(p.pre_in);
    a.pre_out = static_cast<uint16_t*>(p.pre_out);
    a.M = p.M;
    a.N = p.N;
    a.K = p.K;
    a.tiles_m = (int)((p.M + BM - 1) / BM);
    a.tiles_n = (int)((p.N + BN - 1) / BN);
    const int grid = a.tiles_m * a.tiles_n;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL((gemm_kernel<A_K, B_K, EPI, OUT_BF16>), dim3(grid), dim3(NT), 0, s, a);
    return hipGetLastError();
}

}  // namespace

bool gemm_supported(int layout, int epi, bool out_bf16) {
    switch (layout) {
    case LAYOUT_NN:
        return epi == EPI_NONE || epi == EPI_BIAS || epi == EPI_BIAS_GELU;
    case LAYOUT_NT:
        return epi == EPI_NONE || (epi == EPI_GELU_BWD && out_bf16);
    case LAYOUT_TN:
        return epi == EPI_NONE && !out_bf16;
    default:
        return false;
    }
}

const char* gemm_kernel_name(int layout) {
    switch (layout) {
    case LAYOUT_NN: return "gemm_nn";
    case LAYOUT_NT: return "gemm_nt";
    case LAYOUT_TN: return "gemm_tn";
    default: return "gemm_?";
    }
}

hipError_t launch_gemm(const GemmProblem& p, hipStream_t s) {
    if (p.M <= 0 || p.N <= 0) return hipSuccess;
    const bool b16 = p.out_bf16;
    switch (p.layout) {
    case LAYOUT_NN:
        switch (p.epi) {
        case EPI_NONE:
            return b16 ? launch_t<true, false, EPI_NONE, true>(p, s)
                       : launch_t<true, false, EPI_NONE, false>(p, s);
        case EPI_BIAS:
            return b16 ? launch_t<true, false, EPI_BIAS, true>(p, s)
                       : launch_t<true, false, EPI_BIAS, false>(p, s);
        case EPI_BIAS_GELU:
            return b16 ? launch_t<true, false, EPI_BIAS_GELU, true>(p, s)
                       : launch_t<true, false, EPI_BIAS_GELU, false>(p, s);
        default:
            return hipErrorInvalidValue;
        }
    case LAYOUT_NT:
        if (p.epi == EPI_NONE)
            return b16 ? launch_t<true, true, EPI_NONE, true>(p, s)
                       : launch_t<true, true, EPI_NONE, false>(p, s);
        if (p.epi == EPI_GELU_BWD && b16) return launch_t<true, true, EPI_GELU_BWD, true>(p, s);
        return hipErrorInvalidValue;
    case LAYOUT_TN:
        if (p.epi == EPI_NONE && !b16) return launch_t<false, false, EPI_NONE, false>(p, s);
        return hipErrorInvalidValue;
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace atp
