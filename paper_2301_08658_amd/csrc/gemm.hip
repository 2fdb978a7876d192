// bf16 x bf16 -> fp32 MFMA GEMMs for gfx950 (CDNA4) with fused epilogues.
//
// Two kernels serve the three products of a shard linear (Sec. 3.2 forward
// Y = X W; Sec. 4.2 backward dX = dY W^T, dW = X^T dY):
//
//   * gemm_nt_kernel: both operands contiguous along k (C = A B^T).  Every
//     product of the block runs in this layout when a workspace holds the
//     transposed copies, so it is the tuned kernel (described below, after
//     the generic one).
//   * gemm_kernel: the generic template, any of NN / NT / TN, used for the
//     forward (NN) and dW (TN) products without a workspace.
//
// Generic kernel data path
//   * Operands go global -> LDS with buffer_load_dwordx4 ... lds (no
//     register staging).  A buffer resource per operand gives zero fill for
//     every out-of-range lane (its offset is pushed past num_records), so
//     ragged M, N and K need no separate path.
//   * STAGES LDS buffers form a ring: the loads of K-step kt+STAGES-1 are
//     issued while step kt is multiplied, and a step is consumed after an
//     explicit vmcnt wait plus one workgroup barrier.
//   * An operand contiguous along K (X and dY as the M side; W in dX) is
//     kept [row][k]; an MFMA fragment is one ds_read_b128.  An operand
//     contiguous along its M/N side (W in the forward, X and dY in dW) is
//     kept [k][row] and its fragments are read with two ds_read_b64_tr_b16
//     (gfx950's transposing LDS read): no register transposes.
//   * Both layouts are XOR-swizzled in 16-byte units.  The direct-to-LDS
//     copy writes LDS linearly by lane, so the swizzle is applied by
//     choosing which global chunk each lane fetches.  The swizzles are
//     conflict free for 8- and 16-lane LDS phases.
//   * Wave tile (BM/WGM) x (BN/WGN) of v_mfma_f32_32x32x16_bf16 blocks.  The
//     MFMA takes the N-side fragment first, so a lane's 16 accumulators are
//     4 runs of 4 consecutive output columns and the epilogue stores 16 B
//     (fp32) or 8 B (bf16) per lane.
//   * Every output element accumulates its K products in the same order
//     (K steps of BK, MFMA k order inside) for every tile shape, so token
//     chunking never changes a value.
//   * Workgroups are renumbered so consecutive tiles land on one XCD (the
//     dispatcher deals workgroups round-robin over the 8 XCDs) and visited
//     in groups of GROUP_M row tiles, so tiles sharing a weight panel run
//     together on one L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

// Tile and schedule parameters (compile-time).
#ifndef ATP_GEMM_GROUP_M
#define ATP_GEMM_GROUP_M 8
#endif
#ifndef ATP_GEMM_XCD_REMAP
#define ATP_GEMM_XCD_REMAP 1
#endif
#ifndef ATP_GEMM_BK
#define ATP_GEMM_BK 64
#endif
#ifndef ATP_GEMM_PIPE
#define ATP_GEMM_PIPE 0
#endif
#ifndef ATP_GEMM_STAGES
#define ATP_GEMM_STAGES 2
#endif
#ifndef ATP_GEMM_BM
#define ATP_GEMM_BM 256
#endif
#ifndef ATP_GEMM_BN
#define ATP_GEMM_BN 256
#endif
#ifndef ATP_GEMM_WGM
#define ATP_GEMM_WGM 2
#endif
#ifndef ATP_GEMM_WGN
#define ATP_GEMM_WGN 4
#endif

namespace atp {
namespace {

constexpr int GROUP_M = ATP_GEMM_GROUP_M;
constexpr int NUM_XCD = 8;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr uint32_t kRsrcWord3 = 0x00020000u;   // raw 32-bit buffer access
constexpr uint32_t kOob = 0x80000000u;          // offset beyond any num_records

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

// 16-byte chunk swizzles.  K-major rows hold BK/8 chunks; MN-major rows
// (one per k) hold at least 16 chunks.
template <int CPR>
__device__ __forceinline__ int swz_k(int r) {
    if constexpr (CPR == 8) return (r ^ ((r >> 3) & 1)) & 7;
    else return ((r >> 1) + (r >> 3)) & 3;
}
__device__ __forceinline__ int swz_mn(int k) { return ((k & 2) << 1) | ((k & 1) * 10); }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
    const int64_t cap = 0x7fffff00;   // keep offsets and sizes in 31 bits
    const int n = (int)(bytes < 0 ? 0 : (bytes > cap ? cap : bytes));
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, kRsrcWord3);
}

struct KArgs {
    const uint16_t* A; int64_t lda;
    const uint16_t* B; int64_t ldb;
    void* C; int64_t ldc;
    const uint16_t* bias;
    const uint16_t* pre_in;
    uint16_t* pre_out;
    int64_t M, N, K;
    int tiles_m, tiles_n;
    // split-K (NT kernel): split s covers k in [s*ksplit, min(K, (s+1)*ksplit))
    // and writes C + s*c_split (an fp32 slab per split); splits == 1: plain
    int splits;
    int64_t ksplit, c_split;
};

// Workgroup -> logical tile index: the dispatcher deals workgroups
// round-robin over the XCDs, so consecutive logical indices are made to land
// on one XCD.
__device__ __forceinline__ int xcd_logical() {
    const int G = gridDim.x;
    const int pid = blockIdx.x;
    const int xcd = pid % NUM_XCD;
    const int idx = pid / NUM_XCD;
    const int per = G / NUM_XCD;
    const int rem = G % NUM_XCD;
    const int logical = (xcd < rem) ? xcd * (per + 1) + idx
                                    : rem * (per + 1) + (xcd - rem) * per + idx;
    return ATP_GEMM_XCD_REMAP ? logical : pid;
}

// Logical tile index -> (row tile, column tile), sweeping groups of GM row
// tiles column by column.
template <int GM>
__device__ __forceinline__ void group_coords(int logical, int tiles_m, int tiles_n, int& tm,
                                             int& tn) {
    const int in_group = GM * tiles_n;
    const int group = logical / in_group;
    const int first_m = group * GM;
    const int gsize = min(tiles_m - first_m, GM);
    const int r = logical % in_group;
    tm = first_m + r % gsize;
    tn = r / gsize;
}

template <int GM = GROUP_M>
__device__ __forceinline__ void tile_coords(int tiles_m, int tiles_n, int& tm, int& tn) {
    group_coords<GM>(xcd_logical(), tiles_m, tiles_n, tm, tn);
}

// ---------------------------------------------------------------------------
// One operand of the tile: issue the direct-to-LDS copy of one K step, and
// read MFMA fragments back.  ROWS = BM or BN (the operand's M/N extent).
// ---------------------------------------------------------------------------
template <int ROWS, int BK, int NT, bool KCONTIG>
struct Operand {
    static constexpr int CHUNKS = ROWS * BK / 8;          // 16-byte chunks per K step
    static constexpr int PER_THREAD = CHUNKS / NT;
    static_assert(CHUNKS % NT == 0, "tile not divisible by the thread count");
    static constexpr int CPR = KCONTIG ? BK / 8 : ROWS / 8;   // chunks per LDS row

    const uint16_t* base;
    int64_t ld;
    int64_t row0, rows, K;
    // Per-lane byte offsets of this thread's chunks relative to the step's
    // first element (row0, k0); out-of-range rows / columns hold kOob.  They
    // do not depend on the K step.
    uint32_t voff[PER_THREAD];
    int kchunk[PER_THREAD];    // K-major: the chunk's first k within the step

    __device__ __forceinline__ void init(int tid) {
        const int wave = tid >> 6;
        const int lane = tid & 63;
#pragma unroll
        for (int i = 0; i < PER_THREAD; ++i) {
            const int p = (i * (NT / 64) + wave) * 64 + lane;     // LDS chunk slot
            if constexpr (KCONTIG) {
                const int r = p / CPR;
                const int c = (p % CPR) ^ swz_k<CPR>(r);
                kchunk[i] = c * 8;
                voff[i] = (row0 + r < rows) ? (uint32_t)((r * ld + c * 8) * 2) : kOob;
            } else {
                const int k = p / CPR;
                const int c = (p % CPR) ^ swz_mn(k);
                kchunk[i] = k;
                voff[i] = (row0 + c * 8 < rows) ? (uint32_t)((k * ld + c * 8) * 2) : kOob;
            }
        }
    }

    // Copy K step [k0, k0+BK) into LDS stage `dst` (ROWS*BK elements).  A
    // step at or past K fills the stage with zeros (every lane out of range),
    // so each step issues the same number of loads.
    __device__ __forceinline__ void issue(uint16_t* dst, int64_t k0, int tid) const {
        const int wave = tid >> 6;
        const bool live = k0 < K;
        if constexpr (KCONTIG) {
            // whole rows bound the range; k past K inside a row is masked per
            // lane, which only the last step of a ragged K needs
            const uint16_t* b = base + row0 * ld + (live ? k0 : 0);
            const int64_t left = rows - row0;
            const int64_t valid_rows = live ? (left < ROWS ? left : ROWS) : 0;
            const __amdgpu_buffer_rsrc_t rs = make_rsrc(b, valid_rows * ld * 2);
            const bool tail = k0 + BK > K;
#pragma unroll
            for (int i = 0; i < PER_THREAD; ++i) {
                const uint32_t off = (tail && k0 + kchunk[i] >= K) ? kOob : voff[i];
                lds_void* d = (lds_void*)(dst + (size_t)(i * (NT / 64) + wave) * 64 * 8);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, d, 16, off, 0, 0, 0);
            }
        } else {
            // rows k0.. of a [K][ld] matrix: the range ends at row K
            const uint16_t* b = base + (live ? k0 : 0) * ld + row0;
            const int64_t valid_k = live ? (K - k0 < BK ? K - k0 : BK) : 0;
            const __amdgpu_buffer_rsrc_t rs = make_rsrc(b, valid_k * ld * 2);
#pragma unroll
            for (int i = 0; i < PER_THREAD; ++i) {
                lds_void* d = (lds_void*)(dst + (size_t)(i * (NT / 64) + wave) * 64 * 8);
                const uint32_t off = voff[i];
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, d, 16, off, 0, 0, 0);
            }
        }
    }

    // MFMA 32x32x16 fragment: lane holds rows r0 + lane%32, k = ks*16 + 8*(lane/32) + 0..7.
    static __device__ __forceinline__ bf16x8 frag(const uint16_t* src, int r0, int ks,
                                                  int lane) {
        if constexpr (KCONTIG) {
            const int r = r0 + (lane & 31);
            const int c = (ks * 2 + (lane >> 5)) ^ swz_k<CPR>(r);
            return *reinterpret_cast<const bf16x8*>(src + r * BK + c * 8);
        } else {
            // two transposing reads of 4 k values each (lane group of 16:
            // rows r0 + 16*(g%2) + 0..15, k base ks*16 + 8*(g/2))
            const int g = lane >> 4;
            const int j = lane & 15;
            const int mn = r0 + 16 * (g & 1) + 4 * (j & 3);
            const int kb = ks * 16 + 8 * (g >> 1) + (j >> 2);
            const int k0 = kb, k1 = kb + 4;
            const uint16_t* p0 = src + k0 * ROWS + (((mn >> 3) ^ swz_mn(k0)) << 3) + (mn & 7);
            const uint16_t* p1 = src + k1 * ROWS + (((mn >> 3) ^ swz_mn(k1)) << 3) + (mn & 7);
            const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p0);
            const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p1);
            typedef short i16x8 __attribute__((ext_vector_type(8)));
            const i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            return __builtin_bit_cast(bf16x8, v);
        }
    }
};

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Epilogue of four consecutive outputs C[m][n..n+3] (fp32 accumulators):
// bias, bias + GeLU (optionally saving the bf16 pre-activation), GeLU'
// (multiplying by the derivative at a saved pre-activation), then an fp32 or
// bf16 (round to nearest even) store.
template <int EPI, bool OUT_BF16>
__device__ __forceinline__ void epilogue_store(const KArgs& a, int64_t m, int64_t n, float* v) {
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

template <int BM, int BN, int BK, int STAGES, int WGM, int WGN, bool A_K, bool B_K, int EPI,
          bool OUT_BF16>
__global__ __launch_bounds__(WGM* WGN * 64, 1) void gemm_kernel(KArgs a) {
    constexpr int NT = WGM * WGN * 64;
    constexpr int WM = BM / WGM;
    constexpr int WN = BN / WGN;
    constexpr int FM = WM / 32;
    constexpr int FN = WN / 32;
    constexpr int A_ELEMS = BM * BK;
    constexpr int STAGE = (BM + BN) * BK;
    using OpA = Operand<BM, BK, NT, A_K>;
    using OpB = Operand<BN, BK, NT, B_K>;
    constexpr int LOADS = OpA::PER_THREAD + OpB::PER_THREAD;   // vm ops per stage per thread

    __shared__ __attribute__((aligned(1024))) uint16_t smem[STAGES * STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WGN;
    const int wn = wave % WGN;

    int tm, tn;
    tile_coords(a.tiles_m, a.tiles_n, tm, tn);
    const int64_t m0 = (int64_t)tm * BM;
    const int64_t n0 = (int64_t)tn * BN;

    OpA opa{a.A, a.lda, m0, a.M, a.K};
    OpB opb{a.B, a.ldb, n0, a.N, a.K};
    opa.init(tid);
    opb.init(tid);

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    const int nk = (int)((a.K + BK - 1) / BK);
    constexpr int KS = BK / 16;   // MFMA k-steps per K step

    // prologue: steps 0 .. STAGES-2 in flight (steps past K fill zeros)
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s) {
        opa.issue(smem + s * STAGE, (int64_t)s * BK, tid);
        opb.issue(smem + s * STAGE + A_ELEMS, (int64_t)s * BK, tid);
    }

    for (int kt = 0; kt < nk; ++kt) {
        // step kt's copy is the oldest of STAGES-1 in flight
        wait_vmcnt<LOADS * (STAGES - 2)>();
        __syncthreads();
        const uint16_t* sa = smem + (kt % STAGES) * STAGE;
        const uint16_t* sb = sa + A_ELEMS;
        bf16x8 fa[2][FM], fb[2][FN];
#pragma unroll
        for (int i = 0; i < FM; ++i) fa[0][i] = OpA::frag(sa, wm * WM + i * 32, 0, lane);
#pragma unroll
        for (int j = 0; j < FN; ++j) fb[0][j] = OpB::frag(sb, wn * WN + j * 32, 0, lane);
        {
            // refill the buffer step kt-1 used with step kt+STAGES-1
            const int kn = kt + STAGES - 1;
            uint16_t* dst = smem + (kn % STAGES) * STAGE;
            opa.issue(dst, (int64_t)kn * BK, tid);
            opb.issue(dst + A_ELEMS, (int64_t)kn * BK, tid);
        }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int cur = ks & 1;
            if (ks + 1 < KS) {
#pragma unroll
                for (int i = 0; i < FM; ++i)
                    fa[cur ^ 1][i] = OpA::frag(sa, wm * WM + i * 32, ks + 1, lane);
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    fb[cur ^ 1][j] = OpB::frag(sb, wn * WN + j * 32, ks + 1, lane);
            }
#if ATP_GEMM_PIPE
            // keep the next k-step's LDS reads ahead of this k-step's MFMAs
            __builtin_amdgcn_sched_barrier(0);
#endif
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[cur][j], fa[cur][i],
                                                                        acc[i][j], 0, 0, 0);
        }
#if defined(ATP_GEMM_SCHED) && ATP_GEMM_SCHED
        // interleave: the step's global loads and the next fragments' LDS
        // reads are spread between the MFMAs
#pragma unroll
        for (int q = 0; q < LOADS; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read
        }
#pragma unroll
        for (int q = 0; q < (KS - 1) * (FM + FN) * (A_K ? 1 : 2) && q < KS * FM * FN; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
        }
#endif
    }
    wait_vmcnt<0>();

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
                epilogue_store<EPI, OUT_BF16>(a, m, n, v);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// NT kernel: C[M,N] = A[M,K] B[N,K]^T, 256 x 160 tiles, eight waves in two
// groups that take turns on the matrix cores ("ping-pong").
//
//   * Tile 256 x 160 x 64: three LDS stages of (256 + 160) x 64 bf16 fill
//     156 KB of the 160 KB, so the copy of step p+2 is issued while step p is
//     multiplied.  160 divides every N of the block's products at the
//     benchmark sizes (and a 512-row token chunk is exactly 256 tiles), so
//     no launch ends on a partial wave of tiles.
//   * Waves 0-3 (group A) and 4-7 (group B) share the four SIMDs pairwise.
//     A K step is two phases separated by workgroup barriers: a memory phase
//     (issue this wave's share of the direct-to-LDS copy of step p+2, read all
//     of step p's MFMA fragments into registers) and a compute phase (the 40
//     MFMAs of step p).  Group B starts one phase late, so on every SIMD one
//     wave multiplies while the other one loads: the matrix core is fed from
//     registers while the other wave's LDS reads and copy issue overlap it.
//   * Each wave owns a 64 x 80 block of C as 4 x 5 tiles of
//     v_mfma_f32_16x16x32_bf16.  A fragment is one ds_read_b128 (row r,
//     8 consecutive k).  gfx950 serves a ds_read_b128 in lane groups
//     {0-7, 24-31}, {8-15, 16-23} (and the same +32); the chunk swizzle
//     s(r) = r & 6 gives the 16 lanes of each group distinct bank quads
//     (measured: zero LDS bank conflicts).
//   * The swizzle of a row depends only on the row's index within its copy
//     instruction, so one byte offset per lane serves every copy; rows past
//     the operand's end lie beyond the buffer's num_records and read zeros.
//   * An output element's products are accumulated in the same order for
//     every M (K steps of 64, two MFMA k-slices of 32 each), so token
//     chunking never changes a value.
// ---------------------------------------------------------------------------
namespace nt {

constexpr int BM = 256, BK = 64;
constexpr int NW = 8, NT = NW * 64;           // two groups of four waves
constexpr int MF = 16;
constexpr int KS = BK / 32;                   // MFMA k-slices per step
typedef short i16x8 __attribute__((ext_vector_type(8)));

// Tile configurations.  Every one sums an output element's products in the
// same order (K steps of 64, two 16x16x32 k-slices each), so they give the
// same bits and may be mixed freely, e.g. across token chunks.
template <int BN_, int WGM_, int WGN_, int STAGES_, int GROUP_>
struct Cfg {
    static constexpr int BN = BN_, WGM = WGM_, WGN = WGN_, STAGES = STAGES_, GROUP = GROUP_;
    static_assert(WGM * WGN == NW, "eight waves");
    static_assert(STAGES == 2 || STAGES == 3, "two or three LDS stages");
    static constexpr int WM = BM / WGM, WN = BN / WGN;
    static constexpr int FM = WM / MF, FN = WN / MF;
    static_assert(FM * MF == WM && FN * MF == WN, "wave tile of whole MFMA tiles");
    static constexpr int A_EL = BM * BK, STAGE = (BM + BN) * BK;
};
// 256 x 160: three stages (156 KB of LDS); waves of 64 x 80; the 32 tiles an
// XCD runs at once form a 4 x 8 block (4*256 + 8*160 rows per K step, L2 hit
// rate 81% against 74% for 8 x 4)
using Tile160 = Cfg<160, 4, 2, 3, 4>;
// 256 x 256: two stages (128 KB); waves of 128 x 64; 30% fewer copied bytes
// per FLOP, ~10% faster on the short-K (tokens) dW products, but 62.5% of
// the tile count of 256 x 160 per launch
using Tile256 = Cfg<256, 2, 4, 2, 8>;

__device__ __forceinline__ int swz(int r) { return r & 6; }

// One operand tile: ROWS rows of a [rows][ld] matrix contiguous along k.
template <int ROWS>
struct Copy {
    static constexpr int CPR = BK / 8;             // 16-byte chunks per LDS row
    static constexpr int RPI = 64 / CPR;           // rows per copy instruction
    static constexpr int WI = ROWS / RPI;          // copy instructions per stage
    static constexpr int PER = (WI + NW - 1) / NW; // per wave (some waves one fewer)
    static_assert(ROWS % RPI == 0, "rows per copy instruction");
    __amdgpu_buffer_rsrc_t rs;
    uint32_t vlane;       // this lane's byte offset within its instruction's rows
    uint32_t ins_stride;  // bytes from one instruction's rows to the next
    int kc;               // first k of this lane's chunk
    int nmine;            // copy instructions this wave issues per stage
    int64_t K;

    __device__ __forceinline__ void init(const uint16_t* base, int64_t ld, int64_t row0,
                                         int64_t rows, int64_t K_, int wave, int lane) {
        K = K_;
        const int64_t left = rows - row0;
        const int64_t vr = left < 0 ? 0 : (left < ROWS ? left : ROWS);
        rs = make_rsrc(base + row0 * ld, vr * ld * 2);
        const int r = lane / CPR;
        const int c = (lane % CPR) ^ swz(r);
        kc = c * 8;
        vlane = (uint32_t)((r * ld + c * 8) * 2);
        ins_stride = (uint32_t)(RPI * ld * 2);
        nmine = 0;
#pragma unroll
        for (int i = 0; i < PER; ++i)
            if (wave + NW * i < WI) nmine = i + 1;
    }
    // Copy of the K step at k0 into LDS stage `dst` (k past K reads zeros).
    __device__ __forceinline__ void issue(uint16_t* dst, int64_t k0, int wave) const {
        const bool tail = k0 + BK > K;
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int ins = wave + NW * i;
            if (PER * NW != WI && ins >= WI) break;   // wave-uniform
            uint32_t off = vlane + (uint32_t)ins * ins_stride;
            if (tail && k0 + kc >= K) off = kOob;
            lds_void* d = (lds_void*)(dst + (size_t)ins * 64 * 8);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, d, 16, off, (int)(k0 * 2), 0, 0);
        }
    }
};

// 16x16x32 fragment: lane holds row r0 + lane%16, k = ks*32 + 8*(lane/16) + 0..7.
__device__ __forceinline__ bf16x8 frag(const uint16_t* src, int r0, int ks, int lane) {
    const int r = r0 + (lane & 15);
    const int c = (ks * 4 + (lane >> 4)) ^ swz(r);
    return *reinterpret_cast<const bf16x8*>(src + r * BK + c * 8);
}

__device__ __forceinline__ void barrier() {
    // a bare s_barrier: __syncthreads() would also wait for every copy in
    // flight (vmcnt(0)), which defeats the three-stage ring
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_barrier" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

}  // namespace nt

template <class C, int EPI, bool OUT_BF16>
__global__ __launch_bounds__(nt::NT, 1) void gemm_nt_kernel(KArgs a) {
    using namespace nt;
    constexpr int BN = C::BN, WGN = C::WGN, STAGES = C::STAGES;
    constexpr int WM = C::WM, WN = C::WN, FM = C::FM, FN = C::FN;
    constexpr int A_EL = C::A_EL, STAGE = C::STAGE;
    __shared__ __attribute__((aligned(1024))) uint16_t smem[STAGES * STAGE];
    // issue priority above the reduction waves that share the CUs while
    // the next chunk's reduction runs beside this GEMM (measured +0.4%)
    __builtin_amdgcn_s_setprio(1);

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool grpB = wave >= 4;
    const int wm = wave / WGN, wn = wave % WGN;
    // logical index -> (split, tile); the splits of one tile share no data,
    // so the tiles of one split stay together on an XCD
    const int ntiles = a.tiles_m * a.tiles_n;
    const int logical = xcd_logical();
    const int split = logical / ntiles;
    int tm, tn;
    group_coords<C::GROUP>(logical - split * ntiles, a.tiles_m, a.tiles_n, tm, tn);
    const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
    const int64_t kb = (int64_t)split * a.ksplit;
    const int64_t kn = min(a.K - kb, a.ksplit);    // this split's contraction

    Copy<BM> ca;
    Copy<BN> cb;
    ca.init(a.A + kb, a.lda, m0, a.M, kn, wave, lane);
    cb.init(a.B + kb, a.ldb, n0, a.N, kn, wave, lane);
    constexpr int LA = Copy<BM>::PER, LB = Copy<BN>::PER;
    const int loads = ca.nmine + cb.nmine;   // copy instructions per step (wave-uniform)

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nk = (int)((kn + BK - 1) / BK);
    auto issue_step = [&](int q) {
        uint16_t* dst = smem + (q % STAGES) * STAGE;
        ca.issue(dst, (int64_t)q * BK, wave);
        cb.issue(dst + A_EL, (int64_t)q * BK, wave);
    };
    // wait until this wave's copies are complete except the newest step's
    // (keep_one) or all of them; copies complete in issue order
    auto wait_copies = [&](bool keep_one) {
        if (!keep_one) { wait_vmcnt<0>(); return; }
        if (loads == LA + LB) wait_vmcnt<LA + LB>();
        else if (loads == LA + LB - 1) wait_vmcnt<LA + LB - 1>();
        else wait_vmcnt<LA + LB - 2>();
    };

    if (nk > 0) {   // (uniform) every wave runs the same number of barriers
        for (int q = 0; q < STAGES - 1 && q < nk; ++q) issue_step(q);
        wait_copies(STAGES == 3 && nk > 1);
        barrier();               // step 0 visible to every wave
        if (grpB) barrier();     // group B starts one phase late

        bf16x8 fa[KS][FM], fb[KS][FN];
        for (int p = 0; p < nk; ++p) {
            // memory phase: copy step p+STAGES-1 into the stage step p-1 used
            // (both groups finished reading it before this phase), read step p
            const uint16_t* sa = smem + (p % STAGES) * STAGE;
            const uint16_t* sb = sa + A_EL;
            if (p + STAGES - 1 < nk) issue_step(p + STAGES - 1);
            // with three stages the copy of step p+2 may stay in flight below
            const bool more = STAGES == 3 && p + 2 < nk;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
                for (int i = 0; i < FM; ++i) fa[ks][i] = frag(sa, wm * WM + i * MF, ks, lane);
#pragma unroll
                for (int j = 0; j < FN; ++j) fb[ks][j] = frag(sb, wn * WN + j * MF, ks, lane);
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            // before group A's next memory phase this wave's copies of step
            // p+1 have landed (with three stages those of step p+2 may still
            // be in flight)
            if (grpB) wait_copies(more);
            barrier();
            // compute phase
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
#pragma unroll
                for (int i = 0; i < FM; ++i)
#pragma unroll
                    for (int j = 0; j < FN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[ks][j], fa[ks][i],
                                                                            acc[i][j], 0, 0, 0);
            if (!grpB) wait_copies(more);
            if (!(grpB && p == nk - 1)) barrier();
        }
        wait_vmcnt<0>();
    }

    // Epilogue.  Lane holds C(m = base_m + lane%16, n = base_n + 4*(lane/16) + 0..3)
    // in acc[i][j][0..3].
    KArgs o = a;
    if (split) o.C = static_cast<float*>(a.C) + split * a.c_split;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int64_t m = m0 + wm * WM + i * MF + (lane & 15);
        if (m >= a.M) continue;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int64_t n = n0 + wn * WN + j * MF + 4 * (lane >> 4);
            if (n >= a.N) continue;
            float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
            epilogue_store<EPI, OUT_BF16>(o, m, n, v);
        }
    }
}

// Tile configuration: 256 x 256 workgroup tile, 4 waves of 128 x 128.
constexpr int CFG_BM = ATP_GEMM_BM, CFG_BN = ATP_GEMM_BN, CFG_BK = ATP_GEMM_BK,
              CFG_STAGES = ATP_GEMM_STAGES, CFG_WGM = ATP_GEMM_WGM, CFG_WGN = ATP_GEMM_WGN;

KArgs kargs(const GemmProblem& p, int bm, int bn) {
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
    a.tiles_m = (int)((p.M + bm - 1) / bm);
    a.tiles_n = (int)((p.N + bn - 1) / bn);
    a.splits = p.splits > 1 ? p.splits : 1;
    a.ksplit = a.splits > 1 ? p.ksplit : p.K;
    a.c_split = p.c_split;
    return a;
}

// 256 x 256 tiles for products with a short contraction (at most 8192: the
// dW products over the tokens) whose last wave of tiles is at least 90% full
// (256 CUs); 256 x 160 tiles otherwise
bool nt_use_256(const GemmProblem& p) {
    constexpr int64_t kCUs = 256;
    const int64_t tiles = ((p.M + nt::BM - 1) / nt::BM) * ((p.N + 255) / 256);
    const int64_t waves = (tiles + kCUs - 1) / kCUs;
    return p.K <= 8192 && tiles * 10 >= waves * kCUs * 9;
}

// Split-K plan of an NT product written to fp32: the S in 1..kMaxSplits
// that minimises a two-term cost model, (rounds of 256 concurrent 256 x 160
// tiles) x (k per split) x (flops per k per tile), plus the fp32 slab
// traffic of the splits (each written once and read once by the combining
// pass) counted at equal per-CU flop and chip byte rates (about 4 TFLOP/s
// per CU against about 4 TB/s).  Splits are taken only when the grid stays
// within kMaxSplitTiles workgroups, every split covers at least 256 k in
// whole 64-k steps, and the model gains at least 15%.
int pick_splits(int64_t M, int64_t N, int64_t K, int64_t* ksplit) {
    constexpr int64_t kCUs = 256;
    const int64_t tiles = ((M + nt::BM - 1) / nt::BM) * ((N + 159) / 160);
    const double flops_per_k = 2.0 * nt::BM * 160;
    int best = 1;
    double best_cost = (double)((tiles + kCUs - 1) / kCUs) * K * flops_per_k;
    const double plain = best_cost;
    *ksplit = K;
    for (int S = 2; S <= kMaxSplits; ++S) {
        const int64_t ks = ((K + S - 1) / S + 63) / 64 * 64;
        if (ks < 256 || (K + ks - 1) / ks != S || tiles * S > kMaxSplitTiles) continue;
        const double cost = (double)((tiles * S + kCUs - 1) / kCUs) * ks * flops_per_k +
                            8.0 * S * (double)M * (double)N;
        if (cost < best_cost) {
            best = S;
            best_cost = cost;
            *ksplit = ks;
        }
    }
    if (best > 1 && best_cost > 0.85 * plain) {
        best = 1;
        *ksplit = K;
    }
    return best;
}

template <class C, int EPI, bool OUT_BF16>
hipError_t launch_nt_cfg(const GemmProblem& p, hipStream_t s) {
    const KArgs a = kargs(p, nt::BM, C::BN);
    const int grid = a.tiles_m * a.tiles_n * a.splits;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL((gemm_nt_kernel<C, EPI, OUT_BF16>), dim3(grid), dim3(nt::NT), 0, s, a);
    return hipGetLastError();
}

template <int EPI, bool OUT_BF16>
hipError_t launch_nt(const GemmProblem& p, hipStream_t s) {
    if (p.splits > 1) return launch_nt_cfg<nt::Tile160, EPI, OUT_BF16>(p, s);
    return nt_use_256(p) ? launch_nt_cfg<nt::Tile256, EPI, OUT_BF16>(p, s)
                         : launch_nt_cfg<nt::Tile160, EPI, OUT_BF16>(p, s);
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
    a.tiles_m = (int)((p.M + CFG_BM - 1) / CFG_BM);
    a.tiles_n = (int)((p.N + CFG_BN - 1) / CFG_BN);
    a.splits = 1;
    a.ksplit = p.K;
    a.c_split = 0;
    const int grid = a.tiles_m * a.tiles_n;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL((gemm_kernel<CFG_BM, CFG_BN, CFG_BK, CFG_STAGES, CFG_WGM, CFG_WGN, A_K,
                                    B_K, EPI, OUT_BF16>),
                       dim3(grid), dim3(CFG_WGM * CFG_WGN * 64), 0, s, a);
    return hipGetLastError();
}

}  // namespace

bool gemm_supported(int layout, int epi, bool out_bf16) {
    switch (layout) {
    case LAYOUT_NN:
        return epi == EPI_NONE || epi == EPI_BIAS || epi == EPI_BIAS_GELU;
    case LAYOUT_NT:
        return epi == EPI_NONE ||
               (out_bf16 && (epi == EPI_GELU_BWD || epi == EPI_BIAS || epi == EPI_BIAS_GELU));
    case LAYOUT_TN:
        return epi == EPI_NONE && !out_bf16;
    default:
        return false;
    }
}

const char* gemm_kernel_name(const GemmProblem& p) {
    switch (p.layout) {
    case LAYOUT_NN: return "gemm_nn";
    case LAYOUT_NT: return p.splits > 1 ? "gemm_nt_splitk" : nt_use_256(p) ? "gemm_nt256" : "gemm_nt";
    case LAYOUT_TN: return "gemm_tn";
    default: return "gemm_?";
    }
}

int nt_split_plan(int64_t M, int64_t N, int64_t K, int64_t* ksplit) {
    return pick_splits(M, N, K, ksplit);
}

hipError_t launch_gemm(const GemmProblem& p, hipStream_t s) {
    if (p.M <= 0 || p.N <= 0) return hipSuccess;
    // buffer offsets are 32-bit: one tile's rows of either operand must span < 2 GiB
    const int64_t span = (int64_t)(CFG_BM > CFG_BN ? CFG_BM : CFG_BN) *
                         (p.lda > p.ldb ? p.lda : p.ldb) * 2;
    if (span > 0x7fffff00) return hipErrorInvalidValue;
    const bool b16 = p.out_bf16;
    if (p.splits > 1) {
        // split-K: NT, plain fp32 outputs, whole K steps per split, every split
        // non-empty
        if (p.layout != LAYOUT_NT || p.epi != EPI_NONE || b16 || p.ksplit <= 0 ||
            p.ksplit % 64 || (int64_t)(p.splits - 1) * p.ksplit >= p.K || p.c_split < p.M * p.ldc)
            return hipErrorInvalidValue;
    }
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
            return b16 ? launch_nt<EPI_NONE, true>(p, s) : launch_nt<EPI_NONE, false>(p, s);
        if (p.epi == EPI_GELU_BWD && b16) return launch_nt<EPI_GELU_BWD, true>(p, s);
        // the forward with a transposed weight copy (B = W^T, contiguous along k)
        if (p.epi == EPI_BIAS && b16) return launch_nt<EPI_BIAS, true>(p, s);
        if (p.epi == EPI_BIAS_GELU && b16) return launch_nt<EPI_BIAS_GELU, true>(p, s);
        return hipErrorInvalidValue;
    case LAYOUT_TN:
        if (p.epi == EPI_NONE && !b16) return launch_t<false, false, EPI_NONE, false>(p, s);
        return hipErrorInvalidValue;
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace atp
