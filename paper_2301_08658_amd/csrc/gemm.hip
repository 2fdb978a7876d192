// bf16 x bf16 -> fp32 MFMA GEMMs for gfx950 (CDNA4) with fused epilogues.
//
// One kernel, gemm_nt_kernel, serves the three products of a shard linear
// (Sec. 3.2 forward Y = X W; Sec. 4.2 backward dX = dY W^T, dW = X^T dY) in
// each operand layout: an operand is either contiguous along k (X, dY, and
// W in dX; the transposed copies W^T, X^T, dY^T of the workspace path) or
// contiguous along its rows (W in the forward, X and dY in dW without a
// workspace).  The kernel is described below; every layout sums an output
// element's products in the same order, so the layouts give the same bits.
//
//   * Operands go global -> LDS with buffer_load_dwordx4 ... lds (no
//     register staging).  A buffer resource per operand gives zero fill for
//     every out-of-range lane (its offset is pushed past num_records), so
//     ragged M, N and K need no separate path.
//   * Workgroups are renumbered so consecutive tiles land on one XCD (the
//     dispatcher deals workgroups round-robin over the 8 XCDs) and visited
//     in groups of row tiles, so tiles sharing operand panels run together
//     on one L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "epilogue_math.h"
#include "kernels.h"
#include "lds_dma.h"

#ifndef ATP_GEMM_XCD_REMAP
#define ATP_GEMM_XCD_REMAP 1
#endif

namespace atp {
namespace {

constexpr int NUM_XCD = 8;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;


using epi::bf16_to_f32;
using epi::f32_to_bf16_rne;
using epi::gelu_f;
using epi::gelu_grad_f;

// 16-byte chunk swizzles.  K-major rows hold BK/8 chunks; MN-major rows
// (one per k) hold at least 16 chunks.
using dma::kOob;
using dma::kRsrcWord3;
using dma::lds_dma16;
using dma::rsrc_words;

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
    // fused peer sum (nparts > 1): the group's partials summed in group
    // order, the tile's own accumulators at position own
    int nparts, own;
    const float* peers[kMaxFusedParts];
    int64_t ldp;
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


using dma::wait_vmcnt;

// Epilogue of four consecutive outputs C[m][n..n+3] (fp32 accumulators):
// bias, bias + GeLU (optionally saving the bf16 pre-activation), GeLU'
// (multiplying by the derivative at a saved pre-activation), then an fp32 or
// bf16 (round to nearest even) store.
template <int EPI, bool OUT_BF16>
__device__ __forceinline__ void epilogue_store(const KArgs& a, int64_t m, int64_t n, float* v) {
    if (a.nparts > 1) {
        // Partial(SUM) of the group, summed in group order 0..nparts-1 (the
        // reduction kernel's order, so the bits equal a separate reduction
        // of the same partials); position own is this tile's accumulators
        float t[4] = {v[0], v[1], v[2], v[3]};
#pragma unroll
        for (int j = 0; j < kMaxFusedParts; ++j) {
            if (j >= a.nparts) break;
            f32x4 q = f32x4{t[0], t[1], t[2], t[3]};
            if (j != a.own) q = *reinterpret_cast<const f32x4*>(a.peers[j] + m * a.ldp + n);
            if (j == 0) {
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = q[r];
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] += q[r];
            }
        }
    }
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

// ---------------------------------------------------------------------------
// The kernel: C[M,N] = A B with A [M,K] and B [K,N] each stored contiguous
// along k (A_K / B_K; B then reads [N][K], the NT layout) or along its rows
// (A [K][M], B [K][N]); tiles of 256 rows by 160, 256 or 320 columns (the
// configurations below), eight waves in two groups that take turns on the
// matrix cores ("ping-pong").
//
//   * Waves 0-3 (group A) and 4-7 (group B) share the four SIMDs pairwise.
//     A K step is two phases separated by workgroup barriers: a memory phase
//     (issue this wave's share of the direct-to-LDS copy of a later step,
//     read all of step p's MFMA fragments into registers) and a compute phase
//     (the MFMAs of step p).  Group B starts one phase late, so on every SIMD
//     one wave multiplies while the other one loads: the matrix core is fed
//     from registers while the other wave's LDS reads and copy issue overlap
//     it.
//   * The copies run ahead through LDS: shared stages of both operands (three
//     of (256 + 160) x 64 bf16, 156 KB, for 256 x 160 tiles), or split rings
//     (256 x 256: three stages of A filled by group B, two of B filled by
//     group A, 160 KB), so no copy has to land within the phase that issues
//     it.
//   * A wave owns a block of C as 16 x 16 tiles of v_mfma_f32_16x16x32_bf16
//     (64 x 80 for 256 x 160 tiles, 128 x 64 for 256 x 256).  A fragment is
//     one ds_read_b128 (row r, 8 consecutive k).  gfx950 serves a
//     ds_read_b128 in lane groups {0-7, 24-31}, {8-15, 16-23} (and the same
//     +32); the chunk swizzle s(r) = r & 6 gives the 16 lanes of each group
//     distinct bank quads (measured: zero LDS bank conflicts).
//   * The swizzle of a row depends only on the row's index within its copy
//     instruction, so one byte offset per lane serves every copy; rows past
//     the operand's end lie beyond the buffer's num_records and read zeros.
//   * An operand contiguous along its rows is kept [k][row] in LDS and its
//     fragments come from two ds_read_b64_tr_b16 (gfx950's transposing LDS
//     read); a chunk rotation (160-wide tiles) or XOR (256-wide) keeps each
//     32-lane half of a read on distinct banks (measured: zero conflicts).
//     These reads cost 1.5x the LDS time per byte of ds_read_b128; with the
//     split rings a product whose B is row-contiguous (the forward from W as
//     stored) streams about as fast as the k-contiguous layout.
//   * An output element's products are accumulated in the same order for
//     every M and every layout (K steps of 64, two MFMA k-slices of 32
//     each), so token chunking and the layout never change a value.
// ---------------------------------------------------------------------------
namespace nt {

constexpr int BM = 256, BK = 64;              // BK: the K step of the layouts with
                                              // row-contiguous operands
constexpr int NW = 8, NT = NW * 64;           // two groups of four waves
constexpr int MF = 16;
typedef short i16x8 __attribute__((ext_vector_type(8)));

// Tile configurations.  Every one sums an output element's products in the
// same order (32-wide k-slices in ascending k, one 16x16x32 MFMA each, K
// steps of 64 or 32 holding two or one of them), so they give the same bits
// and may be mixed freely, e.g. across token chunks.
template <int BN_, int WGM_, int WGN_, int STAGES_, int GROUP_, int BK_ = 64, bool SPLIT_ = false>
struct Cfg {
    static constexpr int BN = BN_, WGM = WGM_, WGN = WGN_, STAGES = STAGES_, GROUP = GROUP_;
    static constexpr int BK = BK_, KS = BK_ / 32;   // K step, MFMA k-slices per step
    // SPLIT: separate rings, three stages of A and two of B, each filled by
    // one group of waves (see the kernel); STAGES is then unused
    static constexpr bool SPLIT = SPLIT_;
    static constexpr int RA = 3, RB = 2;
    static_assert(WGM * WGN == NW, "eight waves");
    static_assert(STAGES >= 2 && STAGES <= 4, "two to four LDS stages");
    static_assert(BK == 64 || BK == 32, "K steps of 64 or 32");
    static constexpr int WM = BM / WGM, WN = BN / WGN;
    static constexpr int FM = WM / MF, FN = WN / MF;
    static_assert(FM * MF == WM && FN * MF == WN, "wave tile of whole MFMA tiles");
    static constexpr int A_EL = BM * BK, STAGE = (BM + BN) * BK, B_EL = BN * BK;
    static constexpr int LDS_EL = SPLIT ? RA * A_EL + RB * B_EL : STAGES * STAGE;
};
// 256 x 160: three stages (156 KB of LDS); waves of 64 x 80; the 32 tiles an
// XCD runs at once form a 4 x 8 block (4*256 + 8*160 rows per K step, L2 hit
// rate 81% against 74% for 8 x 4)
using Tile160 = Cfg<160, 4, 2, 3, 4>;
// 256 x 256: two stages (128 KB); waves of 128 x 64; 30% fewer copied bytes
// per FLOP than 256 x 160, but 62.5% of its tile count per launch.  Used when
// both operands are row-contiguous (split rings would need more than 256
// registers there); with two shared stages group B's copies must land
// within the phase that issues them, which Tile256S avoids.
using Tile256 = Cfg<256, 2, 4, 2, 8>;
// 256 x 320 in K steps of 32: four stages (144 KB); waves of 128 x 80; 36 KB
// copied per step for the 40 MFMAs each wave issues, against 52 KB for
// 256 x 160 in steps of 64 (k-contiguous operands only)
using Tile320 = Cfg<320, 2, 4, 4, 4, 32>;
// 256 x 256 in K steps of 64 with split rings (160 KB): group B copies A into
// a three-stage ring and group A copies B into a two-stage ring, so every
// copy has at least two phases to land.
// Measured in the benchmark step against Tile256: every 256 x 256 product
// 10-13% faster (20480 x 10240 x 4096: 1523 -> 1344 us).  The 32 tiles an
// XCD runs at once form a block of 4 row tiles x 8 column tiles (against 8 x
// 4: the dominant fp32 products 1.2-1.7% faster, the step 0.4-0.7%, three
// same-box pairs on each of two boxes).
using Tile256S = Cfg<256, 2, 4, 2, 4, 64, true>;

// Chunk swizzle of a k-contiguous LDS row.  Rows of 8 chunks (K step 64):
// r & 6; rows of 4 chunks (K step 32, two rows per 128 bytes): (r >> 2) & 3.
// Both give the 16 lanes of each ds_read_b128 service group distinct bank
// quads under the measured lane grouping.
template <int BK_>
__device__ __forceinline__ int swz(int r) {
    if constexpr (BK_ == 64) return r & 6;
    else return (r >> 2) & 3;
}

// One operand tile: ROWS rows of a [rows][ld] matrix contiguous along k.
template <int ROWS, int BK_, int NI = NW>
struct Copy {
    static constexpr int CPR = BK_ / 8;            // 16-byte chunks per LDS row
    static constexpr int RPI = 64 / CPR;           // rows per copy instruction
    static constexpr int WI = ROWS / RPI;          // copy instructions per stage
    static constexpr int PER = (WI + NI - 1) / NI; // per issuing wave (some one fewer)
    static_assert(ROWS % RPI == 0, "rows per copy instruction");
    u32x4 rs;
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
        rs = rsrc_words(base + row0 * ld, vr * ld * 2);
        const int r = lane / CPR;
        const int c = (lane % CPR) ^ swz<BK_>(r);
        kc = c * 8;
        vlane = (uint32_t)((r * ld + c * 8) * 2);
        ins_stride = (uint32_t)(RPI * ld * 2);
        nmine = 0;
#pragma unroll
        for (int i = 0; i < PER; ++i)
            if (wave + NI * i < WI) nmine = i + 1;
    }
    // Copy of the K step at k0 into LDS stage `dst` (k past K reads zeros);
    // `wave` is this wave's index among the NI issuing waves.
    __device__ __forceinline__ void issue(uint16_t* dst, int64_t k0, int wave) const {
        const bool tail = k0 + BK_ > K;
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int ins = wave + NI * i;
            if (PER * NI != WI && ins >= WI) break;   // wave-uniform
            uint32_t off = vlane + (uint32_t)ins * ins_stride;
            if (tail && k0 + kc >= K) off = kOob;
            lds_dma16(rs, dst + (size_t)ins * 64 * 8, off, (uint32_t)(k0 * 2));
        }
    }
};

// 16x16x32 fragment: lane holds row r0 + lane%16, k = ks*32 + 8*(lane/16) + 0..7.
template <int BK_>
__device__ __forceinline__ bf16x8 frag(const uint16_t* src, int r0, int ks, int lane) {
    const int r = r0 + (lane & 15);
    const int c = (ks * 4 + (lane >> 4)) ^ swz<BK_>(r);
    return *reinterpret_cast<const bf16x8*>(src + r * BK_ + c * 8);
}

// One operand tile stored [k][ROWS]: BK rows of a [K][ld] matrix that is
// contiguous along M or N (X in dW, W in the forward, dY in dW), copied
// 16 bytes (8 columns) per lane.  Each k row holds CPK chunks of 16 bytes;
// chunk c of row k sits at position tpos(k, c), so that the transposing
// fragment reads below touch 16 distinct bank quads per 32-lane half (the
// LDS serves lanes 0-31 and 32-63 of a 64-bit read separately).  Slot p of
// a stage (row p / CPK, position p % CPK) is filled by lane p % 64 of copy
// instruction p / 64, which fetches the chunk that belongs there.
template <int ROWS>
__device__ __forceinline__ int tpos(int k, int c) {
    if constexpr (ROWS == 160) return (c + 2 * ((k >> 3) & 1)) % 20;   // rotation by 0 / 2
    else return c ^ (2 * (k & 3) + 8 * ((k >> 3) & 1));                // XOR, 32 chunks
}
template <int ROWS>
__device__ __forceinline__ int tchunk(int k, int pos) {   // inverse of tpos
    if constexpr (ROWS == 160) return (pos + 20 - 2 * ((k >> 3) & 1)) % 20;
    else return pos ^ (2 * (k & 3) + 8 * ((k >> 3) & 1));
}

template <int ROWS, int NI = NW>
struct CopyT {
    static_assert(ROWS == 160 || ROWS == 256, "tile widths with a conflict-free layout");
    static constexpr int CPK = ROWS / 8;            // 16-byte chunks per k row
    static constexpr int WI = BK * CPK / 64;        // copy instructions per stage
    static constexpr int PER = (WI + NI - 1) / NI;  // per issuing wave (some one fewer)
    static_assert(BK * CPK % 64 == 0, "whole copy instructions");
    const uint16_t* base;   // element (k = 0, column col0)
    int64_t ld, K;
    uint32_t voff[PER];     // this lane's byte offset in each of its instructions
    int nmine;

    __device__ __forceinline__ void init(const uint16_t* base_, int64_t ld_, int64_t col0,
                                         int64_t cols, int64_t K_, int wave, int lane) {
        base = base_ + col0;
        ld = ld_;
        K = K_;
        nmine = 0;
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int ins = wave + NI * i;
            const int p = ins * 64 + lane;
            const int k = p / CPK;
            const int c = tchunk<ROWS>(k, p % CPK);
            voff[i] = (col0 + 8 * c < cols) ? (uint32_t)((k * ld + 8 * c) * 2) : kOob;
            if (ins < WI) nmine = i + 1;
        }
    }
    // Copy of the K step at k0 into LDS stage `dst` (rows past K read zeros);
    // `wave` is this wave's index among the NI issuing waves.
    __device__ __forceinline__ void issue(uint16_t* dst, int64_t k0, int wave) const {
        const int64_t left = K - k0;
        const int64_t vk = left < 0 ? 0 : (left < BK ? left : BK);
        const u32x4 rs = rsrc_words(base + k0 * ld, vk * ld * 2);
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int ins = wave + NI * i;
            if (PER * NI != WI && ins >= WI) break;   // wave-uniform
            lds_dma16(rs, dst + (size_t)ins * 64 * 8, voff[i], 0u);
        }
    }
};

// 16x16x32 fragment of a [k][ROWS] tile: lane holds column r0 + lane%16,
// k = ks*32 + 8*(lane/16) + 0..7, from two transposing reads (within each
// 16-lane group, lane j names 4 consecutive columns of row k + j/4 and
// receives column j's 4 values).
template <int ROWS>
__device__ __forceinline__ bf16x8 frag_t(const uint16_t* src, int r0, int ks, int lane) {
    const int g = lane >> 4, j = lane & 15;
    const int mn = r0 + 4 * (j & 3);
    const int k = ks * 32 + 8 * g + (j >> 2);       // k and k + 4 share tpos
    const uint16_t* p0 = src + k * ROWS + tpos<ROWS>(k, mn >> 3) * 8 + (mn & 7);
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p0);
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p0 + 4 * ROWS));
    const i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}

// Operand copy and fragment read for a tile contiguous along k (KC) or
// along its rows.
template <int ROWS, bool KC, int BK_, int NI = NW>
using OpCopy = typename std::conditional<KC, Copy<ROWS, BK_, NI>, CopyT<ROWS, NI>>::type;
template <int ROWS, bool KC, int BK_>
__device__ __forceinline__ bf16x8 op_frag(const uint16_t* src, int r0, int ks, int lane) {
    if constexpr (KC) return frag<BK_>(src, r0, ks, lane);
    else return frag_t<ROWS>(src, r0, ks, lane);
}

__device__ __forceinline__ void barrier() {
    // a bare s_barrier: __syncthreads() would also wait for every copy in
    // flight (vmcnt(0)), which defeats the three-stage ring
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_barrier" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

}  // namespace nt

template <class C, bool A_K, bool B_K, int EPI, bool OUT_BF16>
__global__ __launch_bounds__(nt::NT, 1) void gemm_nt_kernel(KArgs a) {
    using namespace nt;
    constexpr int BN = C::BN, WGN = C::WGN, STAGES = C::STAGES, BK = C::BK, KS = C::KS;
    static_assert((A_K && B_K) || BK == nt::BK, "row-contiguous operands use K steps of 64");
    constexpr int WM = C::WM, WN = C::WN, FM = C::FM, FN = C::FN;
    constexpr int A_EL = C::A_EL, STAGE = C::STAGE;
    __shared__ __attribute__((aligned(1024))) uint16_t smem[C::LDS_EL];
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

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int nk = (int)((kn + BK - 1) / BK);
    if constexpr (C::SPLIT) {
        // Split rings.  Group A (waves 0-3) copies the B tile of step p+1 in
        // its memory phase of step p into the two-stage B ring; group B
        // (waves 4-7) copies the A tile of step p+2 in its memory phase of
        // step p into the three-stage A ring.  The slots written are those of
        // step p-1, which both groups have read by then.  Group A waits for
        // its copies at the end of its compute phase (two phases after
        // issue), group B for those of step p+1 at the end of its memory
        // phase (three phases after issue), so that no copy must land within
        // the phase it was issued in.  Each wave issues 8 copy instructions
        // per step, as in the shared ring.
        constexpr int B_EL = C::B_EL, RA = C::RA, RB = C::RB;
        uint16_t* ringA = smem;
        uint16_t* ringB = smem + RA * A_EL;
        using CA = OpCopy<BM, A_K, BK, 4>;
        using CB = OpCopy<BN, B_K, BK, 4>;
        static_assert(CA::PER * 4 == CA::WI && CB::PER * 4 == CB::WI, "equal shares");
        constexpr int LA = CA::PER;   // copy instructions per step, group B
        const int w4 = wave & 3;
        const uint16_t* baseA = a.A + (A_K ? kb : kb * a.lda);
        const uint16_t* baseB = a.B + (B_K ? kb : kb * a.ldb);
        // ca copies A (group B), cb copies B (group A)
        auto mainloop = [&](const auto& ca, const auto& cb) {
            if (nk <= 0) return;   // (uniform) every wave runs the same number of barriers
            if (grpB) {
                ca.issue(ringA, 0, w4);
                if (nk > 1) ca.issue(ringA + A_EL, BK, w4);
                if (nk > 1) wait_vmcnt<LA>();   // step 0 landed, step 1 may fly
                else wait_vmcnt<0>();
            } else {
                cb.issue(ringB, 0, w4);
                wait_vmcnt<0>();
            }
            barrier();               // step 0 visible to every wave
            if (grpB) barrier();     // group B starts one phase late

            bf16x8 fa[KS][FM], fb[KS][FN];
            for (int p = 0; p < nk; ++p) {
                const uint16_t* sa = ringA + (p % RA) * A_EL;
                const uint16_t* sb = ringB + (p % RB) * B_EL;
                const bool ahead = p + 2 < nk;
                if (!grpB) {
                    if (p + 1 < nk) cb.issue(ringB + ((p + 1) % RB) * B_EL, (int64_t)(p + 1) * BK, w4);
                } else if (ahead) {
                    ca.issue(ringA + ((p + 2) % RA) * A_EL, (int64_t)(p + 2) * BK, w4);
                }
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
                    for (int i = 0; i < FM; ++i)
                        fa[ks][i] = op_frag<BM, A_K, BK>(sa, wm * WM + i * MF, ks, lane);
#pragma unroll
                    for (int j = 0; j < FN; ++j)
                        fb[ks][j] = op_frag<BN, B_K, BK>(sb, wn * WN + j * MF, ks, lane);
                }
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
                // group B: its copies of step p+1 have landed (those of p+2 may fly)
                if (grpB) {
                    if (ahead) wait_vmcnt<LA>();
                    else wait_vmcnt<0>();
                }
                barrier();
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
#pragma unroll
                    for (int i = 0; i < FM; ++i)
#pragma unroll
                        for (int j = 0; j < FN; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                fb[ks][j], fa[ks][i], acc[i][j], 0, 0, 0);
                // group A: its copies of step p+1 have landed
                if (!grpB) wait_vmcnt<0>();
                if (!(grpB && p == nk - 1)) barrier();
            }
            wait_vmcnt<0>();
        };
        if constexpr (std::is_same<CA, CB>::value) {
            // one copier per wave, its operand picked by a uniform select
            // (the resources stay scalar and one set of offsets is held)
            CA c;
            c.init(grpB ? baseA : baseB, grpB ? a.lda : a.ldb, grpB ? m0 : n0, grpB ? a.M : a.N,
                   kn, w4, lane);
            mainloop(c, c);
        } else {
            // both initialised by every wave, so the resources stay scalar
            CA ca;
            CB cb;
            ca.init(baseA, a.lda, m0, a.M, kn, w4, lane);
            cb.init(baseB, a.ldb, n0, a.N, kn, w4, lane);
            mainloop(ca, cb);
        }
    } else {
        // split k offset: along a row (k-contiguous operand) or down the rows
        OpCopy<BM, A_K, BK> ca;
        OpCopy<BN, B_K, BK> cb;
        ca.init(a.A + (A_K ? kb : kb * a.lda), a.lda, m0, a.M, kn, wave, lane);
        cb.init(a.B + (B_K ? kb : kb * a.ldb), a.ldb, n0, a.N, kn, wave, lane);
        constexpr int LA = OpCopy<BM, A_K, BK>::PER, LB = OpCopy<BN, B_K, BK>::PER;
        const int loads = ca.nmine + cb.nmine;   // copy instructions per step (wave-uniform)


        auto issue_step = [&](int q) {
            uint16_t* dst = smem + (q % STAGES) * STAGE;
            ca.issue(dst, (int64_t)q * BK, wave);
            cb.issue(dst + A_EL, (int64_t)q * BK, wave);
        };
        // wait until this wave's copies are complete except those of the newest
        // `keep` steps (0, 1, 2); copies complete in issue order
        auto wait_copies = [&](int keep) {
            if (keep <= 0) { wait_vmcnt<0>(); return; }
            if (keep == 1) {
                if (loads == LA + LB) wait_vmcnt<LA + LB>();
                else if (loads == LA + LB - 1) wait_vmcnt<LA + LB - 1>();
                else wait_vmcnt<LA + LB - 2>();
                return;
            }
            if (loads == LA + LB) wait_vmcnt<2 * (LA + LB)>();
            else if (loads == LA + LB - 1) wait_vmcnt<2 * (LA + LB - 1)>();
            else wait_vmcnt<2 * (LA + LB - 2)>();
        };

        if (nk > 0) {   // (uniform) every wave runs the same number of barriers
            for (int q = 0; q < STAGES - 1 && q < nk; ++q) issue_step(q);
            // step 0 landed; the later prologue steps may stay in flight
            wait_copies(min(STAGES - 2, nk - 1));
            barrier();               // step 0 visible to every wave
            if (grpB) barrier();     // group B starts one phase late

            bf16x8 fa[KS][FM], fb[KS][FN];
            for (int p = 0; p < nk; ++p) {
                // memory phase: copy step p+STAGES-1 into the stage step p-1 used
                // (both groups finished reading it before this phase), read step p
                const uint16_t* sa = smem + (p % STAGES) * STAGE;
                const uint16_t* sb = sa + A_EL;
                if (p + STAGES - 1 < nk) issue_step(p + STAGES - 1);
                // the copies of steps p+2 .. p+STAGES-1 may stay in flight below
                const int more = min(STAGES - 2, nk - 2 - p);
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
                    for (int i = 0; i < FM; ++i)
                        fa[ks][i] = op_frag<BM, A_K, BK>(sa, wm * WM + i * MF, ks, lane);
#pragma unroll
                    for (int j = 0; j < FN; ++j)
                        fb[ks][j] = op_frag<BN, B_K, BK>(sb, wn * WN + j * MF, ks, lane);
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
    a.nparts = p.nparts > 1 ? p.nparts : 1;
    a.own = p.own;
    for (int j = 0; j < kMaxFusedParts; ++j) a.peers[j] = p.peers[j];
    a.ldp = p.ldp;
    return a;
}

// Products with both operands row-contiguous (TN: dW on the path without a
// workspace): 256 x 256 tiles (30% fewer copied bytes per FLOP) when their
// last wave of 256 concurrent tiles is at least 90% full, 256 x 160 otherwise.
bool fills_waves(const GemmProblem& p, int64_t bn) {
    constexpr int64_t kCUs = 256;
    const int64_t tiles = ((p.M + nt::BM - 1) / nt::BM) * ((p.N + bn - 1) / bn);
    const int64_t waves = (tiles + kCUs - 1) / kCUs;
    return tiles * 10 >= waves * kCUs * 9;
}

bool nt_use_256(const GemmProblem& p) { return fills_waves(p, 256); }

// Buffer offsets are 32-bit and a resource covers at most 0x7fffff00 bytes:
// the rows one tile copies from an operand contiguous along k (BM rows of A,
// BN rows of B) must span less than that.
constexpr int64_t kMaxSpan = 0x7fffff00;
bool rows_fit(int64_t rows, int64_t ld) { return rows * ld * 2 <= kMaxSpan; }

// Tile configuration of an unsplit product with both operands contiguous
// along k: the one with the least modelled time, (waves of 256 concurrent
// tiles) x (tile width / relative per-CU rate), where a last wave that is a
// fraction f full costs 0.5 + 0.5 f of a full one (its tiles share L2 and
// HBM with fewer others).  Relative rates measured on the block's products
// with every CU busy: 256 x 160 0.8, 256 x 320 (K steps of 32) 0.9,
// 256 x 256 with split rings 1.0.  The 256 x 256 tiles are preferred within
// 5%: they leave CUs to the reductions that run beside a one-wave product.
enum NtCfg { NT_160, NT_256S, NT_320 };

double nt_cost(const GemmProblem& p, int64_t bn, double rate) {
    constexpr int64_t kCUs = 256;
    const int64_t tiles = ((p.M + nt::BM - 1) / nt::BM) * ((p.N + bn - 1) / bn);
    const int64_t full = tiles / kCUs, rest = tiles % kCUs;
    const double waves = (double)full + (rest ? 0.5 + 0.5 * (double)rest / kCUs : 0.0);
    return waves * (double)bn / rate;
}

NtCfg nt_pick(const GemmProblem& p, bool allow320) {
    const double c160 = nt_cost(p, 160, 0.8), c256 = nt_cost(p, 256, 1.0);
    const double c320 = allow320 && rows_fit(320, p.ldb) ? nt_cost(p, 320, 0.9) : 1e300;
    const double other = c160 < c320 ? c160 : c320;
    if (c256 <= 1.05 * other) return NT_256S;
    return c160 <= c320 ? NT_160 : NT_320;
}

bool nt_kcontig(const GemmProblem& p) { return p.layout == LAYOUT_NT && p.splits <= 1; }

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

template <class C, bool A_K, bool B_K, int EPI, bool OUT_BF16>
hipError_t launch_pp_cfg(const GemmProblem& p, hipStream_t s) {
    const KArgs a = kargs(p, nt::BM, C::BN);
    const int grid = a.tiles_m * a.tiles_n * a.splits;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL((gemm_nt_kernel<C, A_K, B_K, EPI, OUT_BF16>), dim3(grid), dim3(nt::NT), 0,
                       s, a);
    return hipGetLastError();
}

// The ping-pong kernel for operands contiguous along k (A_K / B_K) or along
// their rows; split-K launches use the 256 x 160 configuration.
template <bool A_K, bool B_K, int EPI, bool OUT_BF16>
hipError_t launch_pp(const GemmProblem& p, hipStream_t s) {
    if (p.splits > 1) return launch_pp_cfg<nt::Tile160, A_K, B_K, EPI, OUT_BF16>(p, s);
    if constexpr (A_K && B_K) {
        switch (nt_pick(p, true)) {
        case NT_256S: return launch_pp_cfg<nt::Tile256S, A_K, B_K, EPI, OUT_BF16>(p, s);
        case NT_320: return launch_pp_cfg<nt::Tile320, A_K, B_K, EPI, OUT_BF16>(p, s);
        default: return launch_pp_cfg<nt::Tile160, A_K, B_K, EPI, OUT_BF16>(p, s);
        }
    } else if constexpr (!A_K && !B_K) {
        // both operands row-contiguous: split rings would need more than 256
        // registers per lane (the transposing fragment reads' addresses)
        return nt_use_256(p) ? launch_pp_cfg<nt::Tile256, A_K, B_K, EPI, OUT_BF16>(p, s)
                             : launch_pp_cfg<nt::Tile160, A_K, B_K, EPI, OUT_BF16>(p, s);
    } else {
        // A contiguous along k, B along its rows (the forward from W as
        // given): the same model without the 256 x 320 tiles (k-contiguous
        // only)
        return nt_pick(p, false) == NT_256S
                   ? launch_pp_cfg<nt::Tile256S, A_K, B_K, EPI, OUT_BF16>(p, s)
                   : launch_pp_cfg<nt::Tile160, A_K, B_K, EPI, OUT_BF16>(p, s);
    }
}

}  // namespace

bool gemm_supported(int layout, int epi, bool out_bf16) {
    switch (layout) {
    case LAYOUT_NN:
        return epi == EPI_NONE || epi == EPI_BIAS || epi == EPI_BIAS_GELU ||
               (out_bf16 && epi == EPI_GELU_BWD);
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
    static const char* const names[3][3] = {{"gemm_nn", "gemm_nn256", "gemm_nn_splitk"},
                                            {"gemm_nt", "gemm_nt256", "gemm_nt_splitk"},
                                            {"gemm_tn", "gemm_tn256", "gemm_tn_splitk"}};
    const int l = p.layout == LAYOUT_NN ? 0 : p.layout == LAYOUT_NT ? 1 : p.layout == LAYOUT_TN ? 2 : -1;
    if (l < 0) return "gemm_?";
    if (nt_kcontig(p)) {
        const NtCfg c = nt_pick(p, true);
        return c == NT_320 ? "gemm_nt320" : c == NT_256S ? "gemm_nt256" : "gemm_nt";
    }
    if (p.layout == LAYOUT_NN && p.splits <= 1)
        return nt_pick(p, false) == NT_256S ? "gemm_nn256" : "gemm_nn";
    return names[l][p.splits > 1 ? 2 : nt_use_256(p) ? 1 : 0];
}

bool nn_streams_like_nt(int64_t M, int64_t N) {
    GemmProblem p;
    p.layout = LAYOUT_NN;
    p.M = M;
    p.N = N;
    return nt_pick(p, false) == NT_256S;
}

int nt_split_plan(int64_t M, int64_t N, int64_t K, int64_t* ksplit) {
    return pick_splits(M, N, K, ksplit);
}

hipError_t launch_gemm(const GemmProblem& p, hipStream_t s) {
    if (p.M <= 0 || p.N <= 0) return hipSuccess;
    // buffer offsets are 32-bit: one tile's rows of either operand must span
    // < 2 GiB (256 rows covers the 160- and 256-wide tiles and the 64 k rows
    // of a row-contiguous operand; nt_pick checks the 320 rows itself)
    if (!rows_fit(256, p.lda) || !rows_fit(256, p.ldb)) return hipErrorInvalidValue;
    const bool b16 = p.out_bf16;
    if (p.nparts > kMaxFusedParts || (p.nparts > 1 && (p.splits > 1 || p.own < 0 ||
                                                       p.own >= p.nparts || p.ldp % 4)))
        return hipErrorInvalidValue;
    if (p.splits > 1) {
        // split-K: plain fp32 outputs, whole K steps per split, every split
        // non-empty
        if (p.epi != EPI_NONE || b16 || p.ksplit <= 0 || p.ksplit % 64 ||
            (int64_t)(p.splits - 1) * p.ksplit >= p.K || p.c_split < p.M * p.ldc)
            return hipErrorInvalidValue;
    }
    switch (p.layout) {
    case LAYOUT_NN:   // X W: A contiguous along k, B = W along its columns
        switch (p.epi) {
        case EPI_NONE:
            return b16 ? launch_pp<true, false, EPI_NONE, true>(p, s)
                       : launch_pp<true, false, EPI_NONE, false>(p, s);
        case EPI_BIAS:
            return b16 ? launch_pp<true, false, EPI_BIAS, true>(p, s)
                       : launch_pp<true, false, EPI_BIAS, false>(p, s);
        case EPI_BIAS_GELU:
            return b16 ? launch_pp<true, false, EPI_BIAS_GELU, true>(p, s)
                       : launch_pp<true, false, EPI_BIAS_GELU, false>(p, s);
        case EPI_GELU_BWD:   // dY W^T with W stored [n][k], times GeLU'(pre)
            if (b16) return launch_pp<true, false, EPI_GELU_BWD, true>(p, s);
            return hipErrorInvalidValue;
        default:
            return hipErrorInvalidValue;
        }
    case LAYOUT_NT:   // dY W^T with B = W (contiguous along the contraction)
        if (p.epi == EPI_NONE)
            return b16 ? launch_pp<true, true, EPI_NONE, true>(p, s)
                       : launch_pp<true, true, EPI_NONE, false>(p, s);
        if (p.epi == EPI_GELU_BWD && b16) return launch_pp<true, true, EPI_GELU_BWD, true>(p, s);
        if (p.epi == EPI_BIAS && b16) return launch_pp<true, true, EPI_BIAS, true>(p, s);
        if (p.epi == EPI_BIAS_GELU && b16) return launch_pp<true, true, EPI_BIAS_GELU, true>(p, s);
        return hipErrorInvalidValue;
    case LAYOUT_TN:   // X^T dY: both operands contiguous along their columns
        if (p.epi == EPI_NONE && !b16) return launch_pp<false, false, EPI_NONE, false>(p, s);
        return hipErrorInvalidValue;
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace atp
