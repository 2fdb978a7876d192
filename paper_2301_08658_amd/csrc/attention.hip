// Causal attention core of one device's heads (Sec. 2.1 Formula (mha); the
// attention block of Sec. 3.2.1 scatters the heads of the reduced QKV block
// over the group that reduced it, each device attends over its run of heads,
// and the outputs are gathered before out-proj).
//
// Forward, one workgroup per (sequence, head, query tile), head dimension
// 128, keys in steps of 64 (flash-attention style: running row maximum and
// sum, the output rescaled as they grow).  Large grids: 128-row tiles, four
// waves of two 16-row blocks.  Small grids: 64-row tiles, two groups of four
// waves of 16 rows that split the tile's keys and merge at the end.
//
//   * S = Q K^T on v_mfma_f32_16x16x32_bf16: Q fragments stay in registers
//     for the whole row tile; K fragments are ds_read_b128 from a [key][d]
//     LDS tile whose 16-byte chunks are XOR-swizzled by key (c ^ (n & 15)),
//     which puts the 16 lanes of each gfx950 read group on distinct banks.
//   * A lane holds S(m = lane % 16, n = 16 j + 4 (lane / 16) + e): the rows
//     are lane-uniform, so the row maximum and sum need only two lane
//     exchanges (lane swaps of 16 and 32).
//   * O += P V: the MFMA sums over its 32 keys in any order as long as both
//     operands agree, so each 32-key slice takes the keys {4g + e} and
//     {16 + 4g + e} for lane group g: then P's fragment is the lane's own
//     eight probabilities (two S tiles, no exchange), and V's fragment is two
//     ds_read_b64_tr_b16 from a [key][d] tile (chunk c at c ^ (2 (n & 3) +
//     8 ((n >> 2) & 1)), distinct banks per 32-lane half).
//   * Exponentials in base 2 (scores scaled by log2(e) / sqrt(128)); the
//     log-sum-exp of each row is saved (natural log) for the backward.
//
// Backward (the gradient of softmax(S) V, S = Q K^T / sqrt(d)): with P
// recomputed from the saved log-sum-exps and delta_t = dO_t . O_t,
//   dV = P^T dO,  dS = P o (dO V^T - delta),  dQ = dS K / sqrt(d),
//   dK = dS^T Q / sqrt(d).
// One kernel per 64-query tile (128 on large grids) first forms delta for
// its rows (stored for the next kernel) and accumulates dQ over its key
// tiles; then one per 64-key tile accumulates dK and dV over the query
// tiles that see it; no atomics, so the result does not depend on
// scheduling.  Every contraction
// over keys or queries uses the same lane-local ordering as the forward's
// P V, so probabilities and score gradients never leave their lanes.  All
// bwd LDS tiles use the layout vpos, which is conflict-free for both
// ds_read_b128 fragments and the transposing reads.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"
#include "lds_dma.h"

namespace atp {
namespace {

constexpr int D = 128;          // head dimension
constexpr int BM = 64;          // query rows per workgroup
constexpr int BN = 64;          // keys per step
constexpr int NWAVE = 4;
constexpr int NTHR = NWAVE * 64;
constexpr int64_t kFwdWideGrid = 512;   // two workgroups per CU on 256 CUs
constexpr int64_t kBwdSplitGrid = 1024;  // 64-row tiles below which loops are split
// forward softmax: largest base-2 gain of a row maximum absorbed without
// rescaling the running output (weights stay below 2^8, exact in bf16's range)
constexpr float kSlack = 8.f;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

__device__ __forceinline__ int kpos(int n, int c) { return c ^ (n & 15); }
__device__ __forceinline__ int vpos(int n, int c) { return c ^ (2 * (n & 3) + 8 * ((n >> 2) & 1)); }

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// The four lanes l, l ^ 16, l ^ 32, l ^ 48 hold one score row's columns.
// Their maximum and sum come from gfx950's lane swaps (v_permlane16_swap
// pairs the 16-lane rows 0-1 and 2-3, v_permlane32_swap the two halves),
// which stay in the VALU instead of a round trip through LDS.  With both
// operands x, the first result is the lower member of each pair and the
// second the upper, so every lane of the four combines the same values in
// the same order: (r0 op r1) op (r2 op r3), bit-identical in all four.
__device__ __forceinline__ float row_max4(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x),
                                                    false, false);
    x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                    false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Maximum of a lane's 16 scores of one row block as a shallow tree: five
// independent three-input maxima over 15 scores, two more over those and
// the last score, and one two-input maximum (three dependent steps instead
// of a chain through all sixteen).
__device__ __forceinline__ float max16(const f32x4 (&v)[4]) {
    const float a = fmaxf(fmaxf(v[0][0], v[0][1]), v[0][2]);
    const float b = fmaxf(fmaxf(v[0][3], v[1][0]), v[1][1]);
    const float c = fmaxf(fmaxf(v[1][2], v[1][3]), v[2][0]);
    const float d = fmaxf(fmaxf(v[2][1], v[2][2]), v[2][3]);
    const float e = fmaxf(fmaxf(v[3][0], v[3][1]), v[3][2]);
    return fmaxf(fmaxf(fmaxf(a, b), c), fmaxf(fmaxf(d, e), v[3][3]));
}

__device__ __forceinline__ float row_sum4(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x),
                                                    false, false);
    x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                    false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Two floats to bf16 (round to nearest even: one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    const f32x2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Element offsets of a lane's transposing reads of a [key][d] tile in the
// vpos layout, rows 4 g + lane%16 / 4 (+ 32 sl, + 16 for the second read:
// same swizzle), columns 16 dt + 4 (lane % 4): one per dt.
__device__ __forceinline__ int tr_offset(int lane, int dt) {
    const int g = lane >> 4, j16 = lane & 15;
    const int r = 4 * g + (j16 >> 2);
    const int col = 16 * dt + 4 * (j16 & 3);
    return r * D + vpos(r, col >> 3) * 8 + (col & 7);
}

struct AttnArgs {
    const uint16_t* qkv;   // [T][ldq]; the device's first head at column col0
    int64_t ldq, col0;
    uint16_t* out;         // [T][ldo]; the device's first head at column ocol0
    int64_t ldo, ocol0;
    float* lse;            // [heads][T], natural log
    int batch, seq, heads, qtiles;
    float scale_log2;      // log2(e) / sqrt(D)
};



// Rows [n0, n0 + 64) of two 128-column runs of one sequence's token rows
// straight into two LDS tiles (the first in the kpos layout when KPOS0,
// else vpos; the second in vpos): copy instruction i (wave w issues
// i = w + 4 r) fills slots 64 i .. 64 i + 63, i.e. row 4 w + 16 r + lane/16,
// position lane % 16, so the lane fetches the chunk its slot holds (kpos and
// vpos are XORs, their own inverses, and depend only on the row's low four
// bits).  Rows past the sequence are past the range and read zeros.
template <bool KPOS0>
struct TileDma2 {
    uint32_t off0, off1, st0, st1;   // lane offsets of r = 0, bytes per 16 rows
    __device__ __forceinline__ void init(int64_t ld0, int64_t ld1, int wave, int lane) {
        const int n = 4 * wave + lane / 16, pos = lane % 16;
        const int c0 = KPOS0 ? kpos(n, pos) : vpos(n, pos);
        off0 = (uint32_t)((n * ld0 + 8 * c0) * 2);
        off1 = (uint32_t)((n * ld1 + 8 * vpos(n, pos)) * 2);
        st0 = (uint32_t)(16 * ld0 * 2);
        st1 = (uint32_t)(16 * ld1 * 2);
    }
    __device__ __forceinline__ void issue(const uint16_t* b0, int64_t ld0, const uint16_t* b1,
                                          int64_t ld1, int64_t tok0, int n0, int seq, uint16_t* t0,
                                          uint16_t* t1, int wave) const {
        const int64_t left = seq - n0;
        const int64_t vr = left < 0 ? 0 : (left < 64 ? left : 64);
        const dma::u32x4 r0 = dma::rsrc_words(b0 + (tok0 + n0) * ld0, vr * ld0 * 2);
        const dma::u32x4 r1 = dma::rsrc_words(b1 + (tok0 + n0) * ld1, vr * ld1 * 2);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int ins = wave + NWAVE * r;
            dma::lds_dma16(r0, t0 + ins * 64 * 8, off0 + r * st0, 0u);
            dma::lds_dma16(r1, t1 + ins * 64 * 8, off1 + r * st1, 0u);
        }
    }
};

// RB row blocks of 16 queries per wave (query tile of 64 RB rows): every K
// and V fragment read from LDS feeds RB MFMAs.  Block r of wave w holds rows
// 64 r + 16 w .. + 15 of the tile.  KG groups of four waves split the tile's
// key tiles between them (group 0 the first half, group 1 the rest, which
// holds the diagonal): each group keeps its own running maximum, sum and
// output for the same rows, and group 1 hands them to group 0 through LDS at
// the end, so no row loop is longer than half the causal row.
template <int RB, int KG>
__global__ __launch_bounds__(NTHR * KG, 2 / KG) void attention_fwd_kernel(AttnArgs a) {
    constexpr int QT = 64 * RB;   // query rows per workgroup
    __shared__ __attribute__((aligned(16))) uint16_t kv[KG][2][2][BN * D];   // [group][buf][K|V]
    __shared__ float mls[KG > 1 ? NWAVE * RB * 2 * 64 : 1];                // group 1's m, l
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int grp = wv / NWAVE, wave = wv % NWAVE;
    // longest rows first: the last query tile of every (sequence, head) leads
    const int per = a.qtiles;
    const int bid = blockIdx.x;
    const int qt = per - 1 - bid / (a.batch * a.heads);
    const int bh = bid % (a.batch * a.heads);
    const int b = bh / a.heads, hh = bh % a.heads;
    const int64_t tok0 = (int64_t)b * a.seq;
    const int64_t qc = a.col0 + (int64_t)hh * 3 * D, kc = qc + D, vc = qc + 2 * D;

    // Q fragments: row mrow[r], d = 32 ks + 8 (lane / 16) + 0..7
    int mrow[RB];
    bf16x8 qf[RB][4];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        mrow[r] = qt * QT + 64 * r + wave * 16 + (lane & 15);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            if (mrow[r] < a.seq)
                qf[r][ks] = *reinterpret_cast<const bf16x8*>(
                    a.qkv + (tok0 + mrow[r]) * a.ldq + qc + 32 * ks + 8 * (lane >> 4));
            else
                qf[r][ks] = __builtin_bit_cast(bf16x8, u32x4{0, 0, 0, 0});
        }
    }

    f32x4 o[RB][8];
    float mrun[RB], lrun[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) o[r][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
        mrun[r] = -INFINITY;
        lrun[r] = 0.f;
    }

    // causal: keys up to the tile's last row inside the sequence; group 0
    // takes key tiles [0, half), group 1 [half, nkt)
    const int last = min(qt * QT + QT, a.seq) - 1;
    const int nkt = last / BN + 1;
    const int half = KG > 1 ? (nkt + 1) / 2 : nkt;
    const int kt0 = grp == 0 ? 0 : half;
    const int mine = grp == 0 ? half : nkt - half;   // <= half
    uint16_t(*buf)[2][BN * D] = kv[grp];
    TileDma2<true> cp;
    cp.init(a.ldq, a.ldq, wave, lane);
    const uint16_t* kbase = a.qkv + kc;
    const uint16_t* vbase = a.qkv + vc;
    if (mine > 0)
        cp.issue(kbase, a.ldq, vbase, a.ldq, tok0, kt0 * BN, a.seq, buf[0][0], buf[0][1], wave);
    dma::wait_vmcnt<0>();
    __syncthreads();
    const int g = lane >> 4, l16 = lane & 15;
    // K fragment offsets (key row 16 j + l16: j adds 16 rows), V read offsets
    int koff[4], voff[8];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) koff[ks] = l16 * D + kpos(l16, 4 * ks + g) * 8;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) voff[dt] = tr_offset(lane, dt);
    // both groups step together (one barrier per step); a group with fewer
    // key tiles idles through the last step
    for (int i = 0; i < half; ++i) {
        if (i < mine) {
            const int kt = kt0 + i;
            const uint16_t* ks_ = buf[i & 1][0];
            const uint16_t* vs_ = buf[i & 1][1];
            // the other buffer was last read in step i - 1, before its barrier
            if (i + 1 < mine)
                cp.issue(kbase, a.ldq, vbase, a.ldq, tok0, (kt + 1) * BN, a.seq,
                         buf[(i + 1) & 1][0], buf[(i + 1) & 1][1], wave);

            // S = Q K^T for RB x 16 rows x 64 keys (raw scores); the 4 RB
            // accumulators advance together over the head dimension, so
            // consecutive products are independent
            f32x4 s[RB][4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int r = 0; r < RB; ++r) s[r][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const bf16x8 kf =
                        *reinterpret_cast<const bf16x8*>(ks_ + 16 * j * D + koff[ks]);
#pragma unroll
                    for (int r = 0; r < RB; ++r)
                        s[r][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[r][ks], s[r][j],
                                                                          0, 0, 0);
                }
            // causal mask (and keys past the sequence): only key tiles that
            // reach past the tile's first row and a ragged last tile have
            // masked keys.  A block whose rows all precede the key tile gets
            // no probability mass from it (its running maximum is finite or,
            // in group 1 before its first visible key, stays -inf with zero
            // weights: exp2(-inf) = 0 and the rescale factor is taken as 1).
            if ((kt + 1) * BN > qt * QT || (kt + 1) * BN > a.seq) {
#pragma unroll
                for (int r = 0; r < RB; ++r)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int nabs = kt * BN + 16 * j + 4 * g + e;
                            if (nabs > mrow[r] || nabs >= a.seq) s[r][j][e] = -INFINITY;
                        }
            }
#pragma unroll
            for (int r = 0; r < RB; ++r) {
                float mx = max16(s[r]);
                mx = row_max4(mx);
                const float mnew = fmaxf(mrun[r], mx * a.scale_log2);   // base-2 scaled domain
                // The reference point of the exponentials moves only when a
                // row of the wave gains more than kSlack on it (one scalar
                // branch for the wave); otherwise the weights exp2(x - m) stay
                // below 2^kSlack and O and l keep their scale.  O / l and
                // m + log2 l do not depend on the reference point, so the
                // results differ from rescaling at every step by rounding only.
                if (__builtin_amdgcn_ballot_w64(mnew > mrun[r] + kSlack) != 0) {
                    // a row with no visible key yet keeps mnew = -inf: subtract 0
                    const float alpha =
                        __builtin_amdgcn_exp2f(mrun[r] - (mnew == -INFINITY ? 0.f : mnew));
                    lrun[r] *= alpha;
#pragma unroll
                    for (int dt = 0; dt < 8; ++dt) o[r][dt] *= alpha;
                    mrun[r] = mnew;
                }
                const float msub = mrun[r] == -INFINITY ? 0.f : mrun[r];
                float rs = 0.f;
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float p = __builtin_amdgcn_exp2f(
                            __builtin_fmaf(s[r][j][e], a.scale_log2, -msub));
                        s[r][j][e] = p;
                        rs += p;
                    }
                lrun[r] += row_sum4(rs);
            }

            // O += P V over two 32-key slices
#pragma unroll
            for (int sl = 0; sl < 2; ++sl) {
                bf16x8 pf[RB];
#pragma unroll
                for (int r = 0; r < RB; ++r) {
                    const u32x4 pw = {pack_bf16x2(s[r][2 * sl][0], s[r][2 * sl][1]),
                                      pack_bf16x2(s[r][2 * sl][2], s[r][2 * sl][3]),
                                      pack_bf16x2(s[r][2 * sl + 1][0], s[r][2 * sl + 1][1]),
                                      pack_bf16x2(s[r][2 * sl + 1][2], s[r][2 * sl + 1][3])};
                    pf[r] = __builtin_bit_cast(bf16x8, pw);
                }
#pragma unroll
                for (int dt = 0; dt < 8; ++dt) {
                    const uint16_t* p0 = vs_ + 32 * sl * D + voff[dt];
                    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p0);
                    const i16x4 hi =
                        __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p0 + 16 * D));
                    const i16x8 vv = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                    const bf16x8 vf = __builtin_bit_cast(bf16x8, vv);
#pragma unroll
                    for (int r = 0; r < RB; ++r)
                        o[r][dt] =
                            __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[r], o[r][dt], 0, 0, 0);
                }
            }
        }
        // this wave's copies of its next step have landed; after the barrier
        // every wave's have, and no wave reads the buffers of this step
        dma::wait_vmcnt<0>();
        __syncthreads();
    }

    if constexpr (KG > 1) {
        // group 1 -> LDS (its own K/V buffers, free now): per wave, block,
        // column tile and lane one f32x4, and per lane m and l
        f32x4* ox = reinterpret_cast<f32x4*>(&kv[1][0][0][0]);
        if (grp == 1) {
#pragma unroll
            for (int r = 0; r < RB; ++r) {
#pragma unroll
                for (int dt = 0; dt < 8; ++dt) ox[((wave * RB + r) * 8 + dt) * 64 + lane] = o[r][dt];
                mls[((wave * RB + r) * 2 + 0) * 64 + lane] = mrun[r];
                mls[((wave * RB + r) * 2 + 1) * 64 + lane] = lrun[r];
            }
        }
        __syncthreads();
        if (grp == 1) return;
#pragma unroll
        for (int r = 0; r < RB; ++r) {
            const float m1 = mls[((wave * RB + r) * 2 + 0) * 64 + lane];
            const float l1 = mls[((wave * RB + r) * 2 + 1) * 64 + lane];
            const float mn = fmaxf(mrun[r], m1);          // finite: key 0 is group 0's
            const float a0 = __builtin_amdgcn_exp2f(mrun[r] - mn);
            const float a1 = __builtin_amdgcn_exp2f(m1 - mn);   // 0 when m1 = -inf
#pragma unroll
            for (int dt = 0; dt < 8; ++dt)
                o[r][dt] = o[r][dt] * a0 + ox[((wave * RB + r) * 8 + dt) * 64 + lane] * a1;
            lrun[r] = lrun[r] * a0 + l1 * a1;
            mrun[r] = mn;
        }
    }

    // O / l as bf16: lane holds O(m = mrow, d = 16 dt + 4 g + 0..3)
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        if (mrow[r] >= a.seq) continue;
        const float inv = 1.0f / lrun[r];
        uint16_t* orow = a.out + (tok0 + mrow[r]) * a.ldo + a.ocol0 + (int64_t)hh * D;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
            const u32x2 w = {pack_bf16x2(o[r][dt][0] * inv, o[r][dt][1] * inv),
                             pack_bf16x2(o[r][dt][2] * inv, o[r][dt][3] * inv)};
            *reinterpret_cast<u32x2*>(orow + 16 * dt + 4 * g) = w;
        }
        if (g == 0)
            a.lse[(int64_t)hh * a.batch * a.seq + tok0 + mrow[r]] =
                (mrun[r] + __log2f(lrun[r])) * 0.69314718055994530942f;
    }
}

// ---------------------------------------------------------------------------
// backward
// ---------------------------------------------------------------------------
struct AttnBwdArgs {
    const uint16_t* qkv;  int64_t ldq, col0;     // device's heads at col0, [q|k|v] each
    const uint16_t* out;  int64_t ldo, ocol0;    // forward output
    const uint16_t* dout; int64_t lddo, docol0;  // its gradient
    const float* lse;                            // [heads][T], natural log
    float* delta;                                // [heads][T] scratch
    uint16_t* dqkv;       int64_t lddq, dcol0;   // gradients, [dq|dk|dv] per head
    int batch, seq, heads, tiles;
    float scale_log2, inv_sqrt_d;
};

// Lane offsets into a [row][d] tile in the vpos layout: ds_read_b128
// fragments of row 16 j + lane%16, chunk 4 ks + lane/16 (boff[ks]; j adds
// 16 rows, same swizzle), and transposing reads (toff[dt], see tr_offset).
__device__ __forceinline__ void offsets(int lane, int (&boff)[4], int (&toff)[8]) {
    const int g = lane >> 4, l16 = lane & 15;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) boff[ks] = l16 * D + vpos(l16, 4 * ks + g) * 8;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) toff[dt] = tr_offset(lane, dt);
}
// Transposing fragment at p (rows p, p + 16 D): lane (group g, j) gets
// column 16 dt + j, keys or queries rb + 4 g + 0..3 and rb + 16 + 4 g + 0..3.
__device__ __forceinline__ bf16x8 frag_tr_at(const uint16_t* p) {
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 16 * D));
    const i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}
__device__ __forceinline__ bf16x8 pack_pair(const f32x4& a, const f32x4& b) {
    const u32x4 w = {pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]), pack_bf16x2(b[0], b[1]),
                     pack_bf16x2(b[2], b[3])};
    return __builtin_bit_cast(bf16x8, w);
}


// dK, dV of one 64-key tile (4 waves x 16 keys).  KG groups of four waves
// split the query tiles that see the key tile (group 0 the first half, group
// 1 the rest); group 1 adds its sums into group 0's through LDS at the end.
template <int KG>
__global__ __launch_bounds__(NTHR * KG, 2 / KG) void attention_dkv_kernel(AttnBwdArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t qd[KG][2][2][BM * D];   // [grp][buf][Q|dO]
    __shared__ float rowv[KG][2][2][BM];                                    // [grp][buf][lse2|delta]
    const int lane = threadIdx.x & 63, g = lane >> 4;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int grp = wv / NWAVE, wave = wv % NWAVE;
    const int tid = (int)threadIdx.x % NTHR;   // thread index within the group
    const int bhn = a.batch * a.heads;
    const int kt = blockIdx.x / bhn;            // short loops (late keys) last
    const int bh = blockIdx.x % bhn;
    const int b = bh / a.heads, hh = bh % a.heads;
    const int64_t tok0 = (int64_t)b * a.seq, T = (int64_t)a.batch * a.seq;
    const int64_t qc = a.col0 + (int64_t)hh * 3 * D;
    const uint16_t* qbase = a.qkv + qc;
    const uint16_t* dobase = a.dout + a.docol0 + (int64_t)hh * D;

    const int kabs = kt * BN + wave * 16 + (lane & 15);
    bf16x8 kf[4], vf[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
        if (kabs < a.seq) {
            const uint16_t* row = a.qkv + (tok0 + kabs) * a.ldq + qc;
            kf[ks] = *reinterpret_cast<const bf16x8*>(row + D + 32 * ks + 8 * g);
            vf[ks] = *reinterpret_cast<const bf16x8*>(row + 2 * D + 32 * ks + 8 * g);
        } else {
            kf[ks] = __builtin_bit_cast(bf16x8, u32x4{0, 0, 0, 0});
            vf[ks] = kf[ks];
        }
    }
    f32x4 dk[8], dv[8];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
        dk[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
        dv[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    auto load_rows = [&](int qt, float& l2, float& dl) {
        const int t = qt * BM + tid;
        if (tid < BM && t < a.seq) {
            l2 = a.lse[(int64_t)hh * T + tok0 + t] * 1.44269504088896340736f;
            dl = a.delta[(int64_t)hh * T + tok0 + t];
        } else {
            l2 = 0.f;
            dl = 0.f;
        }
    };
    int boff[4], toff[8];
    offsets(lane, boff, toff);
    TileDma2<false> cp;
    cp.init(a.ldq, a.lddo, wave, lane);
    // query tiles kt .. tiles-1 see this key tile: group 0 the first half
    const int nsteps = a.tiles - kt;
    const int half = KG > 1 ? (nsteps + 1) / 2 : nsteps;
    const int q0 = kt + (grp == 0 ? 0 : half);
    const int mine = grp == 0 ? half : nsteps - half;   // <= half
    uint16_t(*qb)[2][BM * D] = qd[grp];
    float(*rv)[2][BM] = rowv[grp];
    float l2r = 0.f, dlr = 0.f;
    if (mine > 0) {
        cp.issue(qbase, a.ldq, dobase, a.lddo, tok0, q0 * BM, a.seq, qb[0][0], qb[0][1], wave);
        load_rows(q0, l2r, dlr);
        if (tid < BM) { rv[0][0][tid] = l2r; rv[0][1][tid] = dlr; }
    }
    dma::wait_vmcnt<0>();
    __syncthreads();
    for (int i = 0; i < half; ++i) {
        if (i < mine) {
            const int qt = q0 + i;
            const int buf = i & 1;
            const uint16_t* qs = qb[buf][0];
            const uint16_t* ds_ = qb[buf][1];
            // the other buffers were last read in step i - 1, before its barrier
            if (i + 1 < mine) {
                cp.issue(qbase, a.ldq, dobase, a.lddo, tok0, (qt + 1) * BM, a.seq, qb[buf ^ 1][0],
                         qb[buf ^ 1][1], wave);
                load_rows(qt + 1, l2r, dlr);
            }
            // S^T and dP^T: lane holds (key = kabs, query = 16 j + 4 g + e).
            // The eight accumulators of the four 16-query blocks advance
            // together over the head dimension, so consecutive products are
            // independent; P and dS then replace S and dP in place.
            const bool masked = qt == kt || (qt + 1) * BM > a.seq;
            f32x4 p[4], dsv[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                p[j] = f32x4{0.f, 0.f, 0.f, 0.f};
                dsv[j] = p[j];
            }
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    p[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        *reinterpret_cast<const bf16x8*>(qs + 16 * j * D + boff[ks]), kf[ks],
                        p[j], 0, 0, 0);
                    dsv[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        *reinterpret_cast<const bf16x8*>(ds_ + 16 * j * D + boff[ks]), vf[ks],
                        dsv[j], 0, 0, 0);
                }
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int ql = 16 * j + 4 * g + e;
                    float pv = __builtin_amdgcn_exp2f(
                        __builtin_fmaf(p[j][e], a.scale_log2, -rv[buf][0][ql]));
                    if (masked) {
                        const int qabs = qt * BM + ql;
                        if (qabs < kabs || qabs >= a.seq) pv = 0.f;
                    }
                    p[j][e] = pv;
                    dsv[j][e] = pv * (dsv[j][e] - rv[buf][1][ql]);
                }
            // dV += P^T dO, dK += dS^T Q over two 32-query slices
#pragma unroll
            for (int sl = 0; sl < 2; ++sl) {
                const bf16x8 pf = pack_pair(p[2 * sl], p[2 * sl + 1]);
                const bf16x8 sf = pack_pair(dsv[2 * sl], dsv[2 * sl + 1]);
#pragma unroll
                for (int dt = 0; dt < 8; ++dt) {
                    dv[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        frag_tr_at(ds_ + 32 * sl * D + toff[dt]), pf, dv[dt], 0, 0, 0);
                    dk[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        frag_tr_at(qs + 32 * sl * D + toff[dt]), sf, dk[dt], 0, 0, 0);
                }
            }
            if (i + 1 < mine && tid < BM) {
                rv[buf ^ 1][0][tid] = l2r;
                rv[buf ^ 1][1][tid] = dlr;
            }
        }
        // this wave's copies of its next step have landed; after the barrier
        // every wave's have, and no wave reads this step's buffers any more
        dma::wait_vmcnt<0>();
        __syncthreads();
    }
    if constexpr (KG > 1) {
        // group 1's sums -> LDS (its own Q/dO buffers, free now), added by
        // group 0 in a fixed order: group 0's + group 1's
        f32x4* x = reinterpret_cast<f32x4*>(&qd[1][0][0][0]);
        if (grp == 1) {
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) {
                x[((wave * 2 + 0) * 8 + dt) * 64 + lane] = dk[dt];
                x[((wave * 2 + 1) * 8 + dt) * 64 + lane] = dv[dt];
            }
        }
        __syncthreads();
        if (grp == 1) return;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
            dk[dt] += x[((wave * 2 + 0) * 8 + dt) * 64 + lane];
            dv[dt] += x[((wave * 2 + 1) * 8 + dt) * 64 + lane];
        }
    }
    if (kabs < a.seq) {
        uint16_t* row = a.dqkv + (tok0 + kabs) * a.lddq + a.dcol0 + (int64_t)hh * 3 * D;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
            const u32x2 wk = {pack_bf16x2(dk[dt][0] * a.inv_sqrt_d, dk[dt][1] * a.inv_sqrt_d),
                              pack_bf16x2(dk[dt][2] * a.inv_sqrt_d, dk[dt][3] * a.inv_sqrt_d)};
            const u32x2 wv2 = {pack_bf16x2(dv[dt][0], dv[dt][1]), pack_bf16x2(dv[dt][2], dv[dt][3])};
            *reinterpret_cast<u32x2*>(row + D + 16 * dt + 4 * g) = wk;
            *reinterpret_cast<u32x2*>(row + 2 * D + 16 * dt + 4 * g) = wv2;
        }
    }
}

// dQ of one query tile: RB row blocks of 16 queries per wave (64 RB rows;
// block r of wave w holds rows 64 r + 16 w .. + 15), so every K and V
// fragment read from LDS feeds RB MFMAs.  KG groups of four waves split the
// tile's key tiles (group 0 the first half, group 1 the rest, with the
// diagonal); group 1 adds its sums into group 0's through LDS at the end.
template <int RB, int KG>
__global__ __launch_bounds__(NTHR * KG, 2 / KG) void attention_dq_kernel(AttnBwdArgs a) {
    constexpr int QT = 64 * RB;
    __shared__ __attribute__((aligned(16))) uint16_t kv[KG][2][2][BN * D];   // [grp][buf][K|V]
    const int lane = threadIdx.x & 63, g = lane >> 4;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int grp = wv / NWAVE, wave = wv % NWAVE;
    const int bhn = a.batch * a.heads;
    const int qt = a.tiles - 1 - blockIdx.x / bhn;   // long loops first
    const int bh = blockIdx.x % bhn;
    const int b = bh / a.heads, hh = bh % a.heads;
    const int64_t tok0 = (int64_t)b * a.seq, T = (int64_t)a.batch * a.seq;
    const int64_t qc = a.col0 + (int64_t)hh * 3 * D;

    int qabs[RB];
    bf16x8 qf[RB][4], of[RB][4];
    float l2[RB], dl[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        qabs[r] = qt * QT + 64 * r + wave * 16 + (lane & 15);
        l2[r] = 0.f;
        dl[r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            if (qabs[r] < a.seq) {
                qf[r][ks] = *reinterpret_cast<const bf16x8*>(
                    a.qkv + (tok0 + qabs[r]) * a.ldq + qc + 32 * ks + 8 * g);
                of[r][ks] = *reinterpret_cast<const bf16x8*>(
                    a.dout + (tok0 + qabs[r]) * a.lddo + a.docol0 + (int64_t)hh * D + 32 * ks +
                    8 * g);
            } else {
                qf[r][ks] = __builtin_bit_cast(bf16x8, u32x4{0, 0, 0, 0});
                of[r][ks] = qf[r][ks];
            }
        }
        // delta of the row = dO . O over the head's 128 columns: each of the
        // row's four lanes sums its 32 columns, then the lane swaps add them
        float acc = 0.f;
        if (qabs[r] < a.seq) {
            l2[r] = a.lse[(int64_t)hh * T + tok0 + qabs[r]] * 1.44269504088896340736f;
            const uint16_t* orow = a.out + (tok0 + qabs[r]) * a.ldo + a.ocol0 + (int64_t)hh * D;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                const u32x4 o = *reinterpret_cast<const u32x4*>(orow + 32 * ks + 8 * g);
                const u32x4 d = __builtin_bit_cast(u32x4, of[r][ks]);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc += __uint_as_float(o[e] << 16) * __uint_as_float(d[e] << 16);
                    acc += __uint_as_float(o[e] & 0xffff0000u) * __uint_as_float(d[e] & 0xffff0000u);
                }
            }
        }
        dl[r] = row_sum4(acc);   // every lane of the wave takes part
        // the dK/dV kernel, launched after this one, reads it
        if (grp == 0 && g == 0 && qabs[r] < a.seq) a.delta[(int64_t)hh * T + tok0 + qabs[r]] = dl[r];
    }
    f32x4 dq[RB][8];
#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) dq[r][dt] = f32x4{0.f, 0.f, 0.f, 0.f};

    int boff[4], toff[8];
    offsets(lane, boff, toff);
    const uint16_t* kbase = a.qkv + qc + D;
    const uint16_t* vbase = a.qkv + qc + 2 * D;
    // key tiles up to the tile's last row inside the sequence: group 0 the
    // first half, group 1 the rest
    const int last = min(qt * QT + QT, a.seq) - 1;
    const int nk = last / BN + 1;
    const int half = KG > 1 ? (nk + 1) / 2 : nk;
    const int k0 = grp == 0 ? 0 : half;
    const int mine = grp == 0 ? half : nk - half;   // <= half
    uint16_t(*kb)[2][BN * D] = kv[grp];
    TileDma2<false> cp;
    cp.init(a.ldq, a.ldq, wave, lane);
    if (mine > 0)
        cp.issue(kbase, a.ldq, vbase, a.ldq, tok0, k0 * BN, a.seq, kb[0][0], kb[0][1], wave);
    dma::wait_vmcnt<0>();
    __syncthreads();
    for (int i = 0; i < half; ++i) {
        if (i < mine) {
            const int kt = k0 + i;
            const uint16_t* ks_ = kb[i & 1][0];
            const uint16_t* vs_ = kb[i & 1][1];
            if (i + 1 < mine)
                cp.issue(kbase, a.ldq, vbase, a.ldq, tok0, (kt + 1) * BN, a.seq,
                         kb[(i + 1) & 1][0], kb[(i + 1) & 1][1], wave);
            // S and dP: lane holds (query = qabs[r], key = 16 j + 4 g + e); a
            // key tile reaching past the tile's first row, or a ragged one,
            // has masked keys
            const bool masked = (kt + 1) * BN > qt * QT || (kt + 1) * BN > a.seq;
            // JG 16-key blocks at a time advance together over the head
            // dimension (2 JG RB independent accumulators), then become dS
            constexpr int JG = RB == 1 ? 4 : 2;
            f32x4 dsv[RB][4];
#pragma unroll
            for (int j0 = 0; j0 < 4; j0 += JG) {
                f32x4 sacc[RB][JG], dacc[RB][JG];
#pragma unroll
                for (int r = 0; r < RB; ++r)
#pragma unroll
                    for (int jj = 0; jj < JG; ++jj) {
                        sacc[r][jj] = f32x4{0.f, 0.f, 0.f, 0.f};
                        dacc[r][jj] = sacc[r][jj];
                    }
#pragma unroll
                for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                    for (int jj = 0; jj < JG; ++jj) {
                        const int j = j0 + jj;
                        const bf16x8 kf =
                            *reinterpret_cast<const bf16x8*>(ks_ + 16 * j * D + boff[ks]);
                        const bf16x8 vf =
                            *reinterpret_cast<const bf16x8*>(vs_ + 16 * j * D + boff[ks]);
#pragma unroll
                        for (int r = 0; r < RB; ++r) {
                            sacc[r][jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                kf, qf[r][ks], sacc[r][jj], 0, 0, 0);
                            dacc[r][jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                vf, of[r][ks], dacc[r][jj], 0, 0, 0);
                        }
                    }
#pragma unroll
                for (int jj = 0; jj < JG; ++jj)
#pragma unroll
                    for (int r = 0; r < RB; ++r)
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int j = j0 + jj;
                            float pv = __builtin_amdgcn_exp2f(
                                __builtin_fmaf(sacc[r][jj][e], a.scale_log2, -l2[r]));
                            if (masked) {
                                const int kabs = kt * BN + 16 * j + 4 * g + e;
                                if (kabs > qabs[r] || kabs >= a.seq) pv = 0.f;
                            }
                            dsv[r][j][e] = pv * (dacc[r][jj][e] - dl[r]);
                        }
            }
            // dQ += dS K over two 32-key slices
#pragma unroll
            for (int sl = 0; sl < 2; ++sl) {
                bf16x8 sf[RB];
#pragma unroll
                for (int r = 0; r < RB; ++r) sf[r] = pack_pair(dsv[r][2 * sl], dsv[r][2 * sl + 1]);
#pragma unroll
                for (int dt = 0; dt < 8; ++dt) {
                    const bf16x8 kt_ = frag_tr_at(ks_ + 32 * sl * D + toff[dt]);
#pragma unroll
                    for (int r = 0; r < RB; ++r)
                        dq[r][dt] =
                            __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt_, sf[r], dq[r][dt], 0, 0, 0);
                }
            }
        }
        dma::wait_vmcnt<0>();
        __syncthreads();
    }
    if constexpr (KG > 1) {
        f32x4* x = reinterpret_cast<f32x4*>(&kv[1][0][0][0]);
        if (grp == 1) {
#pragma unroll
            for (int r = 0; r < RB; ++r)
#pragma unroll
                for (int dt = 0; dt < 8; ++dt) x[((wave * RB + r) * 8 + dt) * 64 + lane] = dq[r][dt];
        }
        __syncthreads();
        if (grp == 1) return;
#pragma unroll
        for (int r = 0; r < RB; ++r)
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) dq[r][dt] += x[((wave * RB + r) * 8 + dt) * 64 + lane];
    }
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        if (qabs[r] >= a.seq) continue;
        uint16_t* row = a.dqkv + (tok0 + qabs[r]) * a.lddq + a.dcol0 + (int64_t)hh * 3 * D;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
            const u32x2 w = {pack_bf16x2(dq[r][dt][0] * a.inv_sqrt_d, dq[r][dt][1] * a.inv_sqrt_d),
                             pack_bf16x2(dq[r][dt][2] * a.inv_sqrt_d, dq[r][dt][3] * a.inv_sqrt_d)};
            *reinterpret_cast<u32x2*>(row + 16 * dt + 4 * g) = w;
        }
    }
}

}  // namespace

hipError_t launch_attention_bwd(const AttentionBwdProblem& p, hipStream_t s) {
    if (p.batch <= 0 || p.seq <= 0 || p.heads <= 0) return hipSuccess;
    if (p.head_dim != D) return hipErrorInvalidValue;
    AttnBwdArgs a;
    a.qkv = static_cast<const uint16_t*>(p.qkv);
    a.ldq = p.ld_qkv;
    a.col0 = p.qkv_col0;
    a.out = static_cast<const uint16_t*>(p.out);
    a.ldo = p.ld_out;
    a.ocol0 = p.out_col0;
    a.dout = static_cast<const uint16_t*>(p.dout);
    a.lddo = p.ld_dout;
    a.docol0 = p.out_col0;
    a.lse = p.lse;
    a.delta = p.delta;
    a.dqkv = static_cast<uint16_t*>(p.dqkv);
    a.lddq = p.ld_dqkv;
    a.dcol0 = p.qkv_col0;
    a.batch = (int)p.batch;
    a.seq = (int)p.seq;
    a.heads = p.heads;
    a.tiles = (int)((p.seq + BM - 1) / BM);
    a.scale_log2 = 1.44269504088896340736f / sqrtf((float)D);
    a.inv_sqrt_d = 1.0f / sqrtf((float)D);
    const int64_t grid = (int64_t)a.tiles * a.batch * a.heads;
    if (grid > 0x7fffffff) return hipErrorInvalidValue;
    // the dQ kernel first: it forms delta for its query rows and stores it
    // for the dK/dV kernel.  Small grids split each workgroup's loop over two
    // groups of four waves (one workgroup per CU), so the longest loops take
    // half as many steps; dQ takes 128-row query tiles (two row blocks per
    // wave) when they still give every CU two workgroups.
    const bool split = grid < kBwdSplitGrid;
    if (split) {
        hipLaunchKernelGGL((attention_dq_kernel<1, 2>), dim3((unsigned)grid), dim3(2 * NTHR), 0,
                           s, a);
        hipLaunchKernelGGL((attention_dkv_kernel<2>), dim3((unsigned)grid), dim3(2 * NTHR), 0, s,
                           a);
        return hipGetLastError();
    }
    AttnBwdArgs a2 = a;
    a2.tiles = (int)((p.seq + 127) / 128);
    const int64_t grid2 = (int64_t)a2.tiles * a.batch * a.heads;
    if (grid2 >= kFwdWideGrid)
        hipLaunchKernelGGL((attention_dq_kernel<2, 1>), dim3((unsigned)grid2), dim3(NTHR), 0, s,
                           a2);
    else
        hipLaunchKernelGGL((attention_dq_kernel<1, 1>), dim3((unsigned)grid), dim3(NTHR), 0, s, a);
    hipLaunchKernelGGL((attention_dkv_kernel<1>), dim3((unsigned)grid), dim3(NTHR), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_attention_fwd(const AttentionProblem& p, hipStream_t s) {
    if (p.batch <= 0 || p.seq <= 0 || p.heads <= 0) return hipSuccess;
    if (p.head_dim != D) return hipErrorInvalidValue;
    AttnArgs a;
    a.qkv = static_cast<const uint16_t*>(p.qkv);
    a.ldq = p.ld_qkv;
    a.col0 = p.qkv_col0;
    a.out = static_cast<uint16_t*>(p.out);
    a.ldo = p.ld_out;
    a.ocol0 = p.out_col0;
    a.lse = p.lse;
    a.batch = (int)p.batch;
    a.seq = (int)p.seq;
    a.heads = p.heads;
    a.scale_log2 = 1.44269504088896340736f / sqrtf((float)D);
    // Enough 128-row query tiles for two workgroups on every CU: four waves
    // of two row blocks, two workgroups per CU (measured on the wide layer's
    // share: 546-558 TFLOP/s, against 488-495 for the other shapes).  Fewer:
    // 64-row tiles whose key range is split over two groups of four waves
    // (one workgroup per CU), so the longest causal rows take half as many
    // steps (GPT-3 share 339 against 248 for one group, 191 for 128 rows).
    const int64_t bh = p.batch * (int64_t)p.heads;
    const bool wide = ((p.seq + 127) / 128) * bh >= kFwdWideGrid;
    a.qtiles = (int)(wide ? (p.seq + 127) / 128 : (p.seq + 63) / 64);
    const int64_t grid = (int64_t)a.qtiles * bh;
    if (grid > 0x7fffffff) return hipErrorInvalidValue;
    if (wide)
        hipLaunchKernelGGL((attention_fwd_kernel<2, 1>), dim3((unsigned)grid), dim3(NTHR), 0, s,
                           a);
    else
        hipLaunchKernelGGL((attention_fwd_kernel<1, 2>), dim3((unsigned)grid), dim3(2 * NTHR), 0,
                           s, a);
    return hipGetLastError();
}

}  // namespace atp
