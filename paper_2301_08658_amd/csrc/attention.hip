// Causal attention core of one device's heads (Sec. 2.1 Formula (mha); the
// attention block of Sec. 3.2.1 scatters the heads of the reduced QKV block
// over the group that reduced it, each device attends over its run of heads,
// and the outputs are gathered before out-proj).
//
// Forward, one workgroup per (sequence, head, 64-row query tile), four waves
// of 16 query rows, head dimension 128, keys in steps of 64 (flash-attention
// style: running row maximum and sum, the output rescaled as they grow).
//
//   * S = Q K^T on v_mfma_f32_16x16x32_bf16: Q fragments stay in registers
//     for the whole row tile; K fragments are ds_read_b128 from a [key][d]
//     LDS tile whose 16-byte chunks are XOR-swizzled by key (c ^ (n & 15)),
//     which puts the 16 lanes of each gfx950 read group on distinct banks.
//   * A lane holds S(m = lane % 16, n = 16 j + 4 (lane / 16) + e): the rows
//     are lane-uniform, so the row maximum and sum need only two lane
//     exchanges (xor 16, xor 32).
//   * O += P V: the MFMA sums over its 32 keys in any order as long as both
//     operands agree, so each 32-key slice takes the keys {4g + e} and
//     {16 + 4g + e} for lane group g: then P's fragment is the lane's own
//     eight probabilities (two S tiles, no exchange), and V's fragment is two
//     ds_read_b64_tr_b16 from a [key][d] tile (chunk c at c ^ (2 (n & 3) +
//     8 ((n >> 2) & 1)), distinct banks per 32-lane half).
//   * Exponentials in base 2 (scores scaled by log2(e) / sqrt(128)); the
//     log-sum-exp of each row is saved (natural log) for the backward.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace atp {
namespace {

constexpr int D = 128;          // head dimension
constexpr int BM = 64;          // query rows per workgroup
constexpr int BN = 64;          // keys per step
constexpr int NWAVE = 4;
constexpr int NTHR = NWAVE * 64;
constexpr int CH = D / 8;       // 16-byte chunks per row

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

__device__ __forceinline__ int kpos(int n, int c) { return c ^ (n & 15); }
__device__ __forceinline__ int vpos(int n, int c) { return c ^ (2 * (n & 3) + 8 * ((n >> 2) & 1)); }

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    auto rne = [](float f) -> uint32_t {
        uint32_t u = __float_as_uint(f);
        if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return 0x7fc0u;
        u += 0x7fffu + ((u >> 16) & 1u);
        return u >> 16;
    };
    return rne(a) | (rne(b) << 16);
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

// Copy rows [n0, n0 + BN) of K and V of one head into registers (rows past
// the sequence read zeros): thread t takes chunks t, t + 256, ... of each.
__device__ __forceinline__ void load_kv(const AttnArgs& a, int64_t tok0, int64_t kc, int64_t vc,
                                        int n0, u32x4 (&kr)[4], u32x4 (&vr)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int q = threadIdx.x + i * NTHR;
        const int n = q / CH, c = q % CH;
        if (n0 + n < a.seq) {
            const uint16_t* row = a.qkv + (tok0 + n0 + n) * a.ldq;
            kr[i] = *reinterpret_cast<const u32x4*>(row + kc + 8 * c);
            vr[i] = *reinterpret_cast<const u32x4*>(row + vc + 8 * c);
        } else {
            kr[i] = u32x4{0, 0, 0, 0};
            vr[i] = u32x4{0, 0, 0, 0};
        }
    }
}

__device__ __forceinline__ void store_kv(uint16_t* ks, uint16_t* vs, const u32x4 (&kr)[4],
                                         const u32x4 (&vr)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int q = threadIdx.x + i * NTHR;
        const int n = q / CH, c = q % CH;
        *reinterpret_cast<u32x4*>(ks + n * D + kpos(n, c) * 8) = kr[i];
        *reinterpret_cast<u32x4*>(vs + n * D + vpos(n, c) * 8) = vr[i];
    }
}

__global__ __launch_bounds__(NTHR, 2) void attention_fwd_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t kv[2][2][BN * D];   // [buf][K|V]
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // longest rows first: the last query tile of every (sequence, head) leads
    const int per = a.qtiles;
    const int bid = blockIdx.x;
    const int qt = per - 1 - bid / (a.batch * a.heads);
    const int bh = bid % (a.batch * a.heads);
    const int b = bh / a.heads, hh = bh % a.heads;
    const int64_t tok0 = (int64_t)b * a.seq;
    const int64_t qc = a.col0 + (int64_t)hh * 3 * D, kc = qc + D, vc = qc + 2 * D;

    // Q fragments: row m0 + lane % 16, d = 32 ks + 8 (lane / 16) + 0..7
    const int m0 = qt * BM + wave * 16;
    const int mrow = m0 + (lane & 15);
    bf16x8 qf[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
        if (mrow < a.seq)
            qf[ks] = *reinterpret_cast<const bf16x8*>(a.qkv + (tok0 + mrow) * a.ldq + qc +
                                                      32 * ks + 8 * (lane >> 4));
        else
            qf[ks] = __builtin_bit_cast(bf16x8, u32x4{0, 0, 0, 0});
    }

    f32x4 o[8];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float mrun = -INFINITY, lrun = 0.f;

    const int nkt = qt + 1;   // causal: key tiles 0..qt
    u32x4 kr[4], vr[4];
    load_kv(a, tok0, kc, vc, 0, kr, vr);
    store_kv(kv[0][0], kv[0][1], kr, vr);
    __syncthreads();
    const int g = lane >> 4;
    for (int kt = 0; kt < nkt; ++kt) {
        const uint16_t* ks_ = kv[kt & 1][0];
        const uint16_t* vs_ = kv[kt & 1][1];
        if (kt + 1 < nkt) load_kv(a, tok0, kc, vc, (kt + 1) * BN, kr, vr);

        // S = Q K^T for 16 rows x 64 keys
        f32x4 s[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            s[j] = f32x4{0.f, 0.f, 0.f, 0.f};
            const int n = 16 * j + (lane & 15);
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                const int c = 4 * ks + g;
                const bf16x8 kf = *reinterpret_cast<const bf16x8*>(ks_ + n * D + kpos(n, c) * 8);
                s[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[ks], s[j], 0, 0, 0);
            }
        }
        // scale, causal mask (and keys past the sequence), row maximum
        float mx = -INFINITY;
        const int qabs = mrow;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int nabs = kt * BN + 16 * j + 4 * g + e;
                float v = s[j][e] * a.scale_log2;
                if (nabs > qabs || nabs >= a.seq) v = -INFINITY;
                s[j][e] = v;
                mx = fmaxf(mx, v);
            }
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float mnew = fmaxf(mrun, mx);
        const float alpha = __builtin_amdgcn_exp2f(mrun - mnew);
        float rs = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float p = __builtin_amdgcn_exp2f(s[j][e] - mnew);
                s[j][e] = p;
                rs += p;
            }
        rs += __shfl_xor(rs, 16);
        rs += __shfl_xor(rs, 32);
        lrun = lrun * alpha + rs;
        mrun = mnew;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) o[dt] *= alpha;

        // O += P V over two 32-key slices
#pragma unroll
        for (int sl = 0; sl < 2; ++sl) {
            const u32x4 pw = {pack_bf16x2(s[2 * sl][0], s[2 * sl][1]),
                              pack_bf16x2(s[2 * sl][2], s[2 * sl][3]),
                              pack_bf16x2(s[2 * sl + 1][0], s[2 * sl + 1][1]),
                              pack_bf16x2(s[2 * sl + 1][2], s[2 * sl + 1][3])};
            const bf16x8 pf = __builtin_bit_cast(bf16x8, pw);
            // lane j of group g names 4 columns of key row rb + j / 4
            const int j16 = lane & 15;
            const int r0 = 32 * sl + 4 * g + (j16 >> 2);
            const int r1 = r0 + 16;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) {
                const int col = 16 * dt + 4 * (j16 & 3);
                const int c = col >> 3;
                const uint16_t* p0 = vs_ + r0 * D + vpos(r0, c) * 8 + (col & 7);
                const uint16_t* p1 = vs_ + r1 * D + vpos(r1, c) * 8 + (col & 7);
                const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p0);
                const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p1);
                const i16x8 vv = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vv),
                                                                pf, o[dt], 0, 0, 0);
            }
        }
        if (kt + 1 < nkt) {
            __syncthreads();   // every wave is done with the other buffer
            store_kv(kv[(kt + 1) & 1][0], kv[(kt + 1) & 1][1], kr, vr);
            __syncthreads();
        }
    }

    // O / l as bf16: lane holds O(m = mrow, d = 16 dt + 4 g + 0..3)
    if (mrow < a.seq) {
        const float inv = 1.0f / lrun;
        uint16_t* orow = a.out + (tok0 + mrow) * a.ldo + a.ocol0 + (int64_t)hh * D;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
            const u32x2 w = {pack_bf16x2(o[dt][0] * inv, o[dt][1] * inv),
                             pack_bf16x2(o[dt][2] * inv, o[dt][3] * inv)};
            *reinterpret_cast<u32x2*>(orow + 16 * dt + 4 * g) = w;
        }
        if (g == 0)
            a.lse[(int64_t)hh * a.batch * a.seq + tok0 + mrow] =
                (mrun + __log2f(lrun)) * 0.69314718055994530942f;
    }
}

}  // namespace

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
    a.qtiles = (int)((p.seq + BM - 1) / BM);
    a.scale_log2 = 1.44269504088896340736f / sqrtf((float)D);
    const int64_t grid = (int64_t)a.qtiles * a.batch * a.heads;
    if (grid > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL(attention_fwd_kernel, dim3((unsigned)grid), dim3(NTHR), 0, s, a);
    return hipGetLastError();
}

}  // namespace atp
