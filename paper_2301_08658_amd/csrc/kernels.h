// Internal launch interface between the C ABI / pipeline and the gfx950
// kernels.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace atp {

// Epilogue codes; identical values to atp_epilogue in include/atp.h.
enum Epi : int { EPI_NONE = 0, EPI_BIAS = 1, EPI_BIAS_GELU = 2, EPI_GELU_BWD = 3 };

// Operand layouts of C[M,N] = sum_k A(m,k) B(k,n):
//   NN: A(m,k) = A[m*lda + k],  B(k,n) = B[k*ldb + n]   (forward  Y  = X W)
//   NT: A(m,k) = A[m*lda + k],  B(k,n) = B[n*ldb + k]   (backward dX = dY W^T)
//   TN: A(m,k) = A[k*lda + m],  B(k,n) = B[k*ldb + n]   (backward dW = X^T dY)
enum Layout : int { LAYOUT_NN = 0, LAYOUT_NT = 1, LAYOUT_TN = 2 };

struct GemmProblem {
    int layout;
    const void* A; int64_t lda;   // bf16
    const void* B; int64_t ldb;   // bf16
    void* C; int64_t ldc;         // f32 or bf16, row-major [M, N]
    bool out_bf16;
    int epi;
    const void* bias;             // bf16 [N] for BIAS / BIAS_GELU
    const void* pre_in;           // bf16 [M, N] (ld ldc) for GELU_BWD
    void* pre_out;                // bf16 [M, N] (ld ldc) for BIAS_GELU, nullable
    int64_t M, N, K;
    // split-K (NT, EPI_NONE, fp32 only): split s sums k in [s*ksplit,
    // min(K, (s+1)*ksplit)) into the fp32 slab C + s*c_split (ld ldc);
    // ksplit a multiple of 64, every split non-empty
    int splits = 1;
    int64_t ksplit = 0, c_split = 0;
    // fused peer sum (NN, no split): when nparts > 1 the epilogue forms
    // sum_{j < nparts} P_j in group order before bias / GeLU, with P_own the
    // tile's own accumulators and the others read from peers[j] (fp32, ld ldp)
    int nparts = 1, own = 0;
    const float* peers[8] = {};   // kMaxFusedParts
    int64_t ldp = 0;
};
constexpr int kMaxFusedParts = 8;

// True if the kernel set has an instance for this (layout, epi, out) combination.
bool gemm_supported(int layout, int epi, bool out_bf16);
hipError_t launch_gemm(const GemmProblem& p, hipStream_t s);
// Profiling name of the kernel a problem launches (layout and tile configuration).
const char* gemm_kernel_name(const GemmProblem& p);

// Split-K plan for an NT product [M, N] over K written to fp32: returns the
// split count S (1: no split) and the k per split (a multiple of 64; the
// last split may be shorter).  The plan depends on M, N and K only; S *
// (256-row tiles) * (160-column tiles) never exceeds kMaxSplitTiles.
// True when an unsplit NN product [M, N] (B read along its rows, the
// forward from W stored [k][n]) runs on the 256 x 256 tiles with split copy
// rings, which stream it as fast as NT from a transposed copy.
bool nn_streams_like_nt(int64_t M, int64_t N);

constexpr int kMaxSplits = 16;
constexpr int64_t kMaxSplitTiles = 512;
int nt_split_plan(int64_t M, int64_t N, int64_t K, int64_t* ksplit);

constexpr int kMaxParts = 64;

struct ReduceProblem {
    int nparts;
    const void* parts[kMaxParts];   // each f32 (or bf16 if parts_bf16) [.., ldp]
    bool parts_bf16;
    int64_t ldp;
    int64_t row0, rows, ncols;      // rows [row0, row0+rows), columns [0, ncols)
    int epi;
    const void* bias;               // bf16 [ncols]
    const void* pre_in;             // bf16, ld ldo
    void* out; int64_t ldo; bool out_bf16;
    void* pre_out;                  // bf16, ld ldo, nullable
};
hipError_t launch_reduce(const ReduceProblem& p, hipStream_t s);

// out[r*ldo + c] = sum_{s<S} slab_s[r*ld + c] for slab_s = ws + s*stride,
// r < rows, c < cols (fp32, summed in s order; stored fp32, or bf16 rounded
// to nearest even): the split-K partials of one product combined into one
// partial.
hipError_t launch_split_sum(const float* ws, int S, int64_t stride, int64_t ld, int64_t rows,
                            int64_t cols, void* out, int64_t ldo, bool out_bf16, hipStream_t s);

// Causal attention of `heads` consecutive heads over `batch` sequences of
// `seq` tokens (token rows sequence-major).  Head j's q, k, v are the
// head_dim-wide column runs at qkv_col0 + 3*head_dim*j + {0, 1, 2}*head_dim of
// qkv (bf16, ld ld_qkv); its output goes to columns out_col0 + head_dim*j of
// out (bf16, ld ld_out) and its row log-sum-exps to lse[j*batch*seq + t]
// (fp32, natural log).  head_dim must be 128.
struct AttentionProblem {
    const void* qkv; int64_t ld_qkv, qkv_col0;
    void* out; int64_t ld_out, out_col0;
    float* lse;
    int64_t batch, seq;
    int heads, head_dim;
};
hipError_t launch_attention_fwd(const AttentionProblem& p, hipStream_t s);

// Its gradient: from qkv, the forward output out (its heads at out_col0),
// the output gradient dout (same columns, ld ld_dout) and the saved lse,
// write dq, dk, dv of the heads into dqkv at qkv_col0 (the qkv layout, ld
// ld_dqkv).  delta is fp32 scratch [heads*batch*seq].  Three launches:
// delta = rowsum(dO o O), dK/dV per key tile, dQ per query tile.
struct AttentionBwdProblem {
    const void* qkv; int64_t ld_qkv, qkv_col0;
    const void* out; int64_t ld_out, out_col0;
    const void* dout; int64_t ld_dout;
    const float* lse;
    float* delta;
    void* dqkv; int64_t ld_dqkv;
    int64_t batch, seq;
    int heads, head_dim;
};
hipError_t launch_attention_bwd(const AttentionBwdProblem& p, hipStream_t s);

// db[n] = sum_t dy[t*ld + n], dy bf16 [T, N], db f32 [N], in one fixed order:
// 8-row groups, then the groups of each 64-row block, then the blocks, all
// ascending (the same bits as transpose partials + launch_colsum_finish).
hipError_t launch_colsum(const void* dy, int64_t ld, int64_t T, int64_t N, float* db,
                         hipStream_t s);
// db[n] = sum over b < nb, ascending, of part[b*ldp + n] (fp32).
hipError_t launch_colsum_finish(const float* part, int64_t ldp, int64_t nb, int64_t N, float* db,
                                hipStream_t s);

// dst[c*ldd + r] = src[r*lds + c] for r < rows, c < cols (bf16).  With
// part (rows, cols, lds, ldd multiples of 8): also the column sums of every
// 64-row block of src in launch_colsum's order, part[(r / 64)*ldpart + c]
// (fp32), for launch_colsum_finish.
hipError_t launch_transpose(const void* src, int64_t lds, int64_t rows, int64_t cols, void* dst,
                            int64_t ldd, hipStream_t s, float* part = nullptr,
                            int64_t ldpart = 0);

}  // namespace atp
