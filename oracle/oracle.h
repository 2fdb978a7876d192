/*
 * oracle.h -- plain fp64 CPU reference for the ATP shard block.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library includes,
 * links or calls this code; only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark do.  It shares no source, header,
 * table or helper with the HIP path.
 *
 * Paper: Cheng, Liu, Du, You, "ATP: Adaptive Tensor Parallelism for
 * Foundation Models" (arXiv 2301.08658).  Every function cites the passage
 * it follows.  All arithmetic is IEEE double, evaluated in the order the
 * definitions state (no blocking, no reassociation, no FMA contraction).
 *
 * Layout: every matrix is addressed through explicit element strides, so a
 * transposed operand is the same matrix read with swapped strides.
 */
#ifndef ATP_ORACLE_H
#define ATP_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Placement codes of the sharding spec (Sec. 3.1, "Sharding Spec"):
 * a value >= 0 is Shard(dim); the negative codes are the other two kinds. */
#define ORC_REPLICATE   (-1)
#define ORC_PARTIAL_SUM (-2)

/* Sec. 3.1 "Device Mesh": rank <-> coordinate on a mesh, row-major (the last
 * mesh dimension varies fastest).  Returns the rank. */
int64_t orc_mesh_rank(int ndim, const int32_t* mesh, const int32_t* coord);
/* Inverse of orc_mesh_rank. */
void orc_mesh_coord(int ndim, const int32_t* mesh, int64_t rank, int32_t* coord);

/* Sec. 3.1 "Sharding Spec": the block of a global tensor held by the device
 * at `coord` under the spec `placements` (one entry per mesh dimension).
 * Mesh dimensions are applied in order; Shard(d) splits the current extent
 * of tensor dimension d into mesh[i] equal contiguous parts and keeps part
 * coord[i].  Replicate and Partial leave the extent unchanged.
 * Returns 0, or -1 if an extent is not divisible. */
int orc_spec_block(int mesh_ndim, const int32_t* mesh, const int32_t* coord,
                   const int32_t* placements, int tensor_ndim,
                   const int64_t* shape, int64_t* lo, int64_t* hi);

/* Sec. 3.2: sharding specs of the operands of Y = X W on DeviceMesh(d1,d2).
 *   mode 0 = row-first:    W [Shard(0),Shard(1)], X [Shard(1),Replicate],
 *                          Y [Partial(SUM),Shard(1)]
 *   mode 1 = column-first: W [Shard(1),Shard(0)], X [Replicate,Shard(1)],
 *                          Y [Shard(1),Partial(SUM)]
 * Each output array holds two placements. */
void orc_linear_specs(int mode, int32_t* x_spec, int32_t* w_spec, int32_t* y_spec);

/* Sec. 3.2 (and Eq. of Y = XW): C[m][n] = sum_{k ascending} A[m][k] * B[k][n],
 * with element (i,j) of A at A[i*sa0 + j*sa1] and likewise for B and C. */
void orc_matmul(int64_t M, int64_t K, int64_t N,
                const double* A, int64_t sa0, int64_t sa1,
                const double* B, int64_t sb0, int64_t sb1,
                double* C, int64_t sc0, int64_t sc1);

/* Sec. 2.1 (feed-forward block): GeLU with the Gaussian CDF written through
 * erf, and its derivative Phi(x) + x*phi(x). */
double orc_gelu(double x);
double orc_gelu_grad(double x);

/* Epilogues applied after the grouped reduction (Sec. 3.2.1). */
#define ORC_EPI_NONE      0
#define ORC_EPI_BIAS      1
#define ORC_EPI_BIAS_GELU 2
#define ORC_EPI_GELU_BWD  3

/* Sec. 3.1 Partial(SUM) + Sec. 3.2 grouped all-reduce: for every (t,n)
 *   s = sum_{j = 0..nparts-1} parts[j][t*ldp + n]
 *   EPI_NONE:      out = s
 *   EPI_BIAS:      out = s + bias[n]
 *   EPI_BIAS_GELU: pre = s + bias[n]; out = GeLU(pre); preact_out = pre
 *   EPI_GELU_BWD:  out = s * GeLU'(preact_in[t*ldo + n])
 * preact_out may be NULL. */
void orc_partial_reduce(int nparts, const double* const* parts, int64_t ldp,
                        int64_t T, int64_t N, const double* bias, int epi,
                        const double* preact_in, double* out, int64_t ldo,
                        double* preact_out);

/* Bias gradient: db[n] = sum_{t ascending} dy[t*ld + n]. */
void orc_colsum(int64_t T, int64_t N, const double* dy, int64_t ld, double* db);

/* Sec. 5: the model's tensors are 16-bit (the paper trains in half
 * precision; the GPU path stores activations and activation gradients as
 * bfloat16).  Rounds x to the nearest bfloat16 value (8 significant bits,
 * fp32 exponent range, ties to even, overflow to infinity) and returns it
 * as a double.  Used where one GEMM's output is the next GEMM's input. */
double orc_round_bf16(double x);

/* Number of OpenMP threads the oracle runs with. */
int orc_num_threads(void);

/* Attention core of one head over one sequence of S tokens (Sec. 2.1,
 * Formula (mha), with the causal mask of a decoder-only GPT, Sec. 5):
 *   s[t][u] = (q_t . k_u) / sqrt(d)              for u <= t
 *   p[t][u] = exp(s[t][u] - lse[t]),  lse[t] = log sum_{u<=t} exp(s[t][u])
 *   o[t]    = sum_{u<=t} p[t][u] v_u
 * q, k, v, o are [S][d] rows with leading dimensions ldq, ldk, ldv, ldo;
 * lse is [S]. */
void orc_attention_fwd(int64_t S, int64_t d, const double* q, int64_t ldq, const double* k,
                       int64_t ldk, const double* v, int64_t ldv, double* o, int64_t ldo,
                       double* lse);

/* Its gradient given dO: with P as above and D[t] = sum_u p[t][u] (dO_t . v_u),
 *   dV_u = sum_{t>=u} p[t][u] dO_t
 *   dS[t][u] = p[t][u] (dO_t . v_u - D[t])
 *   dQ_t = sum_{u<=t} dS[t][u] k_u / sqrt(d),   dK_u = sum_{t>=u} dS[t][u] q_t / sqrt(d)
 * (the derivative of softmax and of the scaled products; D[t] equals
 * dO_t . o_t). */
void orc_attention_bwd(int64_t S, int64_t d, const double* q, int64_t ldq, const double* k,
                       int64_t ldk, const double* v, int64_t ldv, const double* dout,
                       int64_t lddo, double* dq, int64_t lddq, double* dk, int64_t lddk,
                       double* dv, int64_t lddv);

#ifdef __cplusplus
}
#endif
#endif
