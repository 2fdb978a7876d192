/*
 * oracle.c -- plain fp64 CPU reference for the ATP shard block.
 *
 * TEST INFRASTRUCTURE ONLY (see oracle.h).  Deliberately slow and obvious:
 * triple loops, ascending summation order, no blocking, compiled without
 * FMA contraction.  OpenMP only splits independent output rows.
 */
#include "oracle.h"

#include <math.h>
#include <stddef.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int64_t orc_mesh_rank(int ndim, const int32_t* mesh, const int32_t* coord) {
    /* Sec. 3.1: ranks enumerate the mesh with the last dimension fastest
     * (the [Replicate, Shard(0)] example puts ranks 0 and 2 in one group of
     * the second mesh dimension). */
    int64_t r = 0;
    for (int i = 0; i < ndim; ++i) r = r * mesh[i] + coord[i];
    return r;
}

void orc_mesh_coord(int ndim, const int32_t* mesh, int64_t rank, int32_t* coord) {
    for (int i = ndim - 1; i >= 0; --i) {
        coord[i] = (int32_t)(rank % mesh[i]);
        rank /= mesh[i];
    }
}

int orc_spec_block(int mesh_ndim, const int32_t* mesh, const int32_t* coord,
                   const int32_t* placements, int tensor_ndim,
                   const int64_t* shape, int64_t* lo, int64_t* hi) {
    for (int d = 0; d < tensor_ndim; ++d) { lo[d] = 0; hi[d] = shape[d]; }
    for (int i = 0; i < mesh_ndim; ++i) {
        int p = placements[i];
        if (p < 0) continue;              /* Replicate or Partial: whole extent */
        if (p >= tensor_ndim) return -1;
        int64_t ext = hi[p] - lo[p];
        if (ext % mesh[i] != 0) return -1;
        int64_t part = ext / mesh[i];
        lo[p] = lo[p] + (int64_t)coord[i] * part;
        hi[p] = lo[p] + part;
    }
    return 0;
}

void orc_linear_specs(int mode, int32_t* x_spec, int32_t* w_spec, int32_t* y_spec) {
    if (mode == 0) {
        /* row-first: weight split by rows on the first mesh level, by
         * columns on the second; the output is partial over the first. */
        w_spec[0] = 0;               w_spec[1] = 1;
        x_spec[0] = 1;               x_spec[1] = ORC_REPLICATE;
        y_spec[0] = ORC_PARTIAL_SUM; y_spec[1] = 1;
    } else {
        /* column-first: weight split by columns on the first level, by rows
         * on the second; the output is partial over the second. */
        w_spec[0] = 1;               w_spec[1] = 0;
        x_spec[0] = ORC_REPLICATE;   x_spec[1] = 1;
        y_spec[0] = 1;               y_spec[1] = ORC_PARTIAL_SUM;
    }
}

void orc_matmul(int64_t M, int64_t K, int64_t N,
                const double* A, int64_t sa0, int64_t sa1,
                const double* B, int64_t sb0, int64_t sb1,
                double* C, int64_t sc0, int64_t sc1) {
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t m = 0; m < M; ++m) {
        double* crow = C + m * sc0;
        for (int64_t n = 0; n < N; ++n) crow[n * sc1] = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            const double a = A[m * sa0 + k * sa1];
            const double* brow = B + k * sb0;
            for (int64_t n = 0; n < N; ++n) crow[n * sc1] += a * brow[n * sb1];
        }
    }
}

double orc_gelu(double x) {
    /* x * Phi(x), with Phi the standard normal CDF: Phi(x) = (1 + erf(x/sqrt2))/2 */
    return 0.5 * x * (1.0 + erf(x / sqrt(2.0)));
}

double orc_gelu_grad(double x) {
    /* d/dx [x Phi(x)] = Phi(x) + x phi(x), phi the standard normal density */
    const double Phi = 0.5 * (1.0 + erf(x / sqrt(2.0)));
    const double phi = exp(-0.5 * x * x) / sqrt(2.0 * 3.141592653589793238462643383279502884);
    return Phi + x * phi;
}

void orc_partial_reduce(int nparts, const double* const* parts, int64_t ldp,
                        int64_t T, int64_t N, const double* bias, int epi,
                        const double* preact_in, double* out, int64_t ldo,
                        double* preact_out) {
    #pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        for (int64_t n = 0; n < N; ++n) {
            double s = 0.0;
            for (int j = 0; j < nparts; ++j) s += parts[j][t * ldp + n];
            double v;
            switch (epi) {
            case ORC_EPI_BIAS:
                v = s + bias[n];
                break;
            case ORC_EPI_BIAS_GELU: {
                const double pre = s + bias[n];
                if (preact_out) preact_out[t * ldo + n] = pre;
                v = orc_gelu(pre);
                break;
            }
            case ORC_EPI_GELU_BWD:
                v = s * orc_gelu_grad(preact_in[t * ldo + n]);
                break;
            default:
                v = s;
                break;
            }
            out[t * ldo + n] = v;
        }
    }
}

void orc_colsum(int64_t T, int64_t N, const double* dy, int64_t ld, double* db) {
    #pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
        double s = 0.0;
        for (int64_t t = 0; t < T; ++t) s += dy[t * ld + n];
        db[n] = s;
    }
}

double orc_round_bf16(double x) {
    if (isnan(x) || isinf(x) || x == 0.0) return x;
    int e;
    (void)frexp(fabs(x), &e);          /* |x| = m * 2^e, m in [0.5, 1) */
    int q = e - 8;                     /* quantum of an 8-significant-bit value */
    if (q < -133) q = -133;            /* subnormal spacing 2^-133 */
    const double r = nearbyint(ldexp(fabs(x), -q));   /* ties to even */
    double y = ldexp(r, q);
    if (y > 3.38953138925153547590e38) y = INFINITY;  /* above the largest bfloat16 */
    return copysign(y, x);
}

int orc_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Scores of row t against keys 0..t, in ascending u. */
static void attn_scores(int64_t t, int64_t d, const double* q, int64_t ldq, const double* k,
                        int64_t ldk, double* s) {
    const double inv = 1.0 / sqrt((double)d);
    for (int64_t u = 0; u <= t; ++u) {
        double acc = 0.0;
        for (int64_t e = 0; e < d; ++e) acc += q[t * ldq + e] * k[u * ldk + e];
        s[u] = acc * inv;
    }
}

/* lse of scores s[0..n-1]: the largest score is taken out before exp. */
static double attn_lse(int64_t n, const double* s) {
    double mx = s[0];
    for (int64_t u = 1; u < n; ++u)
        if (s[u] > mx) mx = s[u];
    double sum = 0.0;
    for (int64_t u = 0; u < n; ++u) sum += exp(s[u] - mx);
    return mx + log(sum);
}

void orc_attention_fwd(int64_t S, int64_t d, const double* q, int64_t ldq, const double* k,
                       int64_t ldk, const double* v, int64_t ldv, double* o, int64_t ldo,
                       double* lse) {
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)(S > 0 ? S : 1));
#pragma omp for schedule(dynamic, 8)
        for (int64_t t = 0; t < S; ++t) {
            attn_scores(t, d, q, ldq, k, ldk, s);
            const double l = attn_lse(t + 1, s);
            for (int64_t e = 0; e < d; ++e) {
                double acc = 0.0;
                for (int64_t u = 0; u <= t; ++u) acc += exp(s[u] - l) * v[u * ldv + e];
                o[t * ldo + e] = acc;
            }
            if (lse) lse[t] = l;
        }
        free(s);
    }
}

void orc_attention_bwd(int64_t S, int64_t d, const double* q, int64_t ldq, const double* k,
                       int64_t ldk, const double* v, int64_t ldv, const double* dout,
                       int64_t lddo, double* dq, int64_t lddq, double* dk, int64_t lddk,
                       double* dv, int64_t lddv) {
    const double inv = 1.0 / sqrt((double)d);
    /* dS (lower triangle, row-major [S][S]) from P and dP = dO V^T */
    double* ds = (double*)calloc((size_t)(S > 0 ? S * S : 1), sizeof(double));
    double* p = (double*)calloc((size_t)(S > 0 ? S * S : 1), sizeof(double));
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)(S > 0 ? S : 1));
#pragma omp for schedule(dynamic, 8)
        for (int64_t t = 0; t < S; ++t) {
            attn_scores(t, d, q, ldq, k, ldk, s);
            const double l = attn_lse(t + 1, s);
            double D = 0.0;
            for (int64_t u = 0; u <= t; ++u) {
                p[t * S + u] = exp(s[u] - l);
                double dp = 0.0;
                for (int64_t e = 0; e < d; ++e) dp += dout[t * lddo + e] * v[u * ldv + e];
                ds[t * S + u] = dp;          /* dP for now */
                D += p[t * S + u] * dp;
            }
            for (int64_t u = 0; u <= t; ++u) ds[t * S + u] = p[t * S + u] * (ds[t * S + u] - D);
        }
        free(s);
    }
#pragma omp parallel for schedule(dynamic, 8)
    for (int64_t t = 0; t < S; ++t)
        for (int64_t e = 0; e < d; ++e) {
            double acc = 0.0;
            for (int64_t u = 0; u <= t; ++u) acc += ds[t * S + u] * k[u * ldk + e];
            dq[t * lddq + e] = acc * inv;
        }
#pragma omp parallel for schedule(dynamic, 8)
    for (int64_t u = 0; u < S; ++u)
        for (int64_t e = 0; e < d; ++e) {
            double ak = 0.0, av = 0.0;
            for (int64_t t = u; t < S; ++t) {
                ak += ds[t * S + u] * q[t * ldq + e];
                av += p[t * S + u] * dout[t * lddo + e];
            }
            dk[u * lddk + e] = ak * inv;
            dv[u * lddv + e] = av;
        }
    free(ds);
    free(p);
}
