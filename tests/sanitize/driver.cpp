// Host-side driver run under AddressSanitizer and UndefinedBehaviorSanitizer
// (test infrastructure).  It exercises the host code of the project on the
// CPU only: the oracle's C routines on small inputs, the mesh planner on
// valid and invalid inputs, and every argument check of the C ABI that
// returns before any device work (no HIP call is reached, no GPU is needed).
// Exit status 0 means every check below held and the sanitizers stayed
// silent (they abort on the first report).
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <vector>

#include "../../include/atp.h"
#include "../../oracle/oracle.h"

static int failures = 0;
#define EXPECT(cond)                                                          \
    do {                                                                      \
        if (!(cond)) {                                                        \
            fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__,      \
                    __LINE__, #cond);                                         \
            ++failures;                                                       \
        }                                                                     \
    } while (0)

static void oracle_routines() {
    // C = A B on a ragged shape, against a plain sum
    const int64_t M = 5, K = 7, N = 3;
    std::vector<double> A(M * K), B(K * N), C(M * N, -1.0);
    for (int64_t i = 0; i < M * K; ++i) A[i] = (double)((i * 7) % 5) - 2.0;
    for (int64_t i = 0; i < K * N; ++i) B[i] = (double)((i * 3) % 4) - 1.5;
    orc_matmul(M, K, N, A.data(), K, 1, B.data(), N, 1, C.data(), N, 1);
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < N; ++n) {
            double s = 0.0;
            for (int64_t k = 0; k < K; ++k) s += A[m * K + k] * B[k * N + n];
            EXPECT(C[m * N + n] == s);
        }
    // Partial(SUM) of three parts with bias + GeLU, the pre-activation saved
    const int64_t T = 4;
    std::vector<double> p0(T * N, 1.0), p1(T * N, 2.0), p2(T * N, -0.5), bias(N, 0.25),
        out(T * N), pre(T * N);
    const double* parts[3] = {p0.data(), p1.data(), p2.data()};
    orc_partial_reduce(3, parts, N, T, N, bias.data(), ORC_EPI_BIAS_GELU, nullptr, out.data(), N,
                       pre.data());
    for (int64_t i = 0; i < T * N; ++i) {
        EXPECT(pre[i] == 2.75);
        EXPECT(fabs(out[i] - orc_gelu(2.75)) < 1e-15);
    }
    EXPECT(orc_gelu(0.0) == 0.0);
    EXPECT(fabs(orc_gelu(1.5) - orc_gelu(-1.5) - 1.5) < 1e-15);
    EXPECT(orc_round_bf16(1.0 + 1.0 / 512.0) == 1.0);   // a tie rounds to even
    // causal attention of one head: a single token returns its value
    const int64_t S = 3, d = 4;
    std::vector<double> q(S * d), k(S * d), v(S * d), o(S * d), lse(S);
    for (int64_t i = 0; i < S * d; ++i) {
        q[i] = 0.1 * (double)(i % 5);
        k[i] = -0.2 * (double)(i % 3);
        v[i] = (double)i;
    }
    orc_attention_fwd(S, d, q.data(), d, k.data(), d, v.data(), d, o.data(), d, lse.data());
    for (int64_t e = 0; e < d; ++e) EXPECT(o[e] == v[e]);
    std::vector<double> dO(S * d, 1.0), dq(S * d), dk(S * d), dv(S * d);
    orc_attention_bwd(S, d, q.data(), d, k.data(), d, v.data(), d, dO.data(), d, dq.data(), d,
                      dk.data(), d, dv.data(), d);
    for (int64_t e = 0; e < d; ++e) {   // the keys' gradients sum to zero
        double s = 0.0;
        for (int64_t u = 0; u < S; ++u) s += dk[u * d + e];
        EXPECT(fabs(s) < 1e-12);
    }
}

static void planner() {
    atp_model_dims dims = {1, 4, 2048, 4096, 2};
    double t = 0.0;
    EXPECT(atp_tcomm(&dims, 2, 4, 1.2, 4.95, &t) == ATP_OK && t > 0.0);
    EXPECT(atp_tcomm(&dims, 8, 1, 0.97, INFINITY, &t) == ATP_OK && t > 0.0);
    EXPECT(atp_tcomm(&dims, 2, 4, 0.0, 4.95, &t) == ATP_ERR_INVALID_ARGUMENT);
    EXPECT(atp_tcomm(nullptr, 2, 4, 1.0, 1.0, &t) == ATP_ERR_INVALID_ARGUMENT);
    // two layers: 4 nodes of 4 GPUs
    std::vector<double> p2p(16, 300.0);
    atp_hcm_layer hcm[2] = {{4, 25.0, nullptr}, {4, 300.0, p2p.data()}};
    atp_mesh_cost best, costs[8];
    int32_t n = 0;
    EXPECT(atp_plan_mesh(hcm, 2, &dims, &best, costs, 8, &n) == ATP_OK && n == 5);
    EXPECT(best.d1 * best.d2 == 16 && best.t_comm > 0.0);
    EXPECT(atp_plan_mesh(hcm, 2, &dims, &best, costs, 2, &n) == ATP_ERR_INVALID_ARGUMENT);
    atp_mesh_cost one;
    EXPECT(atp_hcm_mesh_cost(hcm, 2, &dims, 8, 2, &one) == ATP_OK);
    EXPECT(atp_hcm_mesh_cost(hcm, 2, &dims, 8, 3, &one) == ATP_ERR_SHAPE);
    EXPECT(atp_hcm_mesh_cost(hcm, 0, &dims, 8, 2, &one) == ATP_ERR_INVALID_ARGUMENT);
    hcm[1].group_bw = -1.0;
    EXPECT(atp_hcm_mesh_cost(hcm, 2, &dims, 8, 2, &one) == ATP_ERR_INVALID_ARGUMENT);
}

// Pointers the checks see but never dereference.
static void* const FAKE = reinterpret_cast<void*>(0x10000);
static void* const MISALIGNED = reinterpret_cast<void*>(0x10004);

static void abi_checks() {
    atp_mesh m = {2, 2, 1, 0};
    atp_shard g, G[4];
    EXPECT(atp_shard_geometry(&m, ATP_COL_FIRST, 512, 2048, &g) == ATP_OK);
    EXPECT(g.k_loc == 256 && g.n_loc == 1024 && g.red_size == 2);
    EXPECT(atp_shard_geometry(&m, 7, 512, 2048, &g) == ATP_ERR_INVALID_ARGUMENT);
    EXPECT(atp_shard_geometry(&m, 0, 511, 2048, &g) == ATP_ERR_SHAPE);
    atp_mesh bad = {2, 2, 2, 0};
    EXPECT(atp_shard_geometry(&bad, 0, 512, 512, &g) == ATP_ERR_INVALID_ARGUMENT);
    EXPECT(strstr(atp_last_error(), "outside") != nullptr);
    EXPECT(atp_block_geometry(&m, ATP_BLOCK_COL, 512, G) == ATP_OK);
    EXPECT(atp_block_geometry(&m, ATP_BLOCK_COL, 500, G) == ATP_ERR_UNSUPPORTED);
    int32_t first = 0, count = 0, per = 0;
    EXPECT(atp_attention_heads(&m, ATP_BLOCK_COL, 1024, 8, &first, &count, &per) == ATP_OK);
    EXPECT(per == 4 && count == 2 && first == 0);
    EXPECT(atp_attention_heads(&m, ATP_BLOCK_COL, 1024, 16, &first, &count, &per) ==
           ATP_ERR_UNSUPPORTED);

    // shard linear: every refusal before device work
    EXPECT(atp_shard_linear_fwd(&m, 1, 64, 512, 2048, 3, FAKE, 256, FAKE, 1024, nullptr, 0, FAKE,
                                0, 1024, nullptr, nullptr, nullptr) == ATP_ERR_SHAPE);
    EXPECT(atp_shard_linear_fwd(&m, 1, 64, 512, 2048, 2, MISALIGNED, 256, FAKE, 1024, nullptr, 0,
                                FAKE, 0, 1024, nullptr, nullptr, nullptr) == ATP_ERR_UNSUPPORTED);
    EXPECT(atp_shard_linear_fwd(&m, 1, 64, 512, 2048, 2, FAKE, 256, FAKE, 1024, nullptr,
                                ATP_EPI_BIAS, FAKE, 0, 1024, nullptr, nullptr, nullptr) ==
           ATP_ERR_INVALID_ARGUMENT);   // an epilogue on a Partial(SUM) block
    const float* parts[2] = {static_cast<const float*>(FAKE), nullptr};
    EXPECT(atp_chunked_partial_reduce(2, 64, 256, 2, parts, 256, nullptr, 0, nullptr, FAKE, 0, 256,
                                      nullptr, nullptr, nullptr) == ATP_ERR_INVALID_ARGUMENT);
    EXPECT(atp_chunked_partial_reduce(ATP_MAX_GROUP + 1, 64, 256, 2, parts, 256, nullptr, 0,
                                      nullptr, FAKE, 0, 256, nullptr, nullptr, nullptr) ==
           ATP_ERR_UNSUPPORTED);
    EXPECT(atp_transpose_bf16(-1, 8, FAKE, 8, FAKE, 8, nullptr) == ATP_ERR_INVALID_ARGUMENT);
    EXPECT(atp_transpose_bf16(8, 8, FAKE, 8, FAKE, 8, nullptr) == ATP_ERR_INVALID_ARGUMENT);

    // block calls: layout, partial dtype, a missing table, a short leading dimension
    const int64_t h = 512, T = 256;
    atp_block_weights W;
    memset(&W, 0, sizeof W);
    for (int i = 0; i < 4; ++i) {
        W.w[i] = FAKE;
        W.ldw[i] = G[i].n_loc;
        W.b[i] = FAKE;
    }
    atp_block_fwd_io io;
    memset(&io, 0, sizeof io);
    io.x_loc = FAKE;    io.ldx = G[0].k_loc;
    io.attn_loc = FAKE; io.lda = G[1].k_loc;
    io.qkv = FAKE;      io.ld_qkv = G[0].n_loc;
    io.o = FAKE;        io.ld_o = G[1].n_loc;
    io.h = FAKE;        io.ld_h = G[2].n_loc;
    io.pre = FAKE;
    io.z = FAKE;        io.ld_z = G[3].n_loc;
    void* tabs[4][2];
    for (int i = 0; i < 4; ++i) {
        tabs[i][0] = tabs[i][1] = FAKE;
        io.partials[i] = tabs[i];
        io.ldp[i] = G[i].n_loc;
    }
    W.layout = 5;
    EXPECT(atp_block_fwd(&m, 0, T, h, 2, &W, &io, nullptr, 0, nullptr, nullptr) ==
           ATP_ERR_INVALID_ARGUMENT);
    W.layout = ATP_W_KN;
    io.partial_dtype = 9;
    EXPECT(atp_block_fwd(&m, 0, T, h, 2, &W, &io, nullptr, 0, nullptr, nullptr) ==
           ATP_ERR_INVALID_ARGUMENT);
    io.partial_dtype = ATP_F32;
    io.partials[3] = nullptr;
    EXPECT(atp_block_fwd(&m, 0, T, h, 2, &W, &io, nullptr, 0, nullptr, nullptr) ==
           ATP_ERR_INVALID_ARGUMENT);
    io.partials[3] = tabs[3];
    io.ld_h = G[2].n_loc - 8;
    EXPECT(atp_block_fwd(&m, 0, T, h, 2, &W, &io, nullptr, 0, nullptr, nullptr) ==
           ATP_ERR_INVALID_ARGUMENT);
    EXPECT(atp_block_fwd(&m, 0, T, h, 3, &W, &io, nullptr, 0, nullptr, nullptr) == ATP_ERR_SHAPE);
    atp_block_bwd_io bio;
    memset(&bio, 0, sizeof bio);
    EXPECT(atp_block_bwd(&m, 0, T, h, 2, &W, &bio, nullptr, 0, nullptr, nullptr) ==
           ATP_ERR_INVALID_ARGUMENT);
    EXPECT(atp_block_workspace_bytes(&m, 0, T, h, 2, ATP_W_NK) >
           atp_block_workspace_bytes(&m, 0, T, h, 2, ATP_W_KN) / 2);
    EXPECT(atp_block_workspace_path(&m, 0, T, h, ATP_W_KN, 0, 0) == 0);
    EXPECT(atp_block_workspace_path(&m, 0, 132, h, ATP_W_KN, (size_t)1 << 40, 1) == 0);
    EXPECT(atp_block_workspace_path(&m, 0, T, h, 3, 1, 0) == -1);

    // attention calls and the attention block
    atp_attn_block_fwd_io aio;
    memset(&aio, 0, sizeof aio);
    EXPECT(atp_attention_block_fwd(&m, 0, 2, 128, 1024, 8, 3, &W, &aio, nullptr, 0, nullptr,
                                   nullptr) ==
           ATP_ERR_SHAPE);
    EXPECT(atp_attention_block_fwd(&m, 0, 2, 128, 1024, 8, 2, nullptr, &aio, nullptr, 0,
                                   nullptr, nullptr) ==
           ATP_ERR_INVALID_ARGUMENT);
    EXPECT(atp_attention_fwd(&m, 0, 1, 64, 1024, 8, FAKE, 1536, FAKE, 512, nullptr, nullptr) ==
           ATP_ERR_INVALID_ARGUMENT);   // lse missing
    EXPECT(atp_attention_fwd(&m, 0, 1, 64, 1024, 4, FAKE, 1536, FAKE, 512, nullptr, nullptr) ==
           ATP_ERR_UNSUPPORTED);         // head dimension 256

    // status strings and the profile log with nothing recorded
    EXPECT(strcmp(atp_status_string(ATP_ERR_SHAPE), "ATP_ERR_SHAPE") == 0);
    EXPECT(strcmp(atp_status_string(42), "ATP_ERR_UNKNOWN") == 0);
    atp_kernel_stat st[2];
    EXPECT(atp_profile_collect(st, 2) == 0);
}

int main() {
    oracle_routines();
    planner();
    abi_checks();
    if (failures) {
        fprintf(stderr, "%d expectation(s) failed\n", failures);
        return 1;
    }
    printf("sanitized host checks passed\n");
    return 0;
}
