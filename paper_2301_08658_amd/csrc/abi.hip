// C ABI of the ATP shard-block library: argument checking, shard geometry
// (Sec. 3.2), and the two-stream chunk pipeline (Sec. 4.1, Sec. 4.2) that
// drives the gfx950 kernels.  Declarations and contracts: include/atp.h.
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/atp.h"
#include "errors.h"
#include "kernels.h"

namespace {
thread_local std::string g_last_error;
}  // namespace

namespace atp {
atp_status set_error(atp_status s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}
}  // namespace atp

namespace {

using atp::set_error;

atp_status hip_fail(hipError_t e, const char* what) {
    return set_error(ATP_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

#define ATP_CHECK(expr)                                   \
    do {                                                  \
        atp_status _s = (expr);                           \
        if (_s != ATP_OK) return _s;                      \
    } while (0)

#define HIP_CHECK(expr, what)                             \
    do {                                                  \
        hipError_t _e = (expr);                           \
        if (_e != hipSuccess) return hip_fail(_e, what);  \
    } while (0)

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

atp_status check_mesh(const atp_mesh* m) {
    if (!m) return set_error(ATP_ERR_INVALID_ARGUMENT, "mesh is NULL");
    if (m->d1 <= 0 || m->d2 <= 0)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "mesh dims must be positive (d1=%d d2=%d)", m->d1,
                    m->d2);
    if (m->i1 < 0 || m->i1 >= m->d1 || m->i2 < 0 || m->i2 >= m->d2)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "coordinate (%d,%d) outside mesh (%d,%d)", m->i1,
                    m->i2, m->d1, m->d2);
    return ATP_OK;
}

atp_status geometry(const atp_mesh* m, int32_t mode, int64_t k, int64_t n, atp_shard* g) {
    ATP_CHECK(check_mesh(m));
    if (mode != ATP_ROW_FIRST && mode != ATP_COL_FIRST)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "mode %d is neither row- nor column-first", mode);
    if (k <= 0 || n <= 0) return set_error(ATP_ERR_INVALID_ARGUMENT, "k and n must be positive");
    // Row-first: W [Shard(0), Shard(1)] -> rows split by d1, columns by d2,
    // output partial over mesh axis 0.  Column-first: W [Shard(1), Shard(0)]
    // -> columns split by d1, rows by d2, output partial over mesh axis 1.
    const bool row = (mode == ATP_ROW_FIRST);
    const int32_t dk = row ? m->d1 : m->d2;   // splits k
    const int32_t dn = row ? m->d2 : m->d1;   // splits n
    const int32_t ik = row ? m->i1 : m->i2;
    const int32_t in = row ? m->i2 : m->i1;
    if (k % dk != 0 || n % dn != 0)
        return set_error(ATP_ERR_SHAPE, "k=%lld not divisible by %d or n=%lld not divisible by %d",
                    (long long)k, dk, (long long)n, dn);
    g->k_loc = k / dk;
    g->n_loc = n / dn;
    g->k_off = (int64_t)ik * g->k_loc;
    g->n_off = (int64_t)in * g->n_loc;
    g->red_axis = row ? 0 : 1;
    g->red_size = dk;
    g->red_index = ik;
    g->bwd_axis = row ? 1 : 0;
    g->bwd_size = dn;
    g->bwd_index = in;
    return ATP_OK;
}

atp_status check_chunks(int64_t tokens, int32_t chunks) {
    if (tokens < 0) return set_error(ATP_ERR_INVALID_ARGUMENT, "tokens must be >= 0");
    if (chunks < 1 || chunks > ATP_MAX_CHUNKS)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "chunks=%d outside [1, %d]", chunks,
                    ATP_MAX_CHUNKS);
    if (tokens % chunks != 0)
        return set_error(ATP_ERR_SHAPE, "tokens=%lld not divisible by chunks=%d", (long long)tokens,
                    chunks);
    return ATP_OK;
}

// A matrix with zero rows is never touched and may be NULL.
// `any_cols`: the column count need not be a multiple of 8 (the leading
// dimension still must), for kernels that handle ragged rows element-wise.
atp_status check_mat(const void* p, int64_t rows, int64_t ld, int64_t cols, const char* name,
                     bool any_cols = false) {
    if (ld > (int64_t)1 << 22)
        return set_error(ATP_ERR_UNSUPPORTED, "%s: leading dimension %lld above 4M elements", name,
                    (long long)ld);
    if (rows == 0 && !p) return ATP_OK;
    if (!p) return set_error(ATP_ERR_INVALID_ARGUMENT, "%s is NULL", name);
    if (ld < cols) return set_error(ATP_ERR_INVALID_ARGUMENT, "%s: ld %lld < %lld columns", name,
                               (long long)ld, (long long)cols);
    if (!aligned16(p)) return set_error(ATP_ERR_UNSUPPORTED, "%s is not 16-byte aligned", name);
    if (ld % 8 != 0 || (!any_cols && cols % 8 != 0))
        return set_error(ATP_ERR_UNSUPPORTED, "%s: ld %lld and columns %lld must be multiples of 8",
                    name, (long long)ld, (long long)cols);
    return ATP_OK;
}

atp_status check_vec(const void* p, const char* name) {
    if (!p) return set_error(ATP_ERR_INVALID_ARGUMENT, "%s is NULL", name);
    if (!aligned16(p)) return set_error(ATP_ERR_UNSUPPORTED, "%s is not 16-byte aligned", name);
    return ATP_OK;
}

// Whether two row-major buffers (rows x ld elements of the given sizes) share
// any byte; NULL or empty buffers overlap nothing.
bool overlaps(const void* a, int64_t rows_a, int64_t ld_a, size_t esz_a, const void* b,
              int64_t rows_b, int64_t ld_b, size_t esz_b) {
    if (!a || !b || rows_a == 0 || rows_b == 0) return false;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    const uintptr_t a1 = a0 + (uintptr_t)(rows_a * ld_a) * esz_a;
    const uintptr_t b1 = b0 + (uintptr_t)(rows_b * ld_b) * esz_b;
    return a0 < b1 && b0 < a1;
}

bool valid_epi(int32_t e) { return e >= ATP_EPI_NONE && e <= ATP_EPI_GELU_BWD; }
bool valid_dtype(int32_t d) { return d == ATP_F32 || d == ATP_BF16; }

// ---------------------------------------------------------------------------
// events: synchronisation events per host thread and device, and timing records
// ---------------------------------------------------------------------------
std::mutex g_mu;   // guards the timing records below

// The block calls order their streams with events taken from a pool that
// belongs to the calling host thread (one pool per device), so calls from
// different threads never share an event, and the pool of a thread can
// only grow between that thread's calls (no reallocation while a call uses
// it).  A thread's events are re-recorded by its next call, which is
// correct because a wait refers to the record enqueued before it.  The
// events are not destroyed when a thread exits (the HIP runtime may already
// be shutting down then); each thread holds at most one pool per device.
thread_local std::map<int, std::vector<hipEvent_t>> t_sync_events;   // device -> pool

atp_status sync_events(size_t count, hipEvent_t** out) {
    int dev = 0;
    HIP_CHECK(hipGetDevice(&dev), "hipGetDevice");
    auto& pool = t_sync_events[dev];
    while (pool.size() < count) {
        hipEvent_t e;
        HIP_CHECK(hipEventCreateWithFlags(&e, hipEventDisableTiming), "hipEventCreateWithFlags");
        pool.push_back(e);
    }
    *out = pool.data();
    return ATP_OK;
}

// A second compute stream of the calling host thread on the current device
// (created on first use, default priority, never destroyed: like the event
// pool it may outlive the runtime's shutdown).  The forward puts every other
// chunk product of a linear on it, so one chunk's 160 tiles of 256 x 256 can
// start on the CUs the previous chunk leaves idle.
thread_local std::map<int, hipStream_t> t_lane2;   // device -> stream
atp_status second_lane(hipStream_t* out) {
    int dev = 0;
    HIP_CHECK(hipGetDevice(&dev), "hipGetDevice");
    auto it = t_lane2.find(dev);
    if (it == t_lane2.end()) {
        hipStream_t s = nullptr;
        HIP_CHECK(hipStreamCreateWithFlags(&s, hipStreamNonBlocking), "hipStreamCreateWithFlags");
        it = t_lane2.emplace(dev, s).first;
    }
    *out = it->second;
    return ATP_OK;
}

struct ProfRec {
    std::string name;
    hipEvent_t beg, end;
    double flops, bytes;
};
bool g_prof_on = false;
bool g_prof_detail = false;   // key records by kernel and problem shape
std::vector<ProfRec> g_prof;
std::vector<hipEvent_t> g_prof_free;

hipEvent_t prof_event() {
    if (!g_prof_free.empty()) {
        hipEvent_t e = g_prof_free.back();
        g_prof_free.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// Run `launch` on stream s, bracketed by timing events when profiling is on.
template <class F>
atp_status timed(const std::string& name, double flops, double bytes, hipStream_t s,
                 F&& launch) {
    hipEvent_t b = nullptr, e = nullptr;
    if (g_prof_on) {
        std::lock_guard<std::mutex> lk(g_mu);
        b = prof_event();
        e = prof_event();
        if (b) (void)hipEventRecord(b, s);
    }
    hipError_t err = launch();
    if (err != hipSuccess) return hip_fail(err, name.c_str());
    if (b && e) {
        (void)hipEventRecord(e, s);
        std::lock_guard<std::mutex> lk(g_mu);
        g_prof.push_back(ProfRec{name, b, e, flops, bytes});
    }
    return ATP_OK;
}

atp_status run_gemm(const atp::GemmProblem& p, hipStream_t s) {
    if (p.M <= 0 || p.N <= 0) return ATP_OK;
    const double flops = 2.0 * (double)p.M * (double)p.N * (double)p.K;
    const double bytes = 2.0 * ((double)p.M * p.K + (double)p.K * p.N) +
                         (double)p.M * p.N * (p.out_bf16 ? 2.0 : 4.0) +
                         ((p.epi == atp::EPI_GELU_BWD || p.pre_out) ? 2.0 * p.M * p.N : 0.0);
    // one name per kernel instantiation: layout, epilogue, output type
    std::string name = atp::gemm_kernel_name(p);
    name += "_e" + std::to_string(p.epi) + (p.out_bf16 ? "_bf16" : "_f32");
    if (g_prof_on && g_prof_detail) {
        char buf[96];
        snprintf(buf, sizeof buf, " %lldx%lldx%lld", (long long)p.M, (long long)p.N,
                 (long long)p.K);
        name += buf;
    }
    return timed(name, flops, bytes, s, [&] { return atp::launch_gemm(p, s); });
}

atp_status run_reduce(const atp::ReduceProblem& p, hipStream_t s) {
    if (p.rows <= 0 || p.ncols <= 0) return ATP_OK;
    const double el = (double)p.rows * (double)p.ncols;
    const double bytes = el * ((p.parts_bf16 ? 2.0 : 4.0) * p.nparts + (p.out_bf16 ? 2.0 : 4.0)) +
                         ((p.epi == atp::EPI_GELU_BWD || p.pre_out) ? 2.0 * el : 0.0);
    std::string name = "partial_reduce";
    if (g_prof_on && g_prof_detail) {
        char buf[96];
        snprintf(buf, sizeof buf, " %dx%lldx%lld e%d", p.nparts, (long long)p.rows,
                 (long long)p.ncols, p.epi);
        name += buf;
    }
    return timed(name, 0.0, bytes, s, [&] { return atp::launch_reduce(p, s); });
}

atp_status run_colsum(const void* dy, int64_t ld, int64_t T, int64_t N, float* db,
                      hipStream_t s) {
    return timed("colsum", (double)T * N, 2.0 * T * N + 4.0 * N, s,
                 [&] { return atp::launch_colsum(dy, ld, T, N, db, s); });
}

// The S split-K slabs of an fp32 product summed into its destination rows
// (fp32, or bf16 rounded once).
atp_status run_split_sum(const float* ws, int S, int64_t rows, int64_t cols, void* out,
                         int64_t ldo, bool out_bf16, hipStream_t s) {
    if (rows <= 0 || cols <= 0) return ATP_OK;
    const double el = (double)rows * (double)cols;
    return timed("split_sum", 0.0, el * (4.0 * S + (out_bf16 ? 2.0 : 4.0)), s, [&] {
        return atp::launch_split_sum(ws, S, rows * cols, cols, rows, cols, out, ldo, out_bf16, s);
    });
}

atp::GemmProblem gemm_problem(int layout, const void* A, int64_t lda, const void* B, int64_t ldb,
                              void* C, int64_t ldc, bool out_bf16, int epi, int64_t M,
                              int64_t N, int64_t K) {
    atp::GemmProblem p;
    p.layout = layout;
    p.A = A; p.lda = lda;
    p.B = B; p.ldb = ldb;
    p.C = C; p.ldc = ldc;
    p.out_bf16 = out_bf16;
    p.epi = epi;
    p.bias = nullptr;
    p.pre_in = nullptr;
    p.pre_out = nullptr;
    p.M = M; p.N = N; p.K = K;
    return p;
}

// parts: any array of nparts device pointers (fp32, or bf16 with parts_bf16)
template <class PartTable>
atp::ReduceProblem reduce_problem(int nparts, PartTable parts, int64_t ldp,
                                  int64_t row0, int64_t rows, int64_t ncols, int epi,
                                  const void* bias, const void* pre_in, void* out, int64_t ldo,
                                  bool out_bf16, void* pre_out, bool parts_bf16 = false) {
    atp::ReduceProblem p;
    memset(&p, 0, sizeof p);
    p.nparts = nparts;
    p.parts_bf16 = parts_bf16;
    for (int j = 0; j < nparts; ++j) p.parts[j] = parts[j];
    p.ldp = ldp;
    p.row0 = row0;
    p.rows = rows;
    p.ncols = ncols;
    p.epi = epi;
    p.bias = bias;
    p.pre_in = pre_in;
    p.out = out;
    p.ldo = ldo;
    p.out_bf16 = out_bf16;
    p.pre_out = pre_out;
    return p;
}

// Block-level linear plan: index 0..3 = qkv, out, fc1, fc2.
struct BlockPlan {
    atp_shard g[4];
    int32_t mode[4];
    int64_t K[4], N[4];
};

atp_status block_plan(const atp_mesh* m, int32_t bm, int64_t h, BlockPlan* p) {
    if (bm != ATP_BLOCK_COL && bm != ATP_BLOCK_ROW)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "block mode %d unknown", bm);
    if (h <= 0) return set_error(ATP_ERR_INVALID_ARGUMENT, "h must be positive");
    const int32_t pc = ATP_COL_FIRST, pr = ATP_ROW_FIRST;
    const int32_t modes_col[4] = {pc, pr, pc, pr};
    const int32_t modes_row[4] = {pr, pc, pr, pc};
    const int64_t K[4] = {h, h, h, 4 * h};
    const int64_t N[4] = {3 * h, h, 4 * h, h};
    for (int i = 0; i < 4; ++i) {
        p->mode[i] = (bm == ATP_BLOCK_COL) ? modes_col[i] : modes_row[i];
        p->K[i] = K[i];
        p->N[i] = N[i];
        ATP_CHECK(geometry(m, p->mode[i], K[i], N[i], &p->g[i]));
        if (p->g[i].k_loc % 8 || p->g[i].n_loc % 8)
            return set_error(ATP_ERR_UNSUPPORTED, "local block %lldx%lld of linear %d: sizes must be "
                        "multiples of 8", (long long)p->g[i].k_loc, (long long)p->g[i].n_loc, i);
    }
    return ATP_OK;
}

// Workspace of the block calls.  The forward keeps W^T of the four linears
// ([n_loc][k_loc]); the backward keeps X^T of x (shared by QKV and fc1), the
// attention block and H, and dY^T of the four linears, each [cols][tokens]:
// with them every product runs with both operands contiguous along k, the
// layout the GEMM kernel streams fastest.  Each side adds the split-K slabs
// of its chunk products.  Pieces are 256-byte aligned.
constexpr size_t kWsAlign = 256;
size_t ws_round(size_t b) { return (b + kWsAlign - 1) / kWsAlign * kWsAlign; }

// Row pitch (elements) of a transposed copy whose rows hold `len` values.
// Copies are padded by 128 bytes per row: with dense pitches such as 20480
// or 5120 bytes, the rows that the XCDs read at one k offset land on few
// memory channels, and a product streaming them runs 8-13% slower.
constexpr int64_t kWsPad = 64;
int64_t ws_pitch(int64_t len) { return len + kWsPad; }

// Split-K slabs of the chunked products that feed a reduction: the forward
// X W of a linear whose reduction group has several members, the backward
// dY W^T likewise.  One region serves every chunk of every linear (they run
// in order on one stream); it is sized for the largest plan over all chunk
// counts, so the size does not depend on the chunk count.
size_t slab_bytes(const BlockPlan& P, int64_t tokens, bool bwd, int nlin = 4) {
    size_t most = 0;
    for (int c = 1; c <= ATP_MAX_CHUNKS; ++c) {
        if (tokens % c) continue;
        const int64_t mc = tokens / c;
        for (int L = 0; L < nlin; ++L) {
            const atp_shard& g = P.g[L];
            if ((bwd ? g.bwd_size : g.red_size) <= 1) continue;
            const int64_t N = bwd ? g.k_loc : g.n_loc, K = bwd ? g.n_loc : g.k_loc;
            int64_t ks = 0;
            const int S = atp::nt_split_plan(mc, N, K, &ks);
            if (S > 1) most = std::max(most, (size_t)S * mc * N * 4);
        }
    }
    return most;
}

bool valid_layout(int32_t l) { return l == ATP_W_KN || l == ATP_W_NK; }

// True when the forward of linear L with `chunks` chunks reads weights
// stored [k][n] as they are on the workspace path: its products stream NN
// as fast as NT from a W^T copy and are not split over k.  A linear whose
// group has one member runs one product over all tokens; the others run one
// product per chunk.  Otherwise the forward first copies W^T into the
// workspace.
bool fwd_reads_w(const BlockPlan& P, int L, int64_t tokens, int chunks) {
    const atp_shard& g = P.g[L];
    if (g.red_size <= 1) return atp::nn_streams_like_nt(tokens, g.n_loc);
    const int64_t mc = tokens / chunks;
    int64_t ks = 0;
    return atp::nt_split_plan(mc, g.n_loc, g.k_loc, &ks) <= 1 &&
           atp::nn_streams_like_nt(mc, g.n_loc);
}

// True when some chunk count makes the forward of linear L copy W^T (the
// workspace holds its copy whatever the chunk count, as for the slabs).
bool fwd_may_copy_w(const BlockPlan& P, int L, int64_t tokens) {
    for (int c = 1; c <= ATP_MAX_CHUNKS; ++c)
        if (tokens % c == 0 && !fwd_reads_w(P, L, tokens, c)) return true;
    return false;
}

// The forward's pieces: the slabs, and W^T ([n_loc][k_loc]) of weights
// stored [k_loc][n_loc] that the forward may copy (weights stored
// [n_loc][k_loc] are read as they are).
// (nlin = 2: the attention block's QKV and out-proj only, a subset)
size_t ws_fwd_bytes(const BlockPlan& P, int64_t tokens, int32_t layout, int nlin = 4) {
    size_t b = ws_round(slab_bytes(P, tokens, false, nlin));
    if (layout == ATP_W_KN)
        for (int L = 0; L < nlin; ++L)
            if (fwd_may_copy_w(P, L, tokens))
                b += ws_round((size_t)P.g[L].n_loc * ws_pitch(P.g[L].k_loc) * 2);
    return b;
}

// One [k_loc][n_loc] copy of a weight stored [n_loc][k_loc], for the dX
// products of the backward; sized for the largest weight, reused linear by
// linear (every use is on the compute stream, in order).
size_t wkn_bytes(const BlockPlan& P) {
    size_t most = 0;
    for (int L = 0; L < 4; ++L)
        most = std::max(most, (size_t)P.g[L].k_loc * ws_pitch(P.g[L].n_loc) * 2);
    return most;
}

// fp32 column partials of dY, one row per 64 tokens, for the widest linear
size_t colpart_bytes(const BlockPlan& P, int64_t tokens) {
    int64_t n = 0;
    for (int L = 0; L < 4; ++L) n = std::max(n, P.g[L].n_loc);
    return (size_t)((tokens + 63) / 64) * (size_t)n * 4;
}

size_t ws_bwd_bytes(const BlockPlan& P, int64_t tokens, int32_t layout) {
    const size_t t2 = (size_t)ws_pitch(tokens) * 2;
    size_t b = ws_round(P.g[0].k_loc * t2) + ws_round(P.g[1].k_loc * t2) +
               ws_round(P.g[3].k_loc * t2) + ws_round(slab_bytes(P, tokens, true)) +
               ws_round(colpart_bytes(P, tokens));
    for (int L = 0; L < 4; ++L) b += ws_round(P.g[L].n_loc * t2);
    if (layout == ATP_W_NK) b += ws_round(wkn_bytes(P));
    return b;
}

// True when a call of the pass (0 forward, 1 backward) with a workspace of
// ws_bytes bytes takes the transposed-layout path.
bool takes_ws_path(const BlockPlan& P, int64_t tokens, int32_t layout, size_t ws_bytes,
                   int pass) {
    if (ws_bytes == 0) return false;
    if (pass == 0) return ws_bytes >= ws_fwd_bytes(P, tokens, layout);
    return ws_bytes >= ws_bwd_bytes(P, tokens, layout) && tokens % 8 == 0;
}

// A partial product [M, N] over K (fp32, or bf16 when p.out_bf16): split
// over K into `slab` when a slab is given and the plan says so, the splits'
// fp32 slabs then summed in split order into C (rounded once to bf16 for a
// bf16 partial).
atp_status run_nt_partial(atp::GemmProblem p, float* slab, hipStream_t s) {
    int64_t ks = 0;
    const int S = slab ? atp::nt_split_plan(p.M, p.N, p.K, &ks) : 1;
    if (S <= 1) return run_gemm(p, s);
    void* out = p.C;
    const int64_t ldo = p.ldc;
    const bool b16 = p.out_bf16;
    p.C = slab;
    p.ldc = p.N;
    p.out_bf16 = false;
    p.splits = S;
    p.ksplit = ks;
    p.c_split = p.M * p.N;
    ATP_CHECK(run_gemm(p, s));
    return run_split_sum(slab, S, p.M, p.N, out, ldo, b16, s);
}

// Carves consecutive aligned pieces out of the caller's workspace.
struct Carver {
    char* p;
    uint16_t* take(size_t bytes) {
        uint16_t* r = reinterpret_cast<uint16_t*>(p);
        p += ws_round(bytes);
        return r;
    }
};

atp_status run_transpose(const void* src, int64_t lds, int64_t rows, int64_t cols, void* dst,
                         int64_t ldd, hipStream_t s, float* part = nullptr, int64_t ldpart = 0) {
    return timed("transpose", 0.0, 4.0 * (double)rows * (double)cols, s, [&] {
        return atp::launch_transpose(src, lds, rows, cols, dst, ldd, s, part, ldpart);
    });
}

// db from the 64-row-block column partials a transpose wrote
atp_status run_colsum_finish(const float* part, int64_t ldp, int64_t nb, int64_t N, float* db,
                             hipStream_t s) {
    return timed("colsum", (double)nb * N, 4.0 * (nb + 1) * (double)N, s,
                 [&] { return atp::launch_colsum_finish(part, ldp, nb, N, db, s); });
}

atp_status check_group(void* const* tab, int32_t size, int64_t rows, int64_t ld, int64_t cols,
                       const char* name) {
    if (size > ATP_MAX_GROUP)
        return set_error(ATP_ERR_UNSUPPORTED, "%s: group of %d exceeds %d", name, size,
                    ATP_MAX_GROUP);
    if (size == 1) return ATP_OK;
    if (!tab) return set_error(ATP_ERR_INVALID_ARGUMENT, "%s: pointer table is NULL", name);
    for (int j = 0; j < size; ++j) {
        char nm[64];
        snprintf(nm, sizeof nm, "%s[%d]", name, j);
        ATP_CHECK(check_mat(tab[j], rows, ld, cols, nm));
    }
    return ATP_OK;
}

const char* const kLinearName[4] = {"qkv", "out", "fc1", "fc2"};

// The block's streams: the compute stream (cs), on which every GEMM, split
// sum and column sum runs in issue order, and the comm stream (ms) that runs
// the chunk reductions.  The GEMM kernel's tiles fill the chip by
// themselves (a 512-row chunk is one tile per CU), so a kernel beside one
// delays its last tiles (measured: a second GEMM stream, or transposes and
// column sums beside the GEMMs, made the step 3-6% slower); only the
// reductions, which overlap by design, run beside them.
struct Streams {
    hipStream_t cs, ms;
    Streams(void* c, void* m) : cs(static_cast<hipStream_t>(c)), ms(static_cast<hipStream_t>(m)) {}

    // everything already queued on cs happens before the block's work
    atp_status begin(hipEvent_t start) const {
        HIP_CHECK(hipEventRecord(start, cs), "hipEventRecord");
        if (ms != cs) HIP_CHECK(hipStreamWaitEvent(ms, start, 0), "hipStreamWaitEvent");
        return ATP_OK;
    }
    // cs is ordered after all of the block's work on ms
    atp_status end(hipEvent_t ms_end) const {
        if (ms != cs) {
            HIP_CHECK(hipEventRecord(ms_end, ms), "hipEventRecord");
            HIP_CHECK(hipStreamWaitEvent(cs, ms_end, 0), "hipStreamWaitEvent");
        }
        return ATP_OK;
    }
};

// Capturing a block call on its direct path (no usable workspace) into a HIP
// graph once made hipStreamEndCapture crash inside the runtime (a host
// segmentation fault, at a time when that path also ran GEMMs on a second
// stream; the cause was never identified), so a call that would take the
// direct path refuses a capturing compute stream, before it enqueues
// anything.  Calls on the workspace path are captured and replayed bit for
// bit (tested).
atp_status refuse_capture_of_direct_path(void* compute_stream) {
    hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
    HIP_CHECK(hipStreamIsCapturing(static_cast<hipStream_t>(compute_stream), &st),
              "hipStreamIsCapturing");
    if (st != hipStreamCaptureStatusNone)
        return set_error(ATP_ERR_UNSUPPORTED,
                         "graph capture needs the workspace path (a workspace of "
                         "atp_block_workspace_bytes bytes; the backward also needs "
                         "tokens %% 8 == 0)");
    return ATP_OK;
}

double gemm_flops(int64_t m, int64_t n, int64_t k) { return 2.0 * (double)m * (double)n * (double)k; }

// One device's share of the attention core (Sec. 3.2.1): its QKV block holds
// heads_blk whole heads ([q | k | v] columns each); the block is replicated
// over the group that reduced it, and member j of that group takes the j-th
// of red_size equal runs of heads.
constexpr int kHeadDim = 128;
struct AttnPlan {
    int64_t T, qkv_cols, out_cols;
    int heads_blk, hd, first;
};

atp_status attention_plan(const atp_mesh* mesh, int32_t bm, int64_t batch, int64_t seq,
                          int64_t h, int32_t heads, AttnPlan* ap) {
    ATP_CHECK(check_mesh(mesh));
    BlockPlan P;
    ATP_CHECK(block_plan(mesh, bm, h, &P));
    if (batch < 0 || seq < 0) return set_error(ATP_ERR_INVALID_ARGUMENT, "negative batch or seq");
    if (seq > (1 << 24) || batch > (1 << 24))
        return set_error(ATP_ERR_UNSUPPORTED, "batch and seq must be at most 2^24");
    if (heads <= 0 || h % heads)
        return set_error(ATP_ERR_SHAPE, "h=%lld is not a multiple of heads=%d", (long long)h, heads);
    if (h / heads != kHeadDim)
        return set_error(ATP_ERR_UNSUPPORTED, "head dimension %lld: only %d is built",
                         (long long)(h / heads), kHeadDim);
    const atp_shard& g = P.g[0];
    if (g.n_loc % (3 * kHeadDim))
        return set_error(ATP_ERR_SHAPE, "the QKV block (%lld columns) does not hold whole heads",
                         (long long)g.n_loc);
    ap->heads_blk = (int)(g.n_loc / (3 * kHeadDim));
    if (ap->heads_blk % g.red_size)
        return set_error(ATP_ERR_SHAPE, "%d heads of the QKV block do not divide over a group of %d",
                         ap->heads_blk, g.red_size);
    ap->hd = ap->heads_blk / g.red_size;
    ap->first = g.red_index * ap->hd;
    ap->T = batch * seq;
    ap->qkv_cols = g.n_loc;
    ap->out_cols = (int64_t)ap->heads_blk * kHeadDim;
    return ATP_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// Scratch of atp_attention_bwd_noalloc: the attention backward's delta lives
// in this file-scope device array instead of a caller buffer.  Every GPU the
// library runs on holds its own copy (4 MiB) until the process ends; host
// code never uses the array's name as an address, only the per-device
// address that hipGetSymbolAddress returns with that device current.
// ---------------------------------------------------------------------------
constexpr int64_t kNoAllocDeltaMax = (int64_t)1 << 20;   // floats
static __device__ __align__(256) float scratch[kNoAllocDeltaMax];

namespace {
std::mutex g_scratch_mu;
std::map<int, float*> g_scratch_ptr;   // device -> its copy of `scratch`

// The current device's copy of `scratch`, looked up once per device.
atp_status noalloc_scratch(float** out) {
    int dev = 0;
    HIP_CHECK(hipGetDevice(&dev), "hipGetDevice");
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    auto it = g_scratch_ptr.find(dev);
    if (it == g_scratch_ptr.end()) {
        void* ptr = nullptr;
        HIP_CHECK(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)), "hipGetSymbolAddress");
        if (!ptr) return set_error(ATP_ERR_DEVICE, "hipGetSymbolAddress gave a NULL address");
        it = g_scratch_ptr.emplace(dev, static_cast<float*>(ptr)).first;
    }
    *out = it->second;
    return ATP_OK;
}
}  // namespace

// ===========================================================================
// exported
// ===========================================================================
extern "C" {

const char* atp_status_string(int32_t s) {
    switch (s) {
    case ATP_OK: return "ATP_OK";
    case ATP_ERR_INVALID_ARGUMENT: return "ATP_ERR_INVALID_ARGUMENT";
    case ATP_ERR_SHAPE: return "ATP_ERR_SHAPE";
    case ATP_ERR_UNSUPPORTED: return "ATP_ERR_UNSUPPORTED";
    case ATP_ERR_DEVICE: return "ATP_ERR_DEVICE";
    default: return "ATP_ERR_UNKNOWN";
    }
}

const char* atp_last_error(void) { return g_last_error.c_str(); }

const char* atp_version(void) { return "atp-mi355x 0.1 (gfx950)"; }

atp_status atp_shard_geometry(const atp_mesh* mesh, int32_t mode, int64_t k, int64_t n,
                              atp_shard* out) {
    if (!out) return set_error(ATP_ERR_INVALID_ARGUMENT, "out is NULL");
    return geometry(mesh, mode, k, n, out);
}

atp_status atp_shard_linear_fwd(const atp_mesh* mesh, int32_t mode, int64_t tokens, int64_t k,
                                int64_t n, int32_t chunks, const void* x_loc, int64_t ldx,
                                const void* w_loc, int64_t ldw, const void* bias_loc,
                                int32_t epi, void* y, int32_t y_dtype, int64_t ldy,
                                void* preact, void* stream, void* const* chunk_done) {
    atp_shard g;
    ATP_CHECK(geometry(mesh, mode, k, n, &g));
    ATP_CHECK(check_chunks(tokens, chunks));
    ATP_CHECK(check_mat(x_loc, tokens, ldx, g.k_loc, "x_loc"));
    ATP_CHECK(check_mat(w_loc, g.k_loc, ldw, g.n_loc, "w_loc"));
    ATP_CHECK(check_mat(y, tokens, ldy, g.n_loc, "y"));
    if (!valid_epi(epi) || epi == ATP_EPI_GELU_BWD)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "epilogue %d not valid for a forward GEMM", epi);
    if (!valid_dtype(y_dtype)) return set_error(ATP_ERR_INVALID_ARGUMENT, "y_dtype %d", y_dtype);
    if (g.red_size > 1 && epi != ATP_EPI_NONE)
        return set_error(ATP_ERR_INVALID_ARGUMENT,
                    "reduction group of %d: y is a Partial(SUM) block, it takes no epilogue "
                    "(bias and GeLU act after the reduction)", g.red_size);
    if (epi == ATP_EPI_BIAS || epi == ATP_EPI_BIAS_GELU) ATP_CHECK(check_vec(bias_loc, "bias"));
    if (preact) {
        if (epi != ATP_EPI_BIAS_GELU)
            return set_error(ATP_ERR_INVALID_ARGUMENT, "preact is only written by BIAS_GELU");
        ATP_CHECK(check_mat(preact, tokens, ldy, g.n_loc, "preact"));
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int64_t mc = tokens / chunks;
    const bool b16 = (y_dtype == ATP_BF16);
    const size_t esz = b16 ? 2 : 4;
    for (int32_t c = 0; c < chunks; ++c) {
        const int64_t r0 = (int64_t)c * mc;
        atp::GemmProblem p = gemm_problem(
            atp::LAYOUT_NN, static_cast<const uint16_t*>(x_loc) + r0 * ldx, ldx, w_loc, ldw,
            static_cast<char*>(y) + r0 * ldy * esz, ldy, b16, epi, mc, g.n_loc, g.k_loc);
        p.bias = bias_loc;
        if (preact) p.pre_out = static_cast<uint16_t*>(preact) + r0 * ldy;
        ATP_CHECK(run_gemm(p, s));
        if (chunk_done && chunk_done[c])
            HIP_CHECK(hipEventRecord(static_cast<hipEvent_t>(chunk_done[c]), s), "hipEventRecord");
    }
    return ATP_OK;
}

extern "C++" {
namespace {

template <class PartTable>
atp_status chunked_reduce(int32_t red_size, int64_t tokens, int64_t n_loc, int32_t chunks,
                          PartTable partials, bool parts_bf16, int64_t ldp, const void* bias_loc,
                          int32_t epi, const void* preact_in, void* out, int32_t out_dtype,
                          int64_t ldo, void* preact_out, void* stream, void* const* chunk_ready) {
    if (red_size < 1) return set_error(ATP_ERR_INVALID_ARGUMENT, "red_size must be >= 1");
    if (red_size > ATP_MAX_GROUP)
        return set_error(ATP_ERR_UNSUPPORTED, "red_size %d exceeds %d", red_size, ATP_MAX_GROUP);
    if (n_loc <= 0) return set_error(ATP_ERR_INVALID_ARGUMENT, "n_loc must be positive");
    ATP_CHECK(check_chunks(tokens, chunks));
    if (!partials) return set_error(ATP_ERR_INVALID_ARGUMENT, "partials is NULL");
    for (int j = 0; j < red_size; ++j) {
        char nm[32];
        snprintf(nm, sizeof nm, "partials[%d]", j);
        ATP_CHECK(check_mat(partials[j], tokens, ldp, n_loc, nm));
    }
    ATP_CHECK(check_mat(out, tokens, ldo, n_loc, "out"));
    if (!valid_epi(epi)) return set_error(ATP_ERR_INVALID_ARGUMENT, "epilogue %d", epi);
    if (!valid_dtype(out_dtype)) return set_error(ATP_ERR_INVALID_ARGUMENT, "out_dtype %d", out_dtype);
    if (epi == ATP_EPI_BIAS || epi == ATP_EPI_BIAS_GELU) ATP_CHECK(check_vec(bias_loc, "bias"));
    if (epi == ATP_EPI_GELU_BWD) ATP_CHECK(check_mat(preact_in, tokens, ldo, n_loc, "preact_in"));
    if (preact_out) {
        if (epi != ATP_EPI_BIAS_GELU)
            return set_error(ATP_ERR_INVALID_ARGUMENT, "preact_out is only written by BIAS_GELU");
        ATP_CHECK(check_mat(preact_out, tokens, ldo, n_loc, "preact_out"));
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int64_t mc = tokens / chunks;
    for (int32_t c = 0; c < chunks; ++c) {
        if (chunk_ready && chunk_ready[c])
            HIP_CHECK(hipStreamWaitEvent(s, static_cast<hipEvent_t>(chunk_ready[c]), 0),
                      "hipStreamWaitEvent");
        atp::ReduceProblem p = reduce_problem(red_size, partials, ldp, (int64_t)c * mc, mc, n_loc,
                                              epi, bias_loc, preact_in, out, ldo,
                                              out_dtype == ATP_BF16, preact_out, parts_bf16);
        ATP_CHECK(run_reduce(p, s));
    }
    return ATP_OK;
}

}  // namespace
}  // extern "C++"

atp_status atp_chunked_partial_reduce(int32_t red_size, int64_t tokens, int64_t n_loc,
                                      int32_t chunks, const float* const* partials, int64_t ldp,
                                      const void* bias_loc, int32_t epi, const void* preact_in,
                                      void* out, int32_t out_dtype, int64_t ldo, void* preact_out,
                                      void* stream, void* const* chunk_ready) {
    return chunked_reduce(red_size, tokens, n_loc, chunks, partials, false, ldp, bias_loc, epi,
                          preact_in, out, out_dtype, ldo, preact_out, stream, chunk_ready);
}

atp_status atp_chunked_partial_reduce_bf16(int32_t red_size, int64_t tokens, int64_t n_loc,
                                           int32_t chunks, const void* const* partials,
                                           int64_t ldp, const void* bias_loc, int32_t epi,
                                           const void* preact_in, void* out, int32_t out_dtype,
                                           int64_t ldo, void* preact_out, void* stream,
                                           void* const* chunk_ready) {
    return chunked_reduce(red_size, tokens, n_loc, chunks, partials, true, ldp, bias_loc, epi,
                          preact_in, out, out_dtype, ldo, preact_out, stream, chunk_ready);
}

atp_status atp_shard_linear_fwd_fused(const atp_mesh* mesh, int32_t mode, int64_t tokens,
                                      int64_t k, int64_t n, const void* x_loc, int64_t ldx,
                                      const void* w_loc, int64_t ldw,
                                      const float* const* peers, int64_t ldp,
                                      const void* bias_loc, int32_t epi, void* out,
                                      int32_t out_dtype, int64_t ldo, void* preact,
                                      void* stream) {
    atp_shard g;
    ATP_CHECK(geometry(mesh, mode, k, n, &g));
    if (tokens < 0) return set_error(ATP_ERR_INVALID_ARGUMENT, "tokens must be >= 0");
    ATP_CHECK(check_mat(x_loc, tokens, ldx, g.k_loc, "x_loc"));
    ATP_CHECK(check_mat(w_loc, g.k_loc, ldw, g.n_loc, "w_loc"));
    ATP_CHECK(check_mat(out, tokens, ldo, g.n_loc, "out"));
    if (!valid_epi(epi) || epi == ATP_EPI_GELU_BWD)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "epilogue %d not valid for a forward GEMM", epi);
    if (!valid_dtype(out_dtype)) return set_error(ATP_ERR_INVALID_ARGUMENT, "out_dtype %d", out_dtype);
    if (g.red_size > atp::kMaxFusedParts)
        return set_error(ATP_ERR_UNSUPPORTED, "fused epilogue: group of %d exceeds %d",
                         g.red_size, atp::kMaxFusedParts);
    if (g.red_size > 1) {
        if (!peers) return set_error(ATP_ERR_INVALID_ARGUMENT, "peers is NULL");
        for (int j = 0; j < g.red_size; ++j) {
            if (j == g.red_index) continue;
            char nm[32];
            snprintf(nm, sizeof nm, "peers[%d]", j);
            ATP_CHECK(check_mat(peers[j], tokens, ldp, g.n_loc, nm));
        }
    }
    if (epi == ATP_EPI_BIAS || epi == ATP_EPI_BIAS_GELU) ATP_CHECK(check_vec(bias_loc, "bias"));
    if (preact) {
        if (epi != ATP_EPI_BIAS_GELU)
            return set_error(ATP_ERR_INVALID_ARGUMENT, "preact is only written by BIAS_GELU");
        ATP_CHECK(check_mat(preact, tokens, ldo, g.n_loc, "preact"));
    }
    atp::GemmProblem p = gemm_problem(atp::LAYOUT_NN, x_loc, ldx, w_loc, ldw, out, ldo,
                                      out_dtype == ATP_BF16, epi, tokens, g.n_loc, g.k_loc);
    p.bias = bias_loc;
    p.pre_out = preact;
    if (g.red_size > 1) {
        p.nparts = g.red_size;
        p.own = g.red_index;
        p.ldp = ldp;
        for (int j = 0; j < g.red_size; ++j) p.peers[j] = j == g.red_index ? nullptr : peers[j];
    }
    return run_gemm(p, static_cast<hipStream_t>(stream));
}

atp_status atp_shard_linear_bwd(const atp_mesh* mesh, int32_t mode, int64_t tokens, int64_t k,
                                int64_t n, int32_t chunks, const void* x_loc, int64_t ldx,
                                const void* w_loc, int64_t ldw, const void* dy, int64_t lddy,
                                float* dx_partial, int64_t lddx, float* dw, int64_t lddw,
                                float* db, void* stream, void* const* dx_chunk_done) {
    atp_shard g;
    ATP_CHECK(geometry(mesh, mode, k, n, &g));
    ATP_CHECK(check_chunks(tokens, chunks));
    ATP_CHECK(check_mat(x_loc, tokens, ldx, g.k_loc, "x_loc"));
    ATP_CHECK(check_mat(w_loc, g.k_loc, ldw, g.n_loc, "w_loc"));
    ATP_CHECK(check_mat(dy, tokens, lddy, g.n_loc, "dy"));
    ATP_CHECK(check_mat(dx_partial, tokens, lddx, g.k_loc, "dx_partial"));
    ATP_CHECK(check_mat(dw, g.k_loc, lddw, g.n_loc, "dw"));
    if (db) ATP_CHECK(check_vec(db, "db"));
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int64_t mc = tokens / chunks;
    for (int32_t c = 0; c < chunks; ++c) {
        const int64_t r0 = (int64_t)c * mc;
        // dX = dY W^T : B(k=n', col=k') = W[k'][n'], contiguous along the contraction
        atp::GemmProblem p = gemm_problem(atp::LAYOUT_NT,
                                          static_cast<const uint16_t*>(dy) + r0 * lddy, lddy,
                                          w_loc, ldw, dx_partial + r0 * lddx, lddx, false,
                                          atp::EPI_NONE, mc, g.k_loc, g.n_loc);
        ATP_CHECK(run_gemm(p, s));
        if (dx_chunk_done && dx_chunk_done[c])
            HIP_CHECK(hipEventRecord(static_cast<hipEvent_t>(dx_chunk_done[c]), s),
                      "hipEventRecord");
    }
    // dW = X^T dY over all tokens
    atp::GemmProblem p = gemm_problem(atp::LAYOUT_TN, x_loc, ldx, dy, lddy, dw, lddw, false,
                                      atp::EPI_NONE, g.k_loc, g.n_loc, tokens);
    ATP_CHECK(run_gemm(p, s));
    if (db) ATP_CHECK(run_colsum(dy, lddy, tokens, g.n_loc, db, s));
    return ATP_OK;
}

size_t atp_block_workspace_bytes(const atp_mesh* mesh, int32_t block_mode, int64_t tokens,
                                 int64_t h, int32_t chunks, int32_t weight_layout) {
    (void)chunks;
    BlockPlan P;
    if (!mesh || check_mesh(mesh) != ATP_OK || block_plan(mesh, block_mode, h, &P) != ATP_OK ||
        tokens < 0 || !valid_layout(weight_layout))
        return 0;
    return std::max(ws_fwd_bytes(P, tokens, weight_layout), ws_bwd_bytes(P, tokens, weight_layout));
}

atp_status atp_attention_fwd(const atp_mesh* mesh, int32_t block_mode, int64_t batch,
                             int64_t seq, int64_t h, int32_t heads, const void* qkv,
                             int64_t ld_qkv, void* out, int64_t ld_out, float* lse,
                             void* stream) {
    AttnPlan ap;
    ATP_CHECK(attention_plan(mesh, block_mode, batch, seq, h, heads, &ap));
    ATP_CHECK(check_mat(qkv, ap.T, ld_qkv, ap.qkv_cols, "qkv"));
    ATP_CHECK(check_mat(out, ap.T, ld_out, ap.out_cols, "out"));
    if (ap.T == 0) return ATP_OK;
    ATP_CHECK(check_vec(lse, "lse"));
    if (overlaps(qkv, ap.T, ld_qkv, 2, out, ap.T, ld_out, 2))
        return set_error(ATP_ERR_INVALID_ARGUMENT, "qkv and out must not overlap");
    atp::AttentionProblem p;
    p.qkv = qkv;
    p.ld_qkv = ld_qkv;
    p.qkv_col0 = (int64_t)ap.first * 3 * kHeadDim;
    p.out = out;
    p.ld_out = ld_out;
    p.out_col0 = (int64_t)ap.first * kHeadDim;
    p.lse = lse;
    p.batch = batch;
    p.seq = seq;
    p.heads = ap.hd;
    p.head_dim = kHeadDim;
    // causal: 2 d flops per (query, key <= query) pair in each of QK^T and PV
    const double pairs = (double)batch * ap.hd * (double)seq * (double)(seq + 1) / 2.0;
    const double flops = 4.0 * kHeadDim * pairs;
    const double bytes = (double)ap.T * ap.hd * (4.0 * kHeadDim * 2.0 + 4.0);
    hipStream_t s = static_cast<hipStream_t>(stream);
    return timed("attention_fwd", flops, bytes, s, [&] { return atp::launch_attention_fwd(p, s); });
}

atp_status atp_attention_bwd(const atp_mesh* mesh, int32_t block_mode, int64_t batch,
                             int64_t seq, int64_t h, int32_t heads, const void* qkv,
                             int64_t ld_qkv, const void* out, int64_t ld_out, const float* lse,
                             const void* d_out, int64_t ld_dout, void* d_qkv, int64_t ld_dqkv,
                             float* delta, void* stream) {
    AttnPlan ap;
    ATP_CHECK(attention_plan(mesh, block_mode, batch, seq, h, heads, &ap));
    ATP_CHECK(check_mat(qkv, ap.T, ld_qkv, ap.qkv_cols, "qkv"));
    ATP_CHECK(check_mat(out, ap.T, ld_out, ap.out_cols, "out"));
    ATP_CHECK(check_mat(d_out, ap.T, ld_dout, ap.out_cols, "d_out"));
    ATP_CHECK(check_mat(d_qkv, ap.T, ld_dqkv, ap.qkv_cols, "d_qkv"));
    if (ap.T == 0) return ATP_OK;
    ATP_CHECK(check_vec(lse, "lse"));
    ATP_CHECK(check_vec(delta, "delta"));
    if (overlaps(d_qkv, ap.T, ld_dqkv, 2, qkv, ap.T, ld_qkv, 2) ||
        overlaps(d_qkv, ap.T, ld_dqkv, 2, out, ap.T, ld_out, 2) ||
        overlaps(d_qkv, ap.T, ld_dqkv, 2, d_out, ap.T, ld_dout, 2))
        return set_error(ATP_ERR_INVALID_ARGUMENT, "d_qkv must not overlap an input");
    atp::AttentionBwdProblem p;
    p.qkv = qkv;
    p.ld_qkv = ld_qkv;
    p.qkv_col0 = (int64_t)ap.first * 3 * kHeadDim;
    p.out = out;
    p.ld_out = ld_out;
    p.out_col0 = (int64_t)ap.first * kHeadDim;
    p.dout = d_out;
    p.ld_dout = ld_dout;
    p.lse = lse;
    p.delta = delta;
    p.dqkv = d_qkv;
    p.ld_dqkv = ld_dqkv;
    p.batch = batch;
    p.seq = seq;
    p.heads = ap.hd;
    p.head_dim = kHeadDim;
    // the five products of the backward over the causal pairs
    const double pairs = (double)batch * ap.hd * (double)seq * (double)(seq + 1) / 2.0;
    const double flops = 2.0 * kHeadDim * pairs * 5.0;   // S, dP, dV, dK, dQ (S and dP are
                                                         // computed twice: not counted)
    const double bytes = (double)ap.T * ap.hd * (10.0 * kHeadDim * 2.0 + 12.0);
    hipStream_t s = static_cast<hipStream_t>(stream);
    return timed("attention_bwd", flops, bytes, s, [&] { return atp::launch_attention_bwd(p, s); });
}

atp_status atp_attention_bwd_noalloc(const atp_mesh* mesh, int32_t block_mode, int64_t batch,
                                     int64_t seq, int64_t h, int32_t heads, const void* qkv,
                                     int64_t ld_qkv, const void* out, int64_t ld_out,
                                     const float* lse, const void* d_out, int64_t ld_dout,
                                     void* d_qkv, int64_t ld_dqkv, void* stream) {
    AttnPlan ap;
    ATP_CHECK(attention_plan(mesh, block_mode, batch, seq, h, heads, &ap));
    if ((int64_t)ap.hd * ap.T > kNoAllocDeltaMax)
        return set_error(ATP_ERR_UNSUPPORTED,
                         "%d heads x %lld tokens need %lld scratch values; the library's "
                         "scratch holds %lld (use atp_attention_bwd with a delta buffer)",
                         ap.hd, (long long)ap.T, (long long)ap.hd * ap.T,
                         (long long)kNoAllocDeltaMax);
    float* delta = nullptr;
    if (ap.T > 0) ATP_CHECK(noalloc_scratch(&delta));
    return atp_attention_bwd(mesh, block_mode, batch, seq, h, heads, qkv, ld_qkv, out, ld_out, lse,
                             d_out, ld_dout, d_qkv, ld_dqkv, delta, stream);
}

atp_status atp_transpose_bf16(int64_t rows, int64_t cols, const void* src, int64_t lds, void* dst,
                              int64_t ldd, void* stream) {
    if (rows < 0 || cols < 0) return set_error(ATP_ERR_INVALID_ARGUMENT, "negative size");
    if (rows == 0 || cols == 0) return ATP_OK;    // nothing is read or written
    ATP_CHECK(check_mat(src, rows, lds, cols, "src", true));
    ATP_CHECK(check_mat(dst, cols, ldd, rows, "dst", true));
    if (src == dst)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "src and dst must not be the same buffer");
    return run_transpose(src, lds, rows, cols, dst, ldd, static_cast<hipStream_t>(stream));
}

extern "C++" {
namespace {

// Weights of the block in either storage order: the checks, and the
// operand of each product.  `kn` weights are [k_loc][n_loc], else [n_loc][k_loc].
atp_status check_weights(const BlockPlan& P, const atp_block_weights* w) {
    if (!valid_layout(w->layout))
        return set_error(ATP_ERR_INVALID_ARGUMENT, "weight layout %d unknown", w->layout);
    const bool kn = w->layout == ATP_W_KN;
    for (int i = 0; i < 4; ++i) {
        char nm[32];
        snprintf(nm, sizeof nm, "w[%s]", kLinearName[i]);
        const atp_shard& g = P.g[i];
        ATP_CHECK(check_mat(w->w[i], kn ? g.k_loc : g.n_loc, w->ldw[i], kn ? g.n_loc : g.k_loc,
                            nm));
        snprintf(nm, sizeof nm, "b[%s]", kLinearName[i]);
        ATP_CHECK(check_vec(w->b[i], nm));
    }
    return ATP_OK;
}

atp_status check_partial_dtype(int32_t d) {
    if (!valid_dtype(d)) return set_error(ATP_ERR_INVALID_ARGUMENT, "partial_dtype %d", d);
    return ATP_OK;
}

// Byte offset of row r of a partial buffer with leading dimension ld.
template <class T>
T* row_ptr(T* base, int64_t r, int64_t ld, bool b16) {
    return reinterpret_cast<T*>(reinterpret_cast<typename std::conditional<
        std::is_const<T>::value, const char, char>::type*>(base) + r * ld * (b16 ? 2 : 4));
}

// ------------------------------------------------------------------------
// The attention block's chain reads the weights as stored (no workspace).
// X W: NN from [k][n] weights, NT from [n][k].  dY W^T: NT from [k][n], NN
// from [n][k].  dW = X^T dY ([k][n]) or dW^T = dY^T X ([n][k]) over the
// tokens: TN.
atp::GemmProblem xw_problem(const atp_shard& g, bool kn, const void* W, int64_t ldw,
                            const void* A, int64_t lda, void* C, int64_t ldc, bool b16, int epi,
                            int64_t M) {
    return gemm_problem(kn ? atp::LAYOUT_NN : atp::LAYOUT_NT, A, lda, W, ldw, C, ldc, b16, epi, M,
                        g.n_loc, g.k_loc);
}

atp::GemmProblem dyw_problem(const atp_shard& g, bool kn, const void* W, int64_t ldw,
                             const void* dY, int64_t lddy, void* C, int64_t ldc, bool b16, int epi,
                             int64_t M) {
    return gemm_problem(kn ? atp::LAYOUT_NT : atp::LAYOUT_NN, dY, lddy, W, ldw, C, ldc, b16, epi,
                        M, g.k_loc, g.n_loc);
}

atp_status weight_grads(const atp_shard& g, bool kn, const void* X, int64_t ldx, const void* dY,
                        int64_t lddy, float* dw, int64_t ldw, float* db, int64_t T,
                        hipStream_t s) {
    if (db) ATP_CHECK(run_colsum(dY, lddy, T, g.n_loc, db, s));
    atp::GemmProblem p =
        kn ? gemm_problem(atp::LAYOUT_TN, X, ldx, dY, lddy, dw, ldw, false, atp::EPI_NONE, g.k_loc,
                          g.n_loc, T)
           : gemm_problem(atp::LAYOUT_TN, dY, lddy, X, ldx, dw, ldw, false, atp::EPI_NONE, g.n_loc,
                          g.k_loc, T);
    return run_gemm(p, s);
}

// One reduced product of the chain, chunked (Sec. 4.1): chunk c's GEMM on
// cs writes the own partial rows (or, for a group of one, the whole output
// with its epilogue in one launch), and ms reduces the group's partials of
// those rows with the epilogue as soon as they are written.  `done` is
// recorded after the last chunk's reduction (on ms), or after the single
// launch (on cs).  make(A_rows, C_rows, ldc, b16, epi, M) builds the product;
// with a slab, a chunk product with too few tiles is split over k there.
template <class Make>
atp_status chained_linear(const Streams& S, int red_size, int red_index, void* const* parts,
                          int64_t ldp, bool pb16, const void* A, int64_t lda, int64_t ncols,
                          int epi, const void* bias, const void* pre_in, void* out, int64_t ldo,
                          int64_t T, int32_t chunks, hipEvent_t* ev_chunk, hipEvent_t done,
                          Make make, float* slab = nullptr) {
    if (red_size == 1) {
        atp::GemmProblem p = make(A, out, ldo, true, epi, T);
        p.bias = bias;
        p.pre_in = pre_in;
        ATP_CHECK(run_gemm(p, S.cs));
        HIP_CHECK(hipEventRecord(done, S.cs), "hipEventRecord");
        return ATP_OK;
    }
    const int64_t mc = T / chunks;
    void* own = parts[red_index];
    for (int32_t c = 0; c < chunks; ++c) {
        const int64_t r0 = (int64_t)c * mc;
        atp::GemmProblem p = make(static_cast<const uint16_t*>(A) + r0 * lda,
                                  row_ptr(own, r0, ldp, pb16), ldp, pb16, atp::EPI_NONE, mc);
        ATP_CHECK(run_nt_partial(p, slab, S.cs));
        HIP_CHECK(hipEventRecord(ev_chunk[c], S.cs), "hipEventRecord");
        HIP_CHECK(hipStreamWaitEvent(S.ms, ev_chunk[c], 0), "hipStreamWaitEvent");
        atp::ReduceProblem r = reduce_problem(red_size, parts, ldp, r0, mc, ncols, epi, bias,
                                              pre_in, out, ldo, true, nullptr, pb16);
        ATP_CHECK(run_reduce(r, S.ms));
    }
    HIP_CHECK(hipEventRecord(done, S.ms), "hipEventRecord");
    return ATP_OK;
}

// The attention block's backward with a workspace: X^T and dY^T of one
// linear in the workspace (padded pitch), db from the dY transpose's column
// partials, then dW as an NT product over the tokens (dW^T = dY^T X for
// weights stored [n][k]); the same bits as weight_grads.
atp_status weight_grads_ws(const atp_shard& g, bool kn, const void* X, int64_t ldx,
                           const void* dY, int64_t lddy, float* dw, int64_t ldw, float* db,
                           int64_t T, uint16_t* xt, uint16_t* dyt, float* colpart,
                           hipStream_t s) {
    const int64_t tp = ws_pitch(T);
    ATP_CHECK(run_transpose(X, ldx, T, g.k_loc, xt, tp, s));
    float* part = db ? colpart : nullptr;
    ATP_CHECK(run_transpose(dY, lddy, T, g.n_loc, dyt, tp, s, part, g.n_loc));
    if (part) ATP_CHECK(run_colsum_finish(part, g.n_loc, (T + 63) / 64, g.n_loc, db, s));
    const atp::GemmProblem p =
        kn ? gemm_problem(atp::LAYOUT_NT, xt, tp, dyt, tp, dw, ldw, false, atp::EPI_NONE, g.k_loc,
                          g.n_loc, T)
           : gemm_problem(atp::LAYOUT_NT, dyt, tp, xt, tp, dw, ldw, false, atp::EPI_NONE, g.n_loc,
                          g.k_loc, T);
    return run_gemm(p, s);
}

// Bytes the attention block's backward carves from a workspace: X^T of x
// and of the gathered block, dY^T of d_qkv and d_o, db's column partials
// (a subset of the block backward's pieces, so ws_bwd_bytes covers it).
size_t attn_ws_bwd_bytes(const BlockPlan& P, int64_t tokens) {
    const size_t t2 = (size_t)ws_pitch(tokens) * 2;
    return ws_round(P.g[0].k_loc * t2) + ws_round(P.g[1].k_loc * t2) +
           ws_round(P.g[0].n_loc * t2) + ws_round(P.g[1].n_loc * t2) +
           ws_round(colpart_bytes(P, tokens));
}

atp_status check_attn_weights(const BlockPlan& P, const atp_block_weights* w) {
    if (!valid_layout(w->layout))
        return set_error(ATP_ERR_INVALID_ARGUMENT, "weight layout %d unknown", w->layout);
    const bool kn = w->layout == ATP_W_KN;
    for (int i = 0; i < 2; ++i) {
        char nm[32];
        snprintf(nm, sizeof nm, "w[%s]", kLinearName[i]);
        const atp_shard& g = P.g[i];
        ATP_CHECK(check_mat(w->w[i], kn ? g.k_loc : g.n_loc, w->ldw[i], kn ? g.n_loc : g.k_loc,
                            nm));
        snprintf(nm, sizeof nm, "b[%s]", kLinearName[i]);
        ATP_CHECK(check_vec(w->b[i], nm));
    }
    return ATP_OK;
}

}  // namespace
}  // extern "C++"

int32_t atp_block_workspace_path(const atp_mesh* mesh, int32_t block_mode, int64_t tokens,
                                 int64_t h, int32_t weight_layout, size_t ws_bytes,
                                 int32_t pass) {
    BlockPlan P;
    if (!mesh || check_mesh(mesh) != ATP_OK || block_plan(mesh, block_mode, h, &P) != ATP_OK ||
        tokens < 0 || !valid_layout(weight_layout) || (pass != 0 && pass != 1))
        return -1;
    return takes_ws_path(P, tokens, weight_layout, ws_bytes, pass) ? 1 : 0;
}

atp_status atp_block_geometry(const atp_mesh* mesh, int32_t block_mode, int64_t h,
                              atp_shard out[4]) {
    if (!out) return set_error(ATP_ERR_INVALID_ARGUMENT, "out is NULL");
    BlockPlan P;
    ATP_CHECK(check_mesh(mesh));
    ATP_CHECK(block_plan(mesh, block_mode, h, &P));
    for (int i = 0; i < 4; ++i) out[i] = P.g[i];
    return ATP_OK;
}

atp_status atp_attention_heads(const atp_mesh* mesh, int32_t block_mode, int64_t h,
                               int32_t heads, int32_t* first, int32_t* count,
                               int32_t* per_block) {
    if (!first || !count || !per_block)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "an output pointer is NULL");
    AttnPlan ap;
    ATP_CHECK(attention_plan(mesh, block_mode, 0, 0, h, heads, &ap));
    *first = ap.first;
    *count = ap.hd;
    *per_block = ap.heads_blk;
    return ATP_OK;
}

atp_status atp_block_fwd(const atp_mesh* mesh, int32_t block_mode, int64_t tokens, int64_t h,
                         int32_t chunks, const atp_block_weights* w, const atp_block_fwd_io* io,
                         void* workspace, size_t ws_bytes, void* compute_stream,
                         void* comm_stream) {
    BlockPlan P;
    ATP_CHECK(check_mesh(mesh));
    ATP_CHECK(block_plan(mesh, block_mode, h, &P));
    ATP_CHECK(check_chunks(tokens, chunks));
    if (!w || !io) return set_error(ATP_ERR_INVALID_ARGUMENT, "weights or io is NULL");
    ATP_CHECK(check_weights(P, w));
    ATP_CHECK(check_partial_dtype(io->partial_dtype));
    const bool kn = w->layout == ATP_W_KN;
    const bool pb16 = io->partial_dtype == ATP_BF16;
    // inputs: x feeds qkv and fc1 (same k split), attn feeds out
    if (P.g[0].k_loc != P.g[2].k_loc)
        return set_error(ATP_ERR_SHAPE, "qkv and fc1 contract over different blocks of x");
    ATP_CHECK(check_mat(io->x_loc, tokens, io->ldx, P.g[0].k_loc, "x_loc"));
    ATP_CHECK(check_mat(io->attn_loc, tokens, io->lda, P.g[1].k_loc, "attn_loc"));
    ATP_CHECK(check_mat(io->qkv, tokens, io->ld_qkv, P.g[0].n_loc, "qkv"));
    ATP_CHECK(check_mat(io->o, tokens, io->ld_o, P.g[1].n_loc, "o"));
    ATP_CHECK(check_mat(io->h, tokens, io->ld_h, P.g[2].n_loc, "h"));
    ATP_CHECK(check_mat(io->pre, tokens, io->ld_h, P.g[2].n_loc, "pre"));
    ATP_CHECK(check_mat(io->z, tokens, io->ld_z, P.g[3].n_loc, "z"));
    if (P.g[3].k_loc != P.g[2].n_loc)
        return set_error(ATP_ERR_SHAPE, "fc2 contracts over %lld columns, fc1 produces %lld",
                    (long long)P.g[3].k_loc, (long long)P.g[2].n_loc);
    for (int i = 0; i < 4; ++i) {
        char nm[32];
        snprintf(nm, sizeof nm, "partials[%s]", kLinearName[i]);
        ATP_CHECK(check_group(io->partials[i], P.g[i].red_size, tokens, io->ldp[i], P.g[i].n_loc, nm));
    }
    if (workspace && reinterpret_cast<uintptr_t>(workspace) % kWsAlign)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "workspace must be %zu-byte aligned", kWsAlign);

    // With a large enough workspace every forward product runs with both
    // operands contiguous along k (the layout the GEMM kernel streams
    // fastest; weights stored [k][n] are first copied there as W^T, unless
    // the linear's products stream NN as fast: fwd_reads_w), and chunk
    // products with too few tiles to fill the chip are split over k into
    // slabs there.  The direct path never runs under graph capture.
    const bool ws = workspace && takes_ws_path(P, tokens, w->layout, ws_bytes, 0);
    if (!ws) ATP_CHECK(refuse_capture_of_direct_path(compute_stream));

    Streams S(compute_stream, comm_stream);
    hipEvent_t* ev = nullptr;
    // [0] start  [1] comm end  [2] second lane forked  [3] second lane
    // joined, then per linear per chunk GEMM-done, then fc1 reduce-done per
    // chunk
    const size_t n_ev = 4 + 4 * (size_t)chunks + (size_t)chunks;
    ATP_CHECK(sync_events(n_ev, &ev));
    hipEvent_t* ev_gemm = ev + 4;
    hipEvent_t* ev_red1 = ev + 4 + 4 * chunks;
    ATP_CHECK(S.begin(ev[0]));
    // A second compute lane for the chunk products, only when the caller
    // overlaps at all (comm_stream != compute_stream) and outside graph
    // capture (captures stay on the streams the caller gave)
    hipStream_t lane2 = nullptr;
    if (S.ms != S.cs && chunks > 1) {
        hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
        HIP_CHECK(hipStreamIsCapturing(S.cs, &cap), "hipStreamIsCapturing");
        if (cap == hipStreamCaptureStatusNone) ATP_CHECK(second_lane(&lane2));
    }
    bool lane2_used = false;

    uint16_t* wt[4] = {nullptr, nullptr, nullptr, nullptr};
    float* slab = nullptr;
    if (ws) {
        Carver c{static_cast<char*>(workspace)};
        if (kn)
            for (int L = 0; L < 4; ++L)
                if (fwd_may_copy_w(P, L, tokens)) {
                    uint16_t* t = c.take((size_t)P.g[L].n_loc * ws_pitch(P.g[L].k_loc) * 2);
                    if (!fwd_reads_w(P, L, tokens, chunks)) wt[L] = t;
                }
        slab = reinterpret_cast<float*>(c.take(slab_bytes(P, tokens, false)));
    }
    // W^T of linear L (weights stored [k][n]), written before the linear's
    // first GEMM (same stream)
    bool wt_done[4] = {false, false, false, false};
    auto need_wt = [&](int L) -> atp_status {
        if (!wt[L] || wt_done[L]) return ATP_OK;
        const atp_shard& g = P.g[L];
        ATP_CHECK(run_transpose(w->w[L], w->ldw[L], g.k_loc, g.n_loc, wt[L], ws_pitch(g.k_loc),
                                S.cs));
        wt_done[L] = true;
        return ATP_OK;
    };
    // the product X W of linear L: NT from W^T (the workspace copy, or the
    // weight itself when stored [n][k]), or NN from W stored [k][n] (no copy)
    auto fwd_problem = [&](int L, const void* A, int64_t lda, void* C, int64_t ldc, bool b16,
                           int epi, int64_t M) {
        const atp_shard& g = P.g[L];
        if (!kn)
            return gemm_problem(atp::LAYOUT_NT, A, lda, w->w[L], w->ldw[L], C, ldc, b16, epi, M,
                                g.n_loc, g.k_loc);
        if (wt[L])
            return gemm_problem(atp::LAYOUT_NT, A, lda, wt[L], ws_pitch(g.k_loc), C, ldc, b16,
                                epi, M, g.n_loc, g.k_loc);
        return gemm_problem(atp::LAYOUT_NN, A, lda, w->w[L], w->ldw[L], C, ldc, b16, epi, M,
                            g.n_loc, g.k_loc);
    };

    const int64_t mc = tokens / chunks;
    const void* A_in[4] = {io->x_loc, io->attn_loc, io->x_loc, io->h};
    const int64_t lda_in[4] = {io->ldx, io->lda, io->ldx, io->ld_h};
    void* outp[4] = {io->qkv, io->o, io->h, io->z};
    const int64_t ldo[4] = {io->ld_qkv, io->ld_o, io->ld_h, io->ld_z};
    const bool fc1_reduced = P.g[2].red_size > 1;

    // fc2 reads H: wait for fc1's reduced chunk c (the comm stream runs in
    // order, so chunk chunks-1 means all of H); fc1's single launch is
    // ordered before fc2 on the compute stream already
    auto wait_h = [&](int c, hipStream_t st) -> atp_status {
        if (fc1_reduced) HIP_CHECK(hipStreamWaitEvent(st, ev_red1[c], 0), "hipStreamWaitEvent");
        return ATP_OK;
    };
    auto unchunked = [&](int L) -> atp_status {
        if (L == 3) ATP_CHECK(wait_h(chunks - 1, S.cs));
        ATP_CHECK(need_wt(L));
        atp::GemmProblem p = fwd_problem(L, A_in[L], lda_in[L], outp[L], ldo[L], true,
                                         L == 2 ? atp::EPI_BIAS_GELU : atp::EPI_BIAS, tokens);
        p.bias = w->b[L];
        p.pre_out = (L == 2) ? io->pre : nullptr;
        return run_gemm(p, S.cs);
    };
    // chunk c: the GEMM writes this device's partial rows, the comm stream
    // reduces the group's partials for those rows as soon as they are ready
    auto chunk = [&](int L, int c, hipStream_t st) -> atp_status {
        const atp_shard& g = P.g[L];
        const int64_t r0 = (int64_t)c * mc;
        if (L == 3) ATP_CHECK(wait_h(c, st));
        void* own = io->partials[L][g.red_index];
        atp::GemmProblem p = fwd_problem(L, static_cast<const uint16_t*>(A_in[L]) + r0 * lda_in[L],
                                         lda_in[L], row_ptr(own, r0, io->ldp[L], pb16),
                                         io->ldp[L], pb16, atp::EPI_NONE, mc);
        ATP_CHECK(run_nt_partial(p, slab, st));
        hipEvent_t e = ev_gemm[L * chunks + c];
        HIP_CHECK(hipEventRecord(e, st), "hipEventRecord");
        HIP_CHECK(hipStreamWaitEvent(S.ms, e, 0), "hipStreamWaitEvent");
        atp::ReduceProblem r = reduce_problem(
            g.red_size, io->partials[L], io->ldp[L], r0, mc, g.n_loc,
            L == 2 ? atp::EPI_BIAS_GELU : atp::EPI_BIAS, w->b[L], nullptr, outp[L], ldo[L], true,
            L == 2 ? io->pre : nullptr, pb16);
        ATP_CHECK(run_reduce(r, S.ms));
        if (L == 2) HIP_CHECK(hipEventRecord(ev_red1[c], S.ms), "hipEventRecord");
        return ATP_OK;
    };
    // Odd chunks go to the second lane unless the chunk products split over
    // k (the splits of every chunk share one slab region, so they stay in
    // order on one stream); the lane first waits for everything queued on
    // compute_stream so far (fc1's output, the W^T copy).
    auto linear = [&](int L) -> atp_status {
        const atp_shard& g = P.g[L];
        if (g.red_size == 1) return unchunked(L);
        ATP_CHECK(need_wt(L));
        int64_t ks = 0;
        const bool two = lane2 && (!slab || atp::nt_split_plan(mc, g.n_loc, g.k_loc, &ks) <= 1);
        if (two) {
            HIP_CHECK(hipEventRecord(ev[2], S.cs), "hipEventRecord");
            HIP_CHECK(hipStreamWaitEvent(lane2, ev[2], 0), "hipStreamWaitEvent");
            lane2_used = true;
        }
        for (int c = 0; c < chunks; ++c) ATP_CHECK(chunk(L, c, two && (c & 1) ? lane2 : S.cs));
        return ATP_OK;
    };
    // out-proj first (its reductions start at once), then fc1; of QKV and fc2
    // (behind fc1's output) the one with fewer reduced bytes goes last, so
    // the other's last reductions run beside its GEMMs instead of after them
    auto red_bytes = [&](int L) {
        const atp_shard& g = P.g[L];
        return g.red_size > 1 ? (double)g.red_size * (double)g.n_loc : 0.0;
    };
    const bool qkv_last = red_bytes(0) <= red_bytes(3);
    const int order[4] = {1, 2, qkv_last ? 3 : 0, qkv_last ? 0 : 3};
    for (int L : order) ATP_CHECK(linear(L));
    if (lane2_used) {
        // compute_stream is ordered after the second lane's products
        HIP_CHECK(hipEventRecord(ev[3], lane2), "hipEventRecord");
        HIP_CHECK(hipStreamWaitEvent(S.cs, ev[3], 0), "hipStreamWaitEvent");
    }
    return S.end(ev[1]);
}

atp_status atp_block_bwd(const atp_mesh* mesh, int32_t block_mode, int64_t tokens, int64_t h,
                         int32_t chunks, const atp_block_weights* w, const atp_block_bwd_io* io,
                         void* workspace, size_t ws_bytes, void* compute_stream,
                         void* comm_stream) {
    BlockPlan P;
    ATP_CHECK(check_mesh(mesh));
    ATP_CHECK(block_plan(mesh, block_mode, h, &P));
    ATP_CHECK(check_chunks(tokens, chunks));
    if (!w || !io) return set_error(ATP_ERR_INVALID_ARGUMENT, "weights or io is NULL");
    ATP_CHECK(check_weights(P, w));
    ATP_CHECK(check_partial_dtype(io->partial_dtype));
    const bool kn = w->layout == ATP_W_KN;
    const bool pb16 = io->partial_dtype == ATP_BF16;
    for (int i = 0; i < 4; ++i) {
        char nm[32];
        const atp_shard& g = P.g[i];
        snprintf(nm, sizeof nm, "dw[%s]", kLinearName[i]);
        ATP_CHECK(check_mat(io->dw[i], kn ? g.k_loc : g.n_loc, w->ldw[i], kn ? g.n_loc : g.k_loc,
                            nm));
        if (io->db[i]) {
            snprintf(nm, sizeof nm, "db[%s]", kLinearName[i]);
            ATP_CHECK(check_vec(io->db[i], nm));
        }
    }
    ATP_CHECK(check_mat(io->x_loc, tokens, io->ldx, P.g[0].k_loc, "x_loc"));
    ATP_CHECK(check_mat(io->attn_loc, tokens, io->lda, P.g[1].k_loc, "attn_loc"));
    ATP_CHECK(check_mat(io->h, tokens, io->ld_h, P.g[2].n_loc, "h"));
    ATP_CHECK(check_mat(io->pre, tokens, io->ld_h, P.g[2].n_loc, "pre"));
    ATP_CHECK(check_mat(io->dz, tokens, io->ld_dz, P.g[3].n_loc, "dz"));
    ATP_CHECK(check_mat(io->dqkv, tokens, io->ld_dqkv, P.g[0].n_loc, "dqkv"));
    ATP_CHECK(check_mat(io->d_o, tokens, io->ld_do, P.g[1].n_loc, "d_o"));
    ATP_CHECK(check_mat(io->dh_pre, tokens, io->ld_h, P.g[2].n_loc, "dh_pre"));
    ATP_CHECK(check_mat(io->dx_qkv, tokens, io->ld_dx_qkv, P.g[0].k_loc, "dx_qkv"));
    ATP_CHECK(check_mat(io->dx_fc1, tokens, io->ld_dx_fc1, P.g[2].k_loc, "dx_fc1"));
    ATP_CHECK(check_mat(io->d_attn, tokens, io->ld_d_attn, P.g[1].k_loc, "d_attn"));
    if (P.g[3].k_loc != P.g[2].n_loc)
        return set_error(ATP_ERR_SHAPE, "fc2 / fc1 block mismatch");
    for (int i = 0; i < 4; ++i) {
        char nm[32];
        snprintf(nm, sizeof nm, "dx_partials[%s]", kLinearName[i]);
        ATP_CHECK(check_group(io->dx_partials[i], P.g[i].bwd_size, tokens, io->ld_dxp[i], P.g[i].k_loc,
                              nm));
    }
    if (workspace && reinterpret_cast<uintptr_t>(workspace) % kWsAlign)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "workspace must be %zu-byte aligned", kWsAlign);

    // With a large enough workspace (and whole 16-byte rows of tokens) dW runs
    // from X^T and dY^T (both contiguous along the tokens), dX from W stored
    // [k][n] (a copy in the workspace for weights stored [n][k]), and chunked
    // dX products with too few tiles to fill the chip are split over k into
    // slabs there.  The direct path never runs under graph capture.
    const bool ws = workspace && takes_ws_path(P, tokens, w->layout, ws_bytes, 1);
    if (!ws) ATP_CHECK(refuse_capture_of_direct_path(compute_stream));

    Streams S(compute_stream, comm_stream);
    hipEvent_t* ev = nullptr;
    // [0] start  [1] comm end  [2..3] unused, then per linear per chunk
    // GEMM-done, then fc2 reduce-done per chunk
    const size_t n_ev = 4 + 4 * (size_t)chunks + (size_t)chunks;
    ATP_CHECK(sync_events(n_ev, &ev));
    hipEvent_t* ev_gemm = ev + 4;
    hipEvent_t* ev_red2 = ev + 4 + 4 * chunks;
    ATP_CHECK(S.begin(ev[0]));

    // X^T pieces: 0 = x (QKV and fc1), 1 = attention block (out), 2 = H (fc2)
    const int xsrc[4] = {0, 1, 0, 2};
    uint16_t* xt[3] = {nullptr, nullptr, nullptr};
    uint16_t* dyt[4] = {nullptr, nullptr, nullptr, nullptr};
    uint16_t* wkn = nullptr;    // [k][n] copy of a weight stored [n][k]
    bool xt_done[3] = {false, false, false};
    float* slab = nullptr;
    float* colpart = nullptr;   // db of the workspace path: dY^T's transpose writes partials
    if (ws) {
        Carver c{static_cast<char*>(workspace)};
        const size_t t2 = (size_t)ws_pitch(tokens) * 2;
        xt[0] = c.take(P.g[0].k_loc * t2);
        xt[1] = c.take(P.g[1].k_loc * t2);
        xt[2] = c.take(P.g[3].k_loc * t2);
        for (int L = 0; L < 4; ++L) dyt[L] = c.take(P.g[L].n_loc * t2);
        slab = reinterpret_cast<float*>(c.take(slab_bytes(P, tokens, true)));
        colpart = reinterpret_cast<float*>(c.take(colpart_bytes(P, tokens)));
        if (!kn) wkn = c.take(wkn_bytes(P));
    }

    const int64_t mc = tokens / chunks;
    const void* Xin[4] = {io->x_loc, io->attn_loc, io->x_loc, io->h};
    const int64_t ldx_in[4] = {io->ldx, io->lda, io->ldx, io->ld_h};
    const void* dY[4] = {io->dqkv, io->d_o, io->dh_pre, io->dz};
    const int64_t ld_dy[4] = {io->ld_dqkv, io->ld_do, io->ld_h, io->ld_dz};
    void* dXo[4] = {io->dx_qkv, io->d_attn, io->dx_fc1, io->dh_pre};
    const int64_t ld_dxo[4] = {io->ld_dx_qkv, io->ld_d_attn, io->ld_dx_fc1, io->ld_h};
    const bool fc2_reduced = P.g[3].bwd_size > 1;

    // fc1's dY is dh_pre: wait for fc2's reduced chunk c (chunk chunks-1
    // means all of it, the comm stream runs in order); fc2's single dX
    // launch is ordered before fc1 on the compute stream already
    auto wait_dpre = [&](int c) -> atp_status {
        if (fc2_reduced) HIP_CHECK(hipStreamWaitEvent(S.cs, ev_red2[c], 0), "hipStreamWaitEvent");
        return ATP_OK;
    };
    // the product dY W^T of linear L: NT from W stored [k][n] (or its copy),
    // or NN from W stored [n][k] without a workspace
    int wkn_of = -1;   // the linear whose weight the [k][n] copy holds
    auto dx_problem = [&](int L, const void* A, int64_t lda, void* C, int64_t ldc, bool b16,
                          int epi, int64_t M) -> atp::GemmProblem {
        const atp_shard& g = P.g[L];
        if (kn)
            return gemm_problem(atp::LAYOUT_NT, A, lda, w->w[L], w->ldw[L], C, ldc, b16, epi, M,
                                g.k_loc, g.n_loc);
        if (ws)
            return gemm_problem(atp::LAYOUT_NT, A, lda, wkn, ws_pitch(g.n_loc), C, ldc, b16, epi,
                                M, g.k_loc, g.n_loc);
        return gemm_problem(atp::LAYOUT_NN, A, lda, w->w[L], w->ldw[L], C, ldc, b16, epi, M,
                            g.k_loc, g.n_loc);
    };
    auto need_wkn = [&](int L) -> atp_status {
        if (kn || !ws || wkn_of == L) return ATP_OK;
        const atp_shard& g = P.g[L];
        ATP_CHECK(run_transpose(w->w[L], w->ldw[L], g.n_loc, g.k_loc, wkn, ws_pitch(g.n_loc),
                                S.cs));
        wkn_of = L;
        return ATP_OK;
    };
    auto dx_unchunked = [&](int L) -> atp_status {
        const atp_shard& g = P.g[L];
        if (L == 2) ATP_CHECK(wait_dpre(chunks - 1));
        ATP_CHECK(need_wkn(L));
        atp::GemmProblem p = dx_problem(L, dY[L], ld_dy[L], dXo[L], ld_dxo[L], true,
                                        L == 3 ? atp::EPI_GELU_BWD : atp::EPI_NONE, tokens);
        p.pre_in = (L == 3) ? io->pre : nullptr;
        (void)g;
        return run_gemm(p, S.cs);
    };
    auto dx_chunk = [&](int L, int c) -> atp_status {
        const atp_shard& g = P.g[L];
        const int64_t r0 = (int64_t)c * mc;
        if (L == 2) ATP_CHECK(wait_dpre(c));
        ATP_CHECK(need_wkn(L));
        void* own = io->dx_partials[L][g.bwd_index];
        atp::GemmProblem p = dx_problem(L, static_cast<const uint16_t*>(dY[L]) + r0 * ld_dy[L],
                                        ld_dy[L], row_ptr(own, r0, io->ld_dxp[L], pb16),
                                        io->ld_dxp[L], pb16, atp::EPI_NONE, mc);
        ATP_CHECK(run_nt_partial(p, slab, S.cs));
        hipEvent_t e = ev_gemm[L * chunks + c];
        HIP_CHECK(hipEventRecord(e, S.cs), "hipEventRecord");
        HIP_CHECK(hipStreamWaitEvent(S.ms, e, 0), "hipStreamWaitEvent");
        atp::ReduceProblem r = reduce_problem(
            g.bwd_size, io->dx_partials[L], io->ld_dxp[L], r0, mc, g.k_loc,
            L == 3 ? atp::EPI_GELU_BWD : atp::EPI_NONE, nullptr, L == 3 ? io->pre : nullptr,
            dXo[L], ld_dxo[L], true, nullptr, pb16);
        ATP_CHECK(run_reduce(r, S.ms));
        if (L == 3) HIP_CHECK(hipEventRecord(ev_red2[c], S.ms), "hipEventRecord");
        return ATP_OK;
    };
    auto dx = [&](int L) -> atp_status {
        if (P.g[L].bwd_size == 1) return dx_unchunked(L);
        for (int c = 0; c < chunks; ++c) ATP_CHECK(dx_chunk(L, c));
        return ATP_OK;
    };
    // db (column sums of dY), then dW = X^T dY over all tokens (stored as
    // dW^T = dY^T X for weights stored [n][k]); these need no reduction and
    // run while the dX reductions drain
    auto dw = [&](int L) -> atp_status {
        const atp_shard& g = P.g[L];
        if (L == 2) ATP_CHECK(wait_dpre(chunks - 1));
        if (io->db[L] && !ws)
            ATP_CHECK(run_colsum(dY[L], ld_dy[L], tokens, g.n_loc, io->db[L], S.cs));
        if (!ws) {
            atp::GemmProblem p =
                kn ? gemm_problem(atp::LAYOUT_TN, Xin[L], ldx_in[L], dY[L], ld_dy[L], io->dw[L],
                                  w->ldw[L], false, atp::EPI_NONE, g.k_loc, g.n_loc, tokens)
                   : gemm_problem(atp::LAYOUT_TN, dY[L], ld_dy[L], Xin[L], ldx_in[L], io->dw[L],
                                  w->ldw[L], false, atp::EPI_NONE, g.n_loc, g.k_loc, tokens);
            return run_gemm(p, S.cs);
        }
        // X^T once per source (x serves QKV and fc1), dY^T, then the NT
        // product over the tokens
        const int xi = xsrc[L];
        const int64_t tp = ws_pitch(tokens);
        if (!xt_done[xi]) {
            ATP_CHECK(run_transpose(Xin[L], ldx_in[L], tokens, g.k_loc, xt[xi], tp, S.cs));
            xt_done[xi] = true;
        }
        // dY^T, and with it the column partials of dY for db (one read of dY)
        float* part = io->db[L] ? colpart : nullptr;
        ATP_CHECK(run_transpose(dY[L], ld_dy[L], tokens, g.n_loc, dyt[L], tp, S.cs, part,
                                g.n_loc));
        if (part)
            ATP_CHECK(run_colsum_finish(part, g.n_loc, (tokens + 63) / 64, g.n_loc, io->db[L],
                                        S.cs));
        atp::GemmProblem p =
            kn ? gemm_problem(atp::LAYOUT_NT, xt[xi], tp, dyt[L], tp, io->dw[L], w->ldw[L], false,
                              atp::EPI_NONE, g.k_loc, g.n_loc, tokens)
               : gemm_problem(atp::LAYOUT_NT, dyt[L], tp, xt[xi], tp, io->dw[L], w->ldw[L], false,
                              atp::EPI_NONE, g.n_loc, g.k_loc, tokens);
        return run_gemm(p, S.cs);
    };
    // fc2's dX first (it makes dh_pre, which fc1 waits for); then the
    // attention projections' dX, whose reductions can start at once; then
    // fc1's dX; the four dW last, largest first
    ATP_CHECK(dx(3));
    ATP_CHECK(dx(0));
    ATP_CHECK(dx(1));
    ATP_CHECK(dx(2));
    int order[4] = {3, 2, 0, 1};
    std::stable_sort(order, order + 4, [&](int i, int j) {
        return P.g[i].k_loc * P.g[i].n_loc > P.g[j].k_loc * P.g[j].n_loc;
    });
    for (int L : order) ATP_CHECK(dw(L));
    return S.end(ev[1]);
}

atp_status atp_attention_block_fwd(const atp_mesh* mesh, int32_t block_mode, int64_t batch,
                                   int64_t seq, int64_t h, int32_t heads, int32_t chunks,
                                   const atp_block_weights* w, const atp_attn_block_fwd_io* io,
                                   void* workspace, size_t ws_bytes, void* compute_stream,
                                   void* comm_stream) {
    AttnPlan ap;
    ATP_CHECK(attention_plan(mesh, block_mode, batch, seq, h, heads, &ap));
    BlockPlan P;
    ATP_CHECK(block_plan(mesh, block_mode, h, &P));
    const int64_t T = ap.T;
    ATP_CHECK(check_chunks(T, chunks));
    if (!w || !io) return set_error(ATP_ERR_INVALID_ARGUMENT, "weights or io is NULL");
    ATP_CHECK(check_attn_weights(P, w));
    ATP_CHECK(check_partial_dtype(io->partial_dtype));
    const bool kn = w->layout == ATP_W_KN;
    const bool pb16 = io->partial_dtype == ATP_BF16;
    const atp_shard& gq = P.g[0];
    const atp_shard& go = P.g[1];
    if (go.k_loc != ap.out_cols)
        return set_error(ATP_ERR_SHAPE, "out-proj contracts over %lld columns, the heads give %lld",
                         (long long)go.k_loc, (long long)ap.out_cols);
    ATP_CHECK(check_mat(io->x_loc, T, io->ldx, gq.k_loc, "x_loc"));
    ATP_CHECK(check_mat(io->qkv, T, io->ld_qkv, gq.n_loc, "qkv"));
    ATP_CHECK(check_mat(io->attn, T, io->ld_attn, go.k_loc, "attn"));
    ATP_CHECK(check_mat(io->o, T, io->ld_o, go.n_loc, "o"));
    ATP_CHECK(check_group(io->qkv_partials, gq.red_size, T, io->ldp_qkv, gq.n_loc, "qkv_partials"));
    ATP_CHECK(check_group(io->o_partials, go.red_size, T, io->ldp_o, go.n_loc, "o_partials"));
    if (T > 0) ATP_CHECK(check_vec(io->lse, "lse"));
    if (overlaps(io->qkv, T, io->ld_qkv, 2, io->attn, T, io->ld_attn, 2))
        return set_error(ATP_ERR_INVALID_ARGUMENT, "qkv and attn must not overlap");
    if (workspace && reinterpret_cast<uintptr_t>(workspace) % kWsAlign)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "workspace must be %zu-byte aligned", kWsAlign);
    // With a workspace, as in the block forward: chunk products with too few
    // tiles to fill the chip are split over k into slabs there, from W^T
    // copies kept there (weights stored [k][n]).  As for the block calls,
    // only that path may run under graph capture.
    const bool ws = workspace && ws_bytes >= ws_fwd_bytes(P, T, w->layout, 2);
    if (!ws) ATP_CHECK(refuse_capture_of_direct_path(compute_stream));
    uint16_t* wt[2] = {nullptr, nullptr};
    float* slab = nullptr;
    if (ws) {
        Carver c{static_cast<char*>(workspace)};
        if (kn)
            for (int L = 0; L < 2; ++L)
                if (fwd_may_copy_w(P, L, T)) {
                    uint16_t* t = c.take((size_t)P.g[L].n_loc * ws_pitch(P.g[L].k_loc) * 2);
                    if (!fwd_reads_w(P, L, T, chunks)) wt[L] = t;
                }
        slab = reinterpret_cast<float*>(c.take(slab_bytes(P, T, false, 2)));
    }

    Streams S(compute_stream, comm_stream);
    hipEvent_t* ev = nullptr;
    // [0] start  [1] comm end  [2] QKV reduced  [3] out-proj done, then the
    // chunk events of QKV and of out-proj
    ATP_CHECK(sync_events(4 + 2 * (size_t)chunks, &ev));
    ATP_CHECK(S.begin(ev[0]));
    auto make = [&](int L) {
        return [&, L](const void* A, void* C, int64_t ldc, bool b16, int epi, int64_t M) {
            const int64_t lda = L == 0 ? io->ldx : io->ld_attn;
            const atp_shard& g = P.g[L];
            if (wt[L])
                return gemm_problem(atp::LAYOUT_NT, A, lda, wt[L], ws_pitch(g.k_loc), C, ldc, b16,
                                    epi, M, g.n_loc, g.k_loc);
            return xw_problem(g, kn, w->w[L], w->ldw[L], A, lda, C, ldc, b16, epi, M);
        };
    };
    // W^T of linear L, written before its first product (same stream)
    auto need_wt = [&](int L) -> atp_status {
        if (!wt[L]) return ATP_OK;
        const atp_shard& g = P.g[L];
        return run_transpose(w->w[L], w->ldw[L], g.k_loc, g.n_loc, wt[L], ws_pitch(g.k_loc), S.cs);
    };
    ATP_CHECK(need_wt(0));
    ATP_CHECK(chained_linear(S, gq.red_size, gq.red_index, io->qkv_partials, io->ldp_qkv, pb16,
                             io->x_loc, io->ldx, gq.n_loc, atp::EPI_BIAS, w->b[0], nullptr,
                             io->qkv, io->ld_qkv, T, chunks, ev + 4, ev[2], make(0), slab));
    // a causal sequence spans chunks: the core waits for the whole QKV block
    HIP_CHECK(hipStreamWaitEvent(S.cs, ev[2], 0), "hipStreamWaitEvent");
    if (T > 0) {
        atp::AttentionProblem p;
        p.qkv = io->qkv;
        p.ld_qkv = io->ld_qkv;
        p.qkv_col0 = (int64_t)ap.first * 3 * kHeadDim;
        p.out = io->attn;
        p.ld_out = io->ld_attn;
        p.out_col0 = (int64_t)ap.first * kHeadDim;
        p.lse = io->lse;
        p.batch = batch;
        p.seq = seq;
        p.heads = ap.hd;
        p.head_dim = kHeadDim;
        const double pairs = (double)batch * ap.hd * (double)seq * (double)(seq + 1) / 2.0;
        ATP_CHECK(timed("attention_fwd", 4.0 * kHeadDim * pairs,
                        (double)T * ap.hd * (4.0 * kHeadDim * 2.0 + 4.0), S.cs,
                        [&] { return atp::launch_attention_fwd(p, S.cs); }));
    }
    ATP_CHECK(need_wt(1));
    ATP_CHECK(chained_linear(S, go.red_size, go.red_index, io->o_partials, io->ldp_o, pb16,
                             io->attn, io->ld_attn, go.n_loc, atp::EPI_BIAS, w->b[1], nullptr,
                             io->o, io->ld_o, T, chunks, ev + 4 + chunks, ev[3], make(1), slab));
    return S.end(ev[1]);
}

atp_status atp_attention_block_bwd(const atp_mesh* mesh, int32_t block_mode, int64_t batch,
                                   int64_t seq, int64_t h, int32_t heads, int32_t chunks,
                                   const atp_block_weights* w, const atp_attn_block_bwd_io* io,
                                   void* workspace, size_t ws_bytes, void* compute_stream,
                                   void* comm_stream) {
    AttnPlan ap;
    ATP_CHECK(attention_plan(mesh, block_mode, batch, seq, h, heads, &ap));
    BlockPlan P;
    ATP_CHECK(block_plan(mesh, block_mode, h, &P));
    const int64_t T = ap.T;
    ATP_CHECK(check_chunks(T, chunks));
    if (!w || !io) return set_error(ATP_ERR_INVALID_ARGUMENT, "weights or io is NULL");
    ATP_CHECK(check_attn_weights(P, w));
    ATP_CHECK(check_partial_dtype(io->partial_dtype));
    const bool kn = w->layout == ATP_W_KN;
    const bool pb16 = io->partial_dtype == ATP_BF16;
    const atp_shard& gq = P.g[0];
    const atp_shard& go = P.g[1];
    if (go.k_loc != ap.out_cols)
        return set_error(ATP_ERR_SHAPE, "out-proj contracts over %lld columns, the heads give %lld",
                         (long long)go.k_loc, (long long)ap.out_cols);
    ATP_CHECK(check_mat(io->x_loc, T, io->ldx, gq.k_loc, "x_loc"));
    ATP_CHECK(check_mat(io->qkv, T, io->ld_qkv, gq.n_loc, "qkv"));
    ATP_CHECK(check_mat(io->attn, T, io->ld_attn, go.k_loc, "attn"));
    ATP_CHECK(check_mat(io->d_o, T, io->ld_do, go.n_loc, "d_o"));
    ATP_CHECK(check_mat(io->d_attn, T, io->ld_d_attn, go.k_loc, "d_attn"));
    ATP_CHECK(check_mat(io->d_qkv, T, io->ld_dqkv, gq.n_loc, "d_qkv"));
    ATP_CHECK(check_mat(io->dx, T, io->ld_dx, gq.k_loc, "dx"));
    ATP_CHECK(check_group(io->d_attn_partials, go.bwd_size, T, io->ldp_da, go.k_loc,
                          "d_attn_partials"));
    ATP_CHECK(check_group(io->dx_partials, gq.bwd_size, T, io->ldp_dx, gq.k_loc, "dx_partials"));
    for (int i = 0; i < 2; ++i) {
        char nm[32];
        const atp_shard& g = P.g[i];
        snprintf(nm, sizeof nm, "dw[%s]", kLinearName[i]);
        ATP_CHECK(check_mat(io->dw[i], kn ? g.k_loc : g.n_loc, w->ldw[i], kn ? g.n_loc : g.k_loc,
                            nm));
        if (io->db[i]) {
            snprintf(nm, sizeof nm, "db[%s]", kLinearName[i]);
            ATP_CHECK(check_vec(io->db[i], nm));
        }
    }
    if (T > 0) {
        ATP_CHECK(check_vec(io->lse, "lse"));
        ATP_CHECK(check_vec(io->delta, "delta"));
    }
    if (overlaps(io->d_qkv, T, io->ld_dqkv, 2, io->qkv, T, io->ld_qkv, 2) ||
        overlaps(io->d_qkv, T, io->ld_dqkv, 2, io->attn, T, io->ld_attn, 2) ||
        overlaps(io->d_qkv, T, io->ld_dqkv, 2, io->d_attn, T, io->ld_d_attn, 2))
        return set_error(ATP_ERR_INVALID_ARGUMENT, "d_qkv must not overlap an input");
    if (workspace && reinterpret_cast<uintptr_t>(workspace) % kWsAlign)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "workspace must be %zu-byte aligned", kWsAlign);
    // dW from transposed copies when the workspace holds them (whole 16-byte
    // rows of tokens for the transposes), else from X and dY as given; only
    // the former may run under graph capture
    const bool ws = workspace && ws_bytes >= attn_ws_bwd_bytes(P, T) && T % 8 == 0;
    if (!ws) ATP_CHECK(refuse_capture_of_direct_path(compute_stream));
    uint16_t *xt_x = nullptr, *xt_a = nullptr, *dyt_q = nullptr, *dyt_o = nullptr;
    float* colpart = nullptr;
    if (ws) {
        Carver c{static_cast<char*>(workspace)};
        const size_t t2 = (size_t)ws_pitch(T) * 2;
        xt_x = c.take(gq.k_loc * t2);
        xt_a = c.take(go.k_loc * t2);
        dyt_q = c.take(gq.n_loc * t2);
        dyt_o = c.take(go.n_loc * t2);
        colpart = reinterpret_cast<float*>(c.take(colpart_bytes(P, T)));
    }
    auto dweights = [&](const atp_shard& g, int L, const void* X, int64_t ldx, const void* dY,
                        int64_t lddy, uint16_t* xt, uint16_t* dyt, hipStream_t s) {
        if (ws)
            return weight_grads_ws(g, kn, X, ldx, dY, lddy, io->dw[L], w->ldw[L], io->db[L], T,
                                   xt, dyt, colpart, s);
        return weight_grads(g, kn, X, ldx, dY, lddy, io->dw[L], w->ldw[L], io->db[L], T, s);
    };

    Streams S(compute_stream, comm_stream);
    hipEvent_t* ev = nullptr;
    // [0] start  [1] comm end  [2] d_attn reduced  [3] QKV dX done, then the
    // chunk events of out-proj's dX and of QKV's dX
    ATP_CHECK(sync_events(4 + 2 * (size_t)chunks, &ev));
    ATP_CHECK(S.begin(ev[0]));
    auto make = [&](int L, const void* dY, int64_t lddy) {
        return [&, L, lddy](const void* A, void* C, int64_t ldc, bool b16, int epi, int64_t M) {
            return dyw_problem(P.g[L], kn, w->w[L], w->ldw[L], A, lddy, C, ldc, b16, epi, M);
        };
    };
    // out-proj: dX chunks (reduced on ms into d_attn), then its dW and db
    // on cs while those reductions drain
    ATP_CHECK(chained_linear(S, go.bwd_size, go.bwd_index, io->d_attn_partials, io->ldp_da, pb16,
                             io->d_o, io->ld_do, go.k_loc, atp::EPI_NONE, nullptr, nullptr,
                             io->d_attn, io->ld_d_attn, T, chunks, ev + 4, ev[2],
                             make(1, io->d_o, io->ld_do)));
    ATP_CHECK(dweights(go, 1, io->attn, io->ld_attn, io->d_o, io->ld_do, xt_a, dyt_o, S.cs));
    // the core's backward reads the device's columns of the whole d_attn
    HIP_CHECK(hipStreamWaitEvent(S.cs, ev[2], 0), "hipStreamWaitEvent");
    if (T > 0) {
        atp::AttentionBwdProblem p;
        p.qkv = io->qkv;
        p.ld_qkv = io->ld_qkv;
        p.qkv_col0 = (int64_t)ap.first * 3 * kHeadDim;
        p.out = io->attn;
        p.ld_out = io->ld_attn;
        p.out_col0 = (int64_t)ap.first * kHeadDim;
        p.dout = io->d_attn;
        p.ld_dout = io->ld_d_attn;
        p.lse = io->lse;
        p.delta = io->delta;
        p.dqkv = io->d_qkv;
        p.ld_dqkv = io->ld_dqkv;
        p.batch = batch;
        p.seq = seq;
        p.heads = ap.hd;
        p.head_dim = kHeadDim;
        const double pairs = (double)batch * ap.hd * (double)seq * (double)(seq + 1) / 2.0;
        ATP_CHECK(timed("attention_bwd", 2.0 * kHeadDim * pairs * 5.0,
                        (double)T * ap.hd * (10.0 * kHeadDim * 2.0 + 12.0), S.cs,
                        [&] { return atp::launch_attention_bwd(p, S.cs); }));
    }
    // QKV: dX chunks from the gathered d_qkv (reduced on ms into dx), dW, db
    ATP_CHECK(chained_linear(S, gq.bwd_size, gq.bwd_index, io->dx_partials, io->ldp_dx, pb16,
                             io->d_qkv, io->ld_dqkv, gq.k_loc, atp::EPI_NONE, nullptr, nullptr,
                             io->dx, io->ld_dx, T, chunks, ev + 4 + chunks, ev[3],
                             make(0, io->d_qkv, io->ld_dqkv)));
    ATP_CHECK(dweights(gq, 0, io->x_loc, io->ldx, io->d_qkv, io->ld_dqkv, xt_x, dyt_q, S.cs));
    return S.end(ev[1]);
}

void atp_profile_enable(int32_t on) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_prof_on = (on != 0);
    g_prof_detail = (on == 2);
}

int32_t atp_profile_collect(atp_kernel_stat* out, int32_t max) {
    std::vector<ProfRec> recs;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        recs.swap(g_prof);
    }
    std::vector<atp_kernel_stat> agg;
    int32_t rc = 0;
    for (const ProfRec& r : recs) {
        float ms = 0.0f;
        if (hipEventSynchronize(r.end) != hipSuccess ||
            hipEventElapsedTime(&ms, r.beg, r.end) != hipSuccess) {
            rc = -1;
        }
        size_t i = 0;
        for (; i < agg.size(); ++i)
            if (strncmp(agg[i].name, r.name.c_str(), sizeof agg[i].name - 1) == 0) break;
        if (i == agg.size()) {
            atp_kernel_stat st;
            memset(&st, 0, sizeof st);
            snprintf(st.name, sizeof st.name, "%s", r.name.c_str());
            agg.push_back(st);
        }
        agg[i].launches += 1;
        agg[i].total_ms += ms;
        agg[i].flops += r.flops;
        agg[i].bytes += r.bytes;
    }
    {
        std::lock_guard<std::mutex> lk(g_mu);
        for (const ProfRec& r : recs) {
            g_prof_free.push_back(r.beg);
            g_prof_free.push_back(r.end);
        }
    }
    if (rc < 0) {
        g_last_error = "hipEventElapsedTime failed";
        return -1;
    }
    int32_t n = 0;
    for (; n < (int32_t)agg.size() && n < max; ++n) out[n] = agg[n];
    return n;
}

}  // extern "C"
