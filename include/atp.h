/*
 * atp.h -- C ABI of the MI355X (gfx950) ATP shard-block library.
 *
 * One device's share of a transformer layer under ATP's row-first /
 * column-first 2D tensor parallelism (Cheng, Liu, Du, You, "ATP: Adaptive
 * Tensor Parallelism for Foundation Models", arXiv 2301.08658):
 * the sharded QKV, out-projection, fc1 (+bias+GeLU) and fc2 GEMMs, the
 * reduction of their Partial(SUM) outputs, and the token-chunk pipeline
 * that overlaps each chunk's reduction with the next chunk's GEMM.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Mesh (Sec. 3.1): DeviceMesh(d1, d2); this device sits at (i1, i2),
 *    rank = i1 * d2 + i2.
 *  - Y = X W with X [tokens, k] and W [k, n] (Sec. 3.2, "Y = XW").
 *      ATP_ROW_FIRST: W spec [Shard(0), Shard(1)]: local W rows
 *        [i1*k/d1, (i1+1)*k/d1), columns [i2*n/d2, (i2+1)*n/d2); X holds
 *        the matching k/d1 columns; the output block is Partial(SUM) over
 *        the d1 devices that share i2 (mesh axis 0).
 *      ATP_COL_FIRST: W spec [Shard(1), Shard(0)]: local W rows
 *        [i2*k/d2, ...), columns [i1*n/d1, ...); the output is Partial(SUM)
 *        over the d2 devices that share i1 (mesh axis 1).
 *    In the backward pass (Sec. 4.2) the input gradient dX = dY W^T is
 *    partial over the other axis (the one that split n).
 *  - Tensors are row-major device buffers owned by the caller: element
 *    (r, c) of a matrix with leading dimension ld is at base[r * ld + c].
 *    bf16 = IEEE bfloat16 bits (uint16), f32 = IEEE binary32.
 *    Every device pointer must be 16-byte aligned, every leading dimension
 *    and every local column count a multiple of 8 elements, and leading
 *    dimensions at most 4M (2^22) elements.
 *  - Streams and events are hipStream_t / hipEvent_t passed as void*;
 *    NULL means the default stream.  Calls only enqueue work and return.
 *  - Chunks (Sec. 4.1): the token rows are split into `chunks` contiguous
 *    equal parts; tokens % chunks must be 0.  Chunking never changes a
 *    value: every output element is computed by the same instructions in
 *    the same order whatever the chunk count.
 *  - Reductions sum the group's buffers in group order 0..d-1, so every
 *    member of a group obtains bit-identical results.
 *  - Errors: all arguments are checked before anything is enqueued; a
 *    non-OK status means nothing was enqueued.  atp_last_error() returns
 *    a per-thread message for the last failure.  A HIP launch failure
 *    after checks passed returns ATP_ERR_DEVICE (work enqueued before it
 *    may have run).
 *  - The library never allocates device memory.
 */
#ifndef ATP_H
#define ATP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    ATP_OK = 0,
    ATP_ERR_INVALID_ARGUMENT = 1, /* null pointer, coordinate out of range, bad enum, ld < cols */
    ATP_ERR_SHAPE = 2,            /* k or n not divisible by the mesh, tokens % chunks != 0 */
    ATP_ERR_UNSUPPORTED = 3,      /* alignment, multiple-of-8 rule, group larger than ATP_MAX_GROUP */
    ATP_ERR_DEVICE = 4            /* a HIP call failed */
} atp_status;

typedef enum { ATP_ROW_FIRST = 0, ATP_COL_FIRST = 1 } atp_mode;

/* ATP_BLOCK_COL: the layer of Sec. 3.2.1 -- QKV and fc1 column-first,
 * out-proj and fc2 row-first.  ATP_BLOCK_ROW: the transposed arrangement
 * (QKV and fc1 row-first, out-proj and fc2 column-first); on mesh (d1, d2)
 * it has the local shapes of ATP_BLOCK_COL on (d2, d1). */
typedef enum { ATP_BLOCK_COL = 0, ATP_BLOCK_ROW = 1 } atp_block_mode;

/* Epilogues (Sec. 2.1 and 3.2.1).  With s the reduced sum:
 *   NONE: s;  BIAS: s + b[n];  BIAS_GELU: GeLU(s + b[n]) with the exact erf
 *   form, optionally saving s + b[n];  GELU_BWD: s * GeLU'(pre[t, n]). */
typedef enum {
    ATP_EPI_NONE = 0,
    ATP_EPI_BIAS = 1,
    ATP_EPI_BIAS_GELU = 2,
    ATP_EPI_GELU_BWD = 3
} atp_epilogue;

typedef enum { ATP_F32 = 0, ATP_BF16 = 1 } atp_dtype;

#define ATP_MAX_GROUP 64   /* largest reduction group (d1 or d2) */
#define ATP_MAX_CHUNKS 64

typedef struct { int32_t d1, d2, i1, i2; } atp_mesh;

/* Local block of one linear (Sec. 3.2): W rows [k_off, k_off + k_loc),
 * columns [n_off, n_off + n_loc); forward reduction over mesh axis
 * red_axis (group size red_size, this device at red_index); backward
 * input-gradient reduction over bwd_axis (bwd_size, bwd_index). */
typedef struct {
    int64_t k_loc, n_loc, k_off, n_off;
    int32_t red_axis, red_size, red_index;
    int32_t bwd_axis, bwd_size, bwd_index;
} atp_shard;

/* Shard geometry of Y = XW, Sec. 3.2 (local sizes [b, h1/d1] x [h1/d1, h2/d2]
 * for row-first; communicated block [b, h2/d1] for column-first).
 * Host only, no device work.  Errors: INVALID_ARGUMENT (null, d <= 0,
 * coordinate out of range, bad mode), SHAPE (k or n not divisible). */
atp_status atp_shard_geometry(const atp_mesh* mesh, int32_t mode, int64_t k, int64_t n,
                              atp_shard* out);

/* Local GEMM of one shard linear, chunked (Sec. 3.2, Sec. 4.1):
 *   y[t, :] = epi( x_loc[t, :] . w_loc )   for t in each chunk, in order.
 * x_loc  bf16 [tokens, k_loc], ld ldx.   w_loc bf16 [k_loc, n_loc], ld ldw.
 * If the reduction group has more than one member, y is this device's
 * Partial(SUM) block: epi must be ATP_EPI_NONE (the bias and GeLU belong
 * after the reduction); y_dtype ATP_F32, or ATP_BF16 for partials kept in
 * the training precision as the paper all-reduces them (Sec. 5: FP16),
 * reduced by atp_chunked_partial_reduce_bf16.  With a group of one, epi may
 * be NONE, BIAS or BIAS_GELU and y f32 or bf16; bias_loc bf16 [n_loc]
 * (the block n_off..), preact (nullable, bf16, ld ldy) receives s + b for
 * BIAS_GELU.  chunk_done (nullable) holds `chunks` caller-created events;
 * event c is recorded on `stream` once chunk c's rows of y are written. */
atp_status atp_shard_linear_fwd(const atp_mesh* mesh, int32_t mode, int64_t tokens,
                                int64_t k, int64_t n, int32_t chunks,
                                const void* x_loc, int64_t ldx,
                                const void* w_loc, int64_t ldw,
                                const void* bias_loc, int32_t epi,
                                void* y, int32_t y_dtype, int64_t ldy, void* preact,
                                void* stream, void* const* chunk_done);

/* Reduction of a group's Partial(SUM) blocks -- the arithmetic of the
 * grouped all-reduce of Sec. 3.2 (Sec. 3.1, Partial(SUM)) -- chunked so
 * that chunk c can start as soon as its partials are ready (Sec. 4.1):
 *   out[t, n] = epi( sum_{j=0..red_size-1} partials[j][t * ldp + n] ).
 * partials: host array of red_size device pointers, f32 [tokens, ldp];
 * on one GPU the other members' buffers stand in for the peers' data.
 * bias_loc bf16 [n_loc] for BIAS / BIAS_GELU.  preact_in (bf16, ld ldo)
 * for GELU_BWD; preact_out (nullable, bf16, ld ldo) for BIAS_GELU.
 * out is f32 or bf16 (round to nearest even).  chunk_ready (nullable):
 * `chunks` events; the stream waits for event c before reducing chunk c.
 * Errors: INVALID_ARGUMENT for red_size < 1, a null entry, missing bias or
 * preact_in; UNSUPPORTED for red_size > ATP_MAX_GROUP. */
atp_status atp_chunked_partial_reduce(int32_t red_size, int64_t tokens, int64_t n_loc,
                                      int32_t chunks, const float* const* partials,
                                      int64_t ldp, const void* bias_loc, int32_t epi,
                                      const void* preact_in, void* out, int32_t out_dtype,
                                      int64_t ldo, void* preact_out, void* stream,
                                      void* const* chunk_ready);

/* The same reduction over bf16 Partial(SUM) blocks (partials: red_size
 * device pointers, bf16 [tokens, ldp]): each value widened to f32 and
 * summed in group order, then epi as above.  This is the variant of Sec. 5's
 * half-precision training, where the all-reduced activations are 16-bit;
 * it halves the bytes each reduction reads.  Errors as above. */
atp_status atp_chunked_partial_reduce_bf16(int32_t red_size, int64_t tokens, int64_t n_loc,
                                           int32_t chunks, const void* const* partials,
                                           int64_t ldp, const void* bias_loc, int32_t epi,
                                           const void* preact_in, void* out, int32_t out_dtype,
                                           int64_t ldo, void* preact_out, void* stream,
                                           void* const* chunk_ready);

/* One shard linear with the group's reduction fused into the GEMM's
 * epilogue: the fused GEMM-and-all-reduce design that Sec. 4.1 contrasts
 * with chunked overlapping.  In one launch, unchunked:
 *   out[t, :] = epi( sum_{j=0..red_size-1} P_j[t, :] ),
 * with P_own = x_loc[t, :] . w_loc formed in the tile's registers and never
 * stored, and P_j (j != red_index) read from peers[j] (f32 [tokens, ldp],
 * the other members' partials; peers[red_index] is not read and may be
 * NULL).  The terms are summed in group order, so out has the same bits as
 * atp_shard_linear_fwd + atp_chunked_partial_reduce on the same inputs.
 * x_loc, w_loc, bias_loc, epi (NONE, BIAS, BIAS_GELU), preact (nullable,
 * bf16, ld ldo) as for atp_shard_linear_fwd; out f32 or bf16.
 * Errors: as atp_shard_linear_fwd; UNSUPPORTED for a group of more than 8;
 * INVALID_ARGUMENT for a missing peer or GELU_BWD. */
atp_status atp_shard_linear_fwd_fused(const atp_mesh* mesh, int32_t mode, int64_t tokens,
                                      int64_t k, int64_t n, const void* x_loc, int64_t ldx,
                                      const void* w_loc, int64_t ldw,
                                      const float* const* peers, int64_t ldp,
                                      const void* bias_loc, int32_t epi, void* out,
                                      int32_t out_dtype, int64_t ldo, void* preact,
                                      void* stream);

/* Backward of one shard linear (Sec. 4.2): with dy the gradient of this
 * device's reduced output block (bf16 [tokens, n_loc], ld lddy),
 *   dx_partial = dy . w_loc^T   f32 [tokens, k_loc], ld lddx -- partial over
 *                               the backward group (bwd_size members);
 *   dw         = x_loc^T . dy   f32 [k_loc, n_loc], ld lddw (complete);
 *   db         = sum_t dy       f32 [n_loc] (nullable).
 * dX is computed first, chunk by chunk, recording dx_chunk_done[c]
 * (nullable) so its reduction can overlap the dW GEMM that follows on the
 * same stream. */
atp_status atp_shard_linear_bwd(const atp_mesh* mesh, int32_t mode, int64_t tokens,
                                int64_t k, int64_t n, int32_t chunks,
                                const void* x_loc, int64_t ldx,
                                const void* w_loc, int64_t ldw,
                                const void* dy, int64_t lddy,
                                float* dx_partial, int64_t lddx,
                                float* dw, int64_t lddw, float* db,
                                void* stream, void* const* dx_chunk_done);

/* Storage order of a local weight block.  ATP_W_KN: [k_loc][n_loc], the
 * paper's Y = XW orientation (Sec. 3.2).  ATP_W_NK: [n_loc][k_loc], W^T, the
 * way torch.nn.Linear keeps its weight ([out_features, in_features]). */
typedef enum { ATP_W_KN = 0, ATP_W_NK = 1 } atp_weight_layout;

/* Local weights of the block; index 0..3 = qkv [h,3h], out [h,h],
 * fc1 [h,4h], fc2 [4h,h] (Sec. 2.1).  Each w[i] is the device's bf16
 * block, [k_loc][n_loc] or [n_loc][k_loc] as `layout` says (ld ldw[i]);
 * b[i] its bf16 bias block [n_loc].  A zero-filled struct means ATP_W_KN. */
typedef struct {
    const void* w[4];
    int64_t ldw[4];
    const void* b[4];
    int32_t layout;   /* atp_weight_layout, the same for all four */
} atp_block_weights;

/* Forward inputs and outputs of the block (Sec. 3.2.1).
 *  x_loc   bf16 [tokens, h_x]: the layer-input columns QKV and fc1
 *          contract over (h/d2 for COL, h/d1 for ROW).
 *  attn_loc bf16 [tokens, h_a]: the attention-core output columns that
 *          feed out-proj (h/d1 for COL, h/d2 for ROW).
 *  partials[i]: host array of the red_size device pointers of linear i's
 *          group ([tokens, ldp[i]] of partial_dtype); entry red_index is
 *          this device's own buffer and is written, the others are read.
 *          Unused (may be NULL) when the group has one member.
 *  partial_dtype: ATP_F32 (a zero-filled struct), or ATP_BF16 for the
 *          16-bit Partial(SUM) blocks of Sec. 5's half-precision training:
 *          the own partial is rounded once to bf16 (nearest even) and the
 *          group's bf16 values are summed in f32, halving the bytes every
 *          reduction reads.
 *  qkv, o, h, z: bf16 reduced outputs (+bias; h = GeLU(...)); pre: bf16
 *          fc1 pre-activation saved for the backward, ld ld_h. */
typedef struct {
    const void* x_loc;
    int64_t ldx;
    const void* attn_loc;
    int64_t lda;
    void* const* partials[4];
    int64_t ldp[4];
    void* qkv; int64_t ld_qkv;
    void* o;   int64_t ld_o;
    void* h;   int64_t ld_h;
    void* pre;
    void* z;   int64_t ld_z;
    int32_t partial_dtype;
} atp_block_fwd_io;

/* Backward inputs and outputs of the block (Sec. 4.2).
 *  x_loc, attn_loc, h, pre: the forward's inputs and saved activations.
 *  dz, dqkv, d_o: bf16 gradients of the reduced outputs z, qkv, o.
 *  dx_partials[i]: host array of the bwd_size device pointers of linear
 *          i's backward group ([tokens, ld_dxp[i]] of partial_dtype, f32 or
 *          bf16 as in atp_block_fwd_io), own entry written.
 *  dh_pre: bf16 fc1 upstream gradient = (reduced fc2 dX) * GeLU'(pre).
 *  dx_qkv, dx_fc1, d_attn: bf16 reduced input gradients.
 *  dw[i] f32 in the weights' layout and leading dimension ([k_loc][n_loc]
 *  for ATP_W_KN, [n_loc][k_loc] for ATP_W_NK), db[i] f32 [n_loc]. */
typedef struct {
    const void* x_loc;    int64_t ldx;
    const void* attn_loc; int64_t lda;
    const void* h;        int64_t ld_h;
    const void* pre;
    const void* dz;   int64_t ld_dz;
    const void* dqkv; int64_t ld_dqkv;
    const void* d_o;  int64_t ld_do;
    void* const* dx_partials[4];
    int64_t ld_dxp[4];
    void* dh_pre;
    void* dx_qkv; int64_t ld_dx_qkv;
    void* dx_fc1; int64_t ld_dx_fc1;
    void* d_attn; int64_t ld_d_attn;
    float* dw[4];
    float* db[4];
    int32_t partial_dtype;
} atp_block_bwd_io;

/* Workspace for the block calls' transposed-layout path (bytes): the larger
 * of the forward's need and the backward's for weights in `weight_layout`
 * (atp_weight_layout).  The forward keeps W^T of a weight stored
 * [k_loc][n_loc] (n_loc rows of k_loc + 64 bf16 values) when, at some
 * valid chunk count, its products are split over k or are not shaped for
 * the 256 x 256 tiles that stream W as stored as fast as W^T; weights
 * stored [n_loc][k_loc] need no copy.  The backward keeps X^T of x, the attention
 * block and H, and dY^T of the four linears (cols rows of tokens + 64 bf16
 * values each), for weights stored [n_loc][k_loc] one copy of the largest
 * weight in [k_loc][n_loc] order (k_loc rows of n_loc + 64 values, reused
 * linear by linear), and the fp32 column partials of dY that the
 * transposes leave for db (ceil(tokens / 64) rows of the widest linear's
 * columns).  Each side adds the fp32 split-K slabs of the chunked products
 * that feed a reduction (S * chunk rows * cols * 4 bytes for the largest
 * split plan S over every valid chunk count).  The 64 values of padding
 * keep row pitches off memory-channel-aligned strides; every piece is
 * rounded up to 256 bytes.  `chunks` does not change the size.
 * Returns 0 for invalid arguments. */
size_t atp_block_workspace_bytes(const atp_mesh* mesh, int32_t block_mode, int64_t tokens,
                                 int64_t h, int32_t chunks, int32_t weight_layout);

/* Which path a block call takes (pass 0: atp_block_fwd, 1: atp_block_bwd)
 * for a workspace of ws_bytes bytes: 1 the transposed-layout path (the
 * workspace holds the pass's need, and for the backward tokens % 8 == 0),
 * 0 the direct path, -1 for invalid arguments.  Host only.  A block call
 * that would take the direct path refuses a compute stream under HIP graph
 * capture (see atp_block_fwd). */
int32_t atp_block_workspace_path(const atp_mesh* mesh, int32_t block_mode, int64_t tokens,
                                 int64_t h, int32_t weight_layout, size_t ws_bytes, int32_t pass);

/* Shard geometry of the block's four linears, out[0..3] = qkv, out, fc1,
 * fc2, each as atp_shard_geometry gives it for the linear's mode in
 * block_mode (Sec. 3.2.1: ATP_BLOCK_COL runs QKV and fc1 column-first,
 * out-proj and fc2 row-first).  Host only.  Errors: those of
 * atp_shard_geometry; UNSUPPORTED when a local size is not a multiple
 * of 8. */
atp_status atp_block_geometry(const atp_mesh* mesh, int32_t block_mode, int64_t h,
                              atp_shard out[4]);

/* The device's heads of the attention block (Sec. 3.2.1): its QKV block
 * holds *per_block whole heads of dimension h / heads; the block is
 * scattered over the group that reduced it, and the device attends over
 * heads [*first, *first + *count) of the block (block-local indices).
 * Host only.  Errors: those of atp_block_geometry; SHAPE when h is not a
 * multiple of heads, the QKV block does not hold whole heads or its heads
 * do not divide over the group. */
atp_status atp_attention_heads(const atp_mesh* mesh, int32_t block_mode, int64_t h,
                               int32_t heads, int32_t* first, int32_t* count,
                               int32_t* per_block);

/* Transpose a bf16 matrix: dst[c * ldd + r] = src[r * lds + c] for r < rows,
 * c < cols.  A data-layout step for the products of Sec. 3.2 / 4.2 (it turns
 * an operand contiguous along its M/N side into one contiguous along the
 * contraction), not part of the paper's arithmetic.  src [rows][lds] and dst
 * [cols][ldd] are 16-byte aligned with leading dimensions that are multiples
 * of 8 (at most 2^22); rows and cols may be any size (with either 0 nothing
 * is read or written and the pointers may be NULL); the buffers must not be
 * the same.
 * Errors: INVALID_ARGUMENT for negative sizes, NULL or aliased buffers,
 * leading dimensions below the row length; UNSUPPORTED for alignment. */
atp_status atp_transpose_bf16(int64_t rows, int64_t cols, const void* src, int64_t lds, void* dst,
                              int64_t ldd, void* stream);

/* One device's forward share of the layer (Sec. 3.2.1) with chunk-based
 * overlapping (Sec. 4.1).  Each linear's GEMM runs chunk by chunk; each
 * chunk's reduction runs on comm_stream as soon as that chunk's partial is
 * written; fc2's chunk c waits for fc1's reduced chunk c.  A group of one
 * needs no reduction: its bias (and GeLU) are applied in the GEMM epilogue
 * and it runs as one launch.  The GEMMs are issued on compute_stream in the
 * order out-proj, fc1, then QKV and fc2 (the one whose reductions read fewer
 * bytes last); with chunks > 1, comm_stream != compute_stream and outside
 * HIP graph capture, every other chunk product of a linear whose chunks do
 * not split over k runs on a second stream the library keeps per host
 * thread and device (default priority, never destroyed), so a chunk's
 * product can start on the CUs the previous chunk leaves idle; the call
 * joins that stream back into compute_stream before it returns.  With
 * comm_stream == compute_stream nothing overlaps.
 * workspace (nullable, 256-byte aligned): when ws_bytes is at least the
 * forward's need (atp_block_workspace_path) the products run with both
 * operands contiguous along k, the faster layout (weights stored
 * [k_loc][n_loc] are first copied there as W^T, except for a linear whose
 * products, at this chunk count, run unsplit on the 256 x 256 tiles that
 * stream W as stored as fast; weights stored [n_loc][k_loc] already are
 * contiguous along k), and a chunk product with too few output
 * tiles to fill the chip is split over its contraction, the splits' fp32
 * slabs summed in split order into the own partial before the chunk's
 * reduction reads it.  Without the workspace the products read W as
 * stored.  Every layout sums each element's products in the same order:
 * the paths give the same bits except where a product splits (then they
 * agree to fp32 rounding).  Results do not depend on the streams used, and
 * are the same for every chunk count that gives each chunk product the same
 * split plan (without a workspace: every chunk count).  compute_stream's
 * earlier work happens before the block's, and on return compute_stream is
 * ordered after all of it; the workspace may be reused once compute_stream
 * reaches that point.  A call that would take the direct path refuses a
 * compute_stream under HIP graph capture (UNSUPPORTED) before enqueueing
 * anything.  Concurrent calls from different host threads are safe (each
 * thread keeps its own synchronisation events). */
atp_status atp_block_fwd(const atp_mesh* mesh, int32_t block_mode, int64_t tokens, int64_t h,
                         int32_t chunks, const atp_block_weights* w,
                         const atp_block_fwd_io* io, void* workspace, size_t ws_bytes,
                         void* compute_stream, void* comm_stream);

/* One device's backward share of the layer (Sec. 4.2): dX = dY W^T per
 * linear, chunked and reduced on comm_stream where its group has more than
 * one member, dW = X^T dY and db = column sums of dY; fc1's dY is fc2's
 * reduced dX times GeLU'(pre).  Issue order on compute_stream: fc2's dX
 * (fc1 waits for it), QKV's and out-proj's dX, fc1's dX, then the four dW
 * largest first, so the dX reductions overlap the later GEMMs.
 * workspace: when ws_bytes is at least the backward's need and tokens % 8
 * == 0 (atp_block_workspace_path), X^T and dY^T are written there and every
 * dW runs from them, weights stored [n_loc][k_loc] are copied there in
 * [k_loc][n_loc] order for the dX products, and the chunked dX products are
 * split over their contraction as in atp_block_fwd; otherwise every product
 * reads its operands as stored.  The paths give the same bits except where
 * a product splits (as in atp_block_fwd).  On return compute_stream is
 * ordered after all work.  Graph capture and threads as atp_block_fwd. */
atp_status atp_block_bwd(const atp_mesh* mesh, int32_t block_mode, int64_t tokens, int64_t h,
                         int32_t chunks, const atp_block_weights* w,
                         const atp_block_bwd_io* io, void* workspace, size_t ws_bytes,
                         void* compute_stream, void* comm_stream);

/* One device's attention core (Sec. 2.1 Formula (mha), causal; the
 * attention block of Sec. 3.2.1).  qkv is the device's reduced QKV output
 * block for block_mode on the mesh (bf16 [batch*seq, ld_qkv], token rows
 * sequence-major, the n_loc columns atp_block_fwd's QKV linear produces).
 * The block holds n_loc / 384 whole heads of dimension h / heads, which
 * must be 128, each as [q | k | v] columns.  The block is replicated over
 * the group that reduced it; the attention block scatters it over that
 * group, so the device attends over the r-th of g equal runs of heads,
 * r = its index in the group, g = the group's size.  The output goes to
 * out (bf16 [batch*seq, ld_out], at least n_loc / 3 columns: the gathered
 * input of out-proj): the device writes its heads' columns, the r-th run of
 * h/heads-wide column blocks, and leaves the other members' columns (the
 * all-gather) alone.  lse (fp32 [heads_of_device][batch*seq]) receives the
 * natural-log softmax denominator of every row, for the backward.  The
 * caller owns every buffer; work is enqueued on `stream`.
 * Errors: INVALID_ARGUMENT for a bad mesh, negative sizes, NULL buffers,
 * qkv and out sharing memory, ld below the row length; SHAPE when h is not
 * a multiple of heads or the heads do not divide over the group;
 * UNSUPPORTED for a head dimension other than 128, sizes above 2^24,
 * misalignment. */
atp_status atp_attention_fwd(const atp_mesh* mesh, int32_t block_mode, int64_t batch, int64_t seq,
                             int64_t h, int32_t heads, const void* qkv, int64_t ld_qkv,
                             void* out, int64_t ld_out, float* lse, void* stream);

/* Gradient of atp_attention_fwd (Sec. 2.1 Formula (mha), the backward of
 * Sec. 4.2 applied to the attention core).  qkv, out and lse are the
 * forward's input, output (the gathered block; the device's columns are
 * read) and saved row log-sum-exps; d_out (bf16, same shape and columns as
 * out) is the gradient of the gathered out-proj input.  The device writes
 * dq, dk, dv of its heads into d_qkv (bf16, the QKV block's shape and
 * column order) at its heads' columns and leaves the other members'
 * columns alone (the conjugate of the scatter).  delta is caller-owned fp32
 * scratch of heads_of_device * batch * seq values.  P is recomputed from
 * lse; with delta_t = dO_t . O_t: dV = P^T dO, dS = P o (dO V^T - delta),
 * dQ = dS K / sqrt(d), dK = dS^T Q / sqrt(d), each accumulated by one
 * workgroup (deterministic).  Errors as atp_attention_fwd; d_qkv must not
 * share memory with qkv, out or d_out (INVALID_ARGUMENT). */
atp_status atp_attention_bwd(const atp_mesh* mesh, int32_t block_mode, int64_t batch, int64_t seq,
                             int64_t h, int32_t heads, const void* qkv, int64_t ld_qkv,
                             const void* out, int64_t ld_out, const float* lse, const void* d_out,
                             int64_t ld_dout, void* d_qkv, int64_t ld_dqkv, float* delta,
                             void* stream);

/* The attention block of one device (Sec. 3.2.1, with Sec. 2.1 Formula
 * (mha) as its core), chained: QKV (chunked, reduced with its bias over its
 * group) -> scatter of the reduced QKV block's heads over that group ->
 * causal attention core on the device's run of heads -> all-gather of the
 * heads' outputs (the out-proj input block) -> out-proj (chunked, reduced
 * with its bias).  One GPU holds one device: the all-gather's other columns
 * are the peers' data, as the partial tables are.
 *  x_loc        bf16 [tokens, k_loc of QKV]: the layer input block.
 *  qkv_partials host table of the QKV group's red_size buffers
 *               ([tokens, ldp_qkv] of partial_dtype; own entry written).
 *  qkv          bf16 [tokens, n_loc of QKV]: reduced QKV block (+ bias),
 *               written; token rows sequence-major (b * seq + t).
 *  attn         bf16 [tokens, k_loc of out-proj]: the gathered out-proj
 *               input.  The call writes its heads' columns (as
 *               atp_attention_fwd); the other columns must hold the other
 *               group members' outputs when the call is made.
 *  lse          fp32 [heads of the device][tokens], written.
 *  o_partials / o: out-proj's partial table and reduced output (+ bias).
 * Weights: entries 0 (qkv) and 1 (out) of w, in w->layout; 2 and 3 are
 * not read.  The attention core starts once the whole QKV block is reduced
 * (a causal sequence spans chunks), out-proj's chunks follow on
 * compute_stream and their reductions overlap the next chunk's GEMM on
 * comm_stream (Sec. 4.1).
 * workspace / ws_bytes: optional, caller-owned device memory (256-byte
 * aligned; atp_block_workspace_bytes() for the same mesh, mode, tokens, h,
 * chunks and weight layout is enough).  With it, as in atp_block_fwd, a
 * chunk product with too few tiles to fill the chip is split over k into
 * fp32 slabs there, summed in split order (so its bits can differ from the
 * unsplit product's by fp32 rounding), and weights stored [k][n] are copied
 * there as W^T where the products stream faster from it; without it the
 * products read the weights as stored.  Nothing in the workspace is read
 * before the call writes it.
 * Without such a workspace the call refuses a compute_stream under HIP
 * graph capture (as the block calls do).  Errors as atp_block_fwd and
 * atp_attention_fwd. */
typedef struct {
    const void* x_loc; int64_t ldx;
    void* const* qkv_partials; int64_t ldp_qkv;
    void* qkv; int64_t ld_qkv;
    void* attn; int64_t ld_attn;
    float* lse;
    void* const* o_partials; int64_t ldp_o;
    void* o; int64_t ld_o;
    int32_t partial_dtype;
} atp_attn_block_fwd_io;

atp_status atp_attention_block_fwd(const atp_mesh* mesh, int32_t block_mode, int64_t batch,
                                   int64_t seq, int64_t h, int32_t heads, int32_t chunks,
                                   const atp_block_weights* w, const atp_attn_block_fwd_io* io,
                                   void* workspace, size_t ws_bytes, void* compute_stream,
                                   void* comm_stream);

/* Backward of atp_attention_block_fwd (Sec. 4.2 through the chain):
 * out-proj's dX (chunked, reduced over its backward group) gives d_attn;
 * out-proj's dW and db; the attention core's backward on the device's heads
 * writes their dq, dk, dv columns of d_qkv (the conjugate of the scatter);
 * QKV's dX (chunked, reduced over its backward group), dW and db follow.
 *  x_loc, qkv, attn, lse: the forward's input, outputs and saved lse.
 *  d_o          bf16 gradient of o.
 *  d_attn_partials / d_attn: out-proj's backward table and the reduced
 *               gradient of the gathered block (bf16, written).
 *  delta        fp32 scratch of heads-of-device * tokens values.
 *  d_qkv        bf16 [tokens, n_loc of QKV]: the device's heads' columns are
 *               written; the other columns must hold the other group
 *               members' (the all-gather of the QKV block's gradient).
 *  dx_partials / dx: QKV's backward table and reduced input gradient.
 *  dw[0], db[0] (qkv), dw[1], db[1] (out): f32, as atp_block_bwd_io
 *               (dw in the weights' layout and leading dimension; db
 *               nullable).
 * workspace / ws_bytes: optional, caller-owned device memory (256-byte
 * aligned).  A workspace of atp_block_workspace_bytes() bytes for the same
 * mesh, mode, tokens, h and weight layout (or larger), with tokens a
 * multiple of 8, runs both dW products from transposed copies of X and dY
 * kept there (both operands contiguous along the tokens) and forms db from
 * the dY transpose; otherwise dW reads X and dY as given.  Both paths give
 * the same bits.  The workspace is scratch: nothing in it is read before
 * the call writes it.
 * Without such a workspace (or with tokens not a multiple of 8) the call
 * refuses a compute_stream under HIP graph capture.  Errors as
 * atp_block_bwd and atp_attention_bwd. */
typedef struct {
    const void* x_loc; int64_t ldx;
    const void* qkv; int64_t ld_qkv;
    const void* attn; int64_t ld_attn;
    const float* lse;
    const void* d_o; int64_t ld_do;
    void* const* d_attn_partials; int64_t ldp_da;
    void* d_attn; int64_t ld_d_attn;
    float* delta;
    void* d_qkv; int64_t ld_dqkv;
    void* const* dx_partials; int64_t ldp_dx;
    void* dx; int64_t ld_dx;
    float* dw[2];
    float* db[2];
    int32_t partial_dtype;
} atp_attn_block_bwd_io;

atp_status atp_attention_block_bwd(const atp_mesh* mesh, int32_t block_mode, int64_t batch,
                                   int64_t seq, int64_t h, int32_t heads, int32_t chunks,
                                   const atp_block_weights* w, const atp_attn_block_bwd_io* io,
                                   void* workspace, size_t ws_bytes, void* compute_stream,
                                   void* comm_stream);

/* atp_attention_bwd without the delta argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): delta lives in a scratch array
 * the library holds on each GPU it runs on (4 MiB, 2^20 fp32 values, kept
 * until the process ends; its address is looked up once per device, on the
 * first call there).  The call allocates nothing.  heads-of-device * batch *
 * seq must be at most 2^20, else ATP_ERR_UNSUPPORTED before any work.  Every
 * call on one GPU shares that GPU's array (the backward writes each value
 * before reading it, so nothing needs clearing): calls that overlap on one
 * GPU -- on different streams, or from different threads -- race.  Other
 * arguments, results and errors as atp_attention_bwd. */
atp_status atp_attention_bwd_noalloc(const atp_mesh* mesh, int32_t block_mode, int64_t batch,
                                     int64_t seq, int64_t h, int32_t heads, const void* qkv,
                                     int64_t ld_qkv, const void* out, int64_t ld_out,
                                     const float* lse, const void* d_out, int64_t ld_dout,
                                     void* d_qkv, int64_t ld_dqkv, void* stream);

/* Per-kernel timing of the library's own launches.  When enabled, every
 * kernel the library enqueues is bracketed by HIP events on its stream;
 * atp_profile_collect synchronises those events, fills up to `max`
 * records (one per kernel name: launches, total milliseconds, total
 * algorithmic FLOPs and bytes) and clears the log.  Returns the number of
 * records, or -1 on a HIP error. */
typedef struct {
    char name[64];
    int64_t launches;
    double total_ms;
    double flops;
    double bytes;
} atp_kernel_stat;

/* on: 0 = off, 1 = one record per kernel, 2 = one record per kernel and
 * problem shape (names carry M x N x K and the epilogue). */
void atp_profile_enable(int32_t on);
int32_t atp_profile_collect(atp_kernel_stat* out, int32_t max);

const char* atp_status_string(int32_t status);
const char* atp_last_error(void);
const char* atp_version(void);

/* ------------------------------------------------------------------------
 * Mesh planner (host only; no GPU needed, nothing is enqueued).
 *
 * Picks the DeviceMesh(d1, d2) of least tensor-parallel communication time
 * for N devices on an interconnect described by a hierarchical
 * communication matrix (HCM, Sec. 3.4): the search space is every (d1, d2)
 * with d1 * d2 = N (Sec. 3.2), the per-axis all-reduce bandwidths come from
 * Eq. (bwd) and Eq. (allreduce) (Sec. 3.5), the time from Eq. (tcomm)
 * (Sec. 3.3).
 *
 * HCM: `n_layers` layers, outermost first (e.g. nodes, then GPUs in a
 * node).  Device r of the mesh (r = i1 * d2 + i2) has, at layer j, the rank
 * index (r / D_j) % R_j, with D_j the product of the rank counts of the
 * layers inside j.  Axis 1 all-reduces run among the devices with equal i2,
 * axis 2 among those with equal i1.
 *
 * B1' / B2' (Eq. (bwd)): at every layer an axis group spans with more than
 * one rank of one parent, each spanned rank u offers the group
 * min(group_bw, sum of p2p[u][v] over the group's other ranks v there),
 * divided by the number of that axis's groups spanning the layer through u;
 * B' is the least such value over the group's layers.  This is the paper's
 * division by d2 when a node hosts d2 groups, its P2P correction of
 * DeviceMesh(8, 2), and no division when ranks are single devices (its
 * switch and torus cases).  B = d / (2 (d - 1)) B' (Eq. (allreduce)); an
 * axis of size 1 has no all-reduce (B' = 0, B = +inf, its Eq. (tcomm) term
 * is 0).  T_comm = 2 L b s elem_bytes (7 h / (d1 B2) + 2 h / (d2 B1)) / 1e9
 * seconds for bandwidths in GB/s; +inf when a spanned rank has no
 * bandwidth to the rest of its group.
 *
 * Errors: ATP_ERR_INVALID_ARGUMENT for NULL pointers, n_layers outside
 * 1..ATP_PLAN_MAX_LAYERS, a rank count < 1, a group_bw <= 0 or not finite, a
 * negative or non-finite p2p entry, model sizes < 1, elem_bytes < 1, a
 * bandwidth given to atp_tcomm that is not > 0 (+inf is allowed), or a
 * `costs` array too small; ATP_ERR_SHAPE when d1 * d2 differs from the
 * HCM's device count; ATP_ERR_UNSUPPORTED above ATP_PLAN_MAX_DEVICES devices.
 * ------------------------------------------------------------------------ */
#define ATP_PLAN_MAX_LAYERS 16
#define ATP_PLAN_MAX_DEVICES 65536

typedef struct {
    int32_t ranks;       /* ranks of this layer under one parent, >= 1 */
    double group_bw;     /* GB/s from one rank of this layer to outside it */
    const double* p2p;   /* [ranks][ranks] row-major GB/s between ranks of one
                            parent (diagonal ignored); NULL = every pair at
                            group_bw, as behind a switch.  Host memory, read
                            during the call only. */
} atp_hcm_layer;

typedef struct {
    int64_t layers;      /* L, transformer layers */
    int64_t batch;       /* b */
    int64_t seq;         /* s */
    int64_t hidden;      /* h */
    int32_t elem_bytes;  /* bytes per all-reduced element (2 for fp16 / bf16) */
} atp_model_dims;

typedef struct {
    int32_t d1, d2;
    double b1_eff, b2_eff;  /* B1', B2' in GB/s (0 for an axis of size 1) */
    double b1, b2;          /* Eq. (allreduce) bandwidths, GB/s (+inf for size 1) */
    double t_comm;          /* Eq. (tcomm), seconds */
} atp_mesh_cost;

/* Eq. (tcomm) for given algorithm bandwidths b1, b2 (GB/s, > 0, +inf = no
 * all-reduce on that axis), e.g. calibrated from measured all-reduces
 * (Sec. 5.3).  *t_out in seconds. */
atp_status atp_tcomm(const atp_model_dims* dims, int32_t d1, int32_t d2, double b1, double b2,
                     double* t_out);

/* B1', B2', B1, B2 and T_comm of DeviceMesh(d1, d2) on the HCM. */
atp_status atp_hcm_mesh_cost(const atp_hcm_layer* hcm, int32_t n_layers,
                             const atp_model_dims* dims, int32_t d1, int32_t d2,
                             atp_mesh_cost* out);

/* Every candidate mesh of the HCM's N devices, largest d1 first: when
 * `costs` is not NULL their costs go to costs[0 .. n-1] (max_costs must be
 * >= n); *n_meshes (if not NULL) receives n; *best receives the cost of the
 * mesh of least T_comm (ties: the larger d1). */
atp_status atp_plan_mesh(const atp_hcm_layer* hcm, int32_t n_layers, const atp_model_dims* dims,
                         atp_mesh_cost* best, atp_mesh_cost* costs, int32_t max_costs,
                         int32_t* n_meshes);

#ifdef __cplusplus
}
#endif
#endif
