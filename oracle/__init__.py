"""Plain fp64 CPU oracle for the ATP chunked 2D-TP shard block.

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` may import this package.  The
product library never links, imports or calls it, and it imports nothing
from the product package: the two share no code.  Inputs reach both sides
from ``synth_inputs`` (seeded random draws, no arithmetic of the method).

Paper: Cheng, Liu, Du, You, "ATP: Adaptive Tensor Parallelism for Foundation
Models" (arXiv 2301.08658).  What is computed and where the paper says so:

* Sec. 3.1 -- device mesh, rank order, sharding spec (Shard / Replicate /
  Partial(SUM)) and the block a device holds: ``spec_block``, ``mesh_rank``.
* Sec. 3.2 -- row-first and column-first tensor parallelism for Y = XW on
  DeviceMesh(d1, d2): the specs of X, W and Y (``linear_specs``), the local
  GEMM and the grouped all-reduce of the Partial(SUM) output
  (``shard_geometry``, ``local_partial``, ``partial_reduce``).
* Sec. 3.2.1 -- the transformer layer: QKV / fc1 column-first, out-proj /
  fc2 row-first, GeLU between fc1 and fc2 (``block_fwd_*``); the "ROW" block
  swaps the two kinds (the transposed arrangement; the paper only draws the
  first).
* Sec. 4.1 -- chunking along the token rows does not change any value; the
  oracle therefore has no notion of chunks.
* Sec. 4.2 -- backward of Y = XW: dX = dY W^T, dW = X^T dY (``linear_bwd``,
  ``block_bwd``).
* Sec. 2.1 Formula (mha) and Sec. 3.2.1's attention block -- the causal
  attention core of one head (``attention_fwd`` / ``attention_bwd``) and one
  device's share of it: the heads of its reduced QKV block scattered over
  the QKV output's reduction group (``attention_core_local``,
  ``attention_core_bwd_local``); the unsharded attention block, QKV ->
  core -> out-proj, forward and backward (``attention_block_global``,
  ``attention_block_global_bwd``).

Every array crossing into C is float64; bf16 inputs are widened exactly.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

REPLICATE = -1
PARTIAL_SUM = -2
ROW_FIRST = 0
COL_FIRST = 1
BLOCK_COL = 0
BLOCK_ROW = 1
EPI_NONE, EPI_BIAS, EPI_BIAS_GELU, EPI_GELU_BWD = 0, 1, 2, 3


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so with gcc (fp64, no FMA contraction)."""
    if not force and os.path.exists(_LIB_PATH) and \
            os.path.getmtime(_LIB_PATH) >= os.path.getmtime(_SRC):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp"
    cmd = ["gcc", "-O3", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-shared", "-fPIC", "-std=c11", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or \
            os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    i32p = ctypes.POINTER(ctypes.c_int32)
    i64p = ctypes.POINTER(ctypes.c_int64)
    dp = ctypes.POINTER(ctypes.c_double)
    i64 = ctypes.c_int64
    lib.orc_mesh_rank.argtypes = [ctypes.c_int, i32p, i32p]
    lib.orc_mesh_rank.restype = i64
    lib.orc_mesh_coord.argtypes = [ctypes.c_int, i32p, i64, i32p]
    lib.orc_spec_block.argtypes = [ctypes.c_int, i32p, i32p, i32p, ctypes.c_int,
                                   i64p, i64p, i64p]
    lib.orc_spec_block.restype = ctypes.c_int
    lib.orc_linear_specs.argtypes = [ctypes.c_int, i32p, i32p, i32p]
    lib.orc_matmul.argtypes = [i64, i64, i64, dp, i64, i64, dp, i64, i64, dp, i64, i64]
    lib.orc_gelu.argtypes = [ctypes.c_double]
    lib.orc_gelu.restype = ctypes.c_double
    lib.orc_gelu_grad.argtypes = [ctypes.c_double]
    lib.orc_gelu_grad.restype = ctypes.c_double
    lib.orc_partial_reduce.argtypes = [ctypes.c_int, ctypes.POINTER(dp), i64, i64, i64,
                                       dp, ctypes.c_int, dp, dp, i64, dp]
    lib.orc_colsum.argtypes = [i64, i64, dp, i64, dp]
    lib.orc_num_threads.restype = ctypes.c_int
    lib.orc_round_bf16.argtypes = [ctypes.c_double]
    lib.orc_round_bf16.restype = ctypes.c_double
    lib.orc_attention_fwd.argtypes = [i64, i64, dp, i64, dp, i64, dp, i64, dp, i64, dp]
    lib.orc_attention_bwd.argtypes = [i64, i64, dp, i64, dp, i64, dp, i64, dp, i64,
                                      dp, i64, dp, i64, dp, i64]
    _lib = lib
    return lib


def _i32(vals):
    return (ctypes.c_int32 * len(vals))(*vals)


def _dptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _f64(a) -> np.ndarray:
    """Exact widening to float64 (torch tensors of any float dtype or numpy)."""
    if hasattr(a, "detach"):
        import torch
        a = a.detach().to("cpu", torch.float64).numpy()
    return np.asarray(a, dtype=np.float64)


def num_threads() -> int:
    return int(_load().orc_num_threads())


# --------------------------------------------------------------------------
# Sec. 3.1 -- mesh and sharding spec
# --------------------------------------------------------------------------
def mesh_rank(mesh, coord) -> int:
    return int(_load().orc_mesh_rank(len(mesh), _i32(mesh), _i32(coord)))


def mesh_coord(mesh, rank):
    out = (ctypes.c_int32 * len(mesh))()
    _load().orc_mesh_coord(len(mesh), _i32(mesh), rank, out)
    return tuple(int(v) for v in out)


def spec_block(mesh, coord, placements, shape):
    """Index ranges [(lo, hi), ...] of the block held at `coord` (Sec. 3.1)."""
    nd = len(shape)
    lo = (ctypes.c_int64 * nd)()
    hi = (ctypes.c_int64 * nd)()
    rc = _load().orc_spec_block(len(mesh), _i32(mesh), _i32(coord), _i32(placements), nd,
                                (ctypes.c_int64 * nd)(*shape), lo, hi)
    if rc != 0:
        raise ValueError("extent not divisible by the mesh")
    return [(int(lo[d]), int(hi[d])) for d in range(nd)]


def local_tensor(t: np.ndarray, mesh, coord, placements) -> np.ndarray:
    rng = spec_block(mesh, coord, placements, t.shape)
    return t[tuple(slice(a, b) for a, b in rng)]


def linear_specs(mode):
    """(x_spec, w_spec, y_spec) of Y = XW in row-first / column-first mode (Sec. 3.2)."""
    x = (ctypes.c_int32 * 2)()
    w = (ctypes.c_int32 * 2)()
    y = (ctypes.c_int32 * 2)()
    _load().orc_linear_specs(int(mode), x, w, y)
    return tuple(x), tuple(w), tuple(y)


def shard_geometry(mesh, coord, mode, K, N):
    """Local block of W and the reduction group of Y = XW, derived from the specs.

    Returns a dict with k_lo/k_hi (rows of W = columns of X), n_lo/n_hi
    (columns of W and Y), red_axis (the mesh dimension that is Partial(SUM)),
    red_size and red_index (this device's position in its group).
    """
    xs, ws, ys = linear_specs(mode)
    (k_lo, k_hi), (n_lo, n_hi) = spec_block(mesh, coord, ws, (K, N))
    red_axis = ys.index(PARTIAL_SUM)
    return dict(k_lo=k_lo, k_hi=k_hi, n_lo=n_lo, n_hi=n_hi, red_axis=red_axis,
                red_size=int(mesh[red_axis]), red_index=int(coord[red_axis]))


def reduction_group(mesh, coord, axis):
    """Coordinates of the devices that reduce together with `coord` along `axis`,
    ordered by their index along that axis (Sec. 3.3: one row or column)."""
    out = []
    for j in range(mesh[axis]):
        c = list(coord)
        c[axis] = j
        out.append(tuple(c))
    return out


# --------------------------------------------------------------------------
# arithmetic
# --------------------------------------------------------------------------
def matmul(A, B) -> np.ndarray:
    """C = A @ B in fp64, ascending-k sums (Y = XW of Sec. 3.2).  Transposed
    views are copied to row-major first (only the memory order changes)."""
    A = np.ascontiguousarray(_f64(A))
    B = np.ascontiguousarray(_f64(B))
    M, K = A.shape
    K2, N = B.shape
    assert K == K2
    C = np.empty((M, N), dtype=np.float64)
    if M and N:
        isz = 8
        _load().orc_matmul(M, K, N, _dptr(A), A.strides[0] // isz, A.strides[1] // isz,
                           _dptr(B), B.strides[0] // isz, B.strides[1] // isz,
                           _dptr(C), N, 1)
    return C


def round_bf16(x):
    """Sec. 5: inter-layer tensors are 16-bit; round fp64 values to bfloat16
    (ties to even).  Returned as fp64."""
    lib = _load()
    x = _f64(x)
    return np.vectorize(lib.orc_round_bf16, otypes=[np.float64])(x)


def gelu(x):
    lib = _load()
    x = _f64(x)
    return np.vectorize(lib.orc_gelu, otypes=[np.float64])(x)


def gelu_grad(x):
    lib = _load()
    x = _f64(x)
    return np.vectorize(lib.orc_gelu_grad, otypes=[np.float64])(x)


def partial_reduce(parts, bias=None, epi=EPI_NONE, preact_in=None):
    """Grouped reduction of Partial(SUM) blocks, summed in group order, then the
    epilogue (Sec. 3.2, Sec. 3.2.1).  Returns (out, preact) -- preact is the
    pre-activation for EPI_BIAS_GELU, else None."""
    parts = [np.ascontiguousarray(_f64(p)) for p in parts]
    T, N = parts[0].shape
    for p in parts:
        assert p.shape == (T, N)
    out = np.empty((T, N), dtype=np.float64)
    pre = np.empty((T, N), dtype=np.float64) if epi == EPI_BIAS_GELU else None
    b = np.ascontiguousarray(_f64(bias)) if bias is not None else None
    pin = np.ascontiguousarray(_f64(preact_in)) if preact_in is not None else None
    if epi in (EPI_BIAS, EPI_BIAS_GELU):
        assert b is not None and b.shape == (N,)
    if epi == EPI_GELU_BWD:
        assert pin is not None and pin.shape == (T, N)
    arr = (ctypes.POINTER(ctypes.c_double) * len(parts))(*[_dptr(p) for p in parts])
    null = ctypes.POINTER(ctypes.c_double)()
    if T and N:
        _load().orc_partial_reduce(len(parts), arr, N, T, N,
                                   _dptr(b) if b is not None else null, int(epi),
                                   _dptr(pin) if pin is not None else null,
                                   _dptr(out), N, _dptr(pre) if pre is not None else null)
    return out, pre


def colsum(dy) -> np.ndarray:
    dy = np.ascontiguousarray(_f64(dy))
    T, N = dy.shape
    db = np.zeros((N,), dtype=np.float64)
    if T and N:
        _load().orc_colsum(T, N, _dptr(dy), N, _dptr(db))
    return db


# --------------------------------------------------------------------------
# one linear on one device (Sec. 3.2) and its backward (Sec. 4.2)
# --------------------------------------------------------------------------
def local_partial(X, W, mesh, coord, mode):
    """The device's Partial(SUM) block of Y = XW, from the global X and W."""
    xs, ws, _ = linear_specs(mode)
    x_loc = local_tensor(_f64(X), mesh, coord, xs)
    w_loc = local_tensor(_f64(W), mesh, coord, ws)
    return matmul(x_loc, w_loc)


def linear_fwd_reduced(x_loc, w_loc, red_index, peers, bias=None, epi=EPI_NONE):
    """Reduced output of one shard linear: the device's own partial x_loc @ w_loc
    sits at position `red_index` of its group, `peers` fill the other positions
    (in group order); then the epilogue.  Returns (out, preact)."""
    own = matmul(x_loc, w_loc)
    parts = list(peers[:red_index]) + [own] + list(peers[red_index:])
    return partial_reduce(parts, bias, epi)


def linear_bwd(x_loc, w_loc, dy_loc):
    """Sec. 4.2: dX_part = dY W^T (still partial over the group that split N),
    dW = X^T dY (complete), db = column sums of dY."""
    x_loc = _f64(x_loc)
    w_loc = _f64(w_loc)
    dy_loc = _f64(dy_loc)
    dx = matmul(dy_loc, w_loc.T)
    dw = matmul(x_loc.T, dy_loc)
    db = colsum(dy_loc)
    return dx, dw, db


# --------------------------------------------------------------------------
# the block: QKV, out-proj, fc1 (+GeLU), fc2 on one device (Sec. 3.2.1)
# --------------------------------------------------------------------------
LINEARS = ("qkv", "out", "fc1", "fc2")


def block_linear_modes(block_mode):
    """Per-linear mode.  COL is the layer of Sec. 3.2.1 (QKV and fc1 column-first,
    out-proj and fc2 row-first); ROW swaps the two kinds."""
    if block_mode == BLOCK_COL:
        return dict(qkv=COL_FIRST, out=ROW_FIRST, fc1=COL_FIRST, fc2=ROW_FIRST)
    return dict(qkv=ROW_FIRST, out=COL_FIRST, fc1=ROW_FIRST, fc2=COL_FIRST)


def block_shapes(h):
    """Global (K, N) of each linear for hidden size h (Sec. 2.1)."""
    return dict(qkv=(h, 3 * h), out=(h, h), fc1=(h, 4 * h), fc2=(4 * h, h))


def block_fwd_local(block_mode, mesh, coord, x_loc, a_loc, w, b, peers, round_h=None):
    """Forward of one device's share of the block, from its local inputs.

    x_loc: the device's block of the layer input X (the columns its QKV and
    fc1 shards contract over); a_loc: its block of the attention-core output
    that feeds out-proj; w[name], b[name]: local weight and bias blocks;
    peers[name]: the other group members' partial blocks in group order.
    Everything is fp64: fc2 reads the exact GeLU output (the reference).
    `round_h` is a diagnostic only: a function applied to H before fc2 reads
    it (e.g. ``round_bf16``, to mimic a 16-bit stored activation, Sec. 5).
    Returns dict of qkv, o, h (GeLU output), pre (fc1 pre-activation), z.
    """
    modes = block_linear_modes(block_mode)
    out = {}

    def red_index(name):
        axis = 1 if modes[name] == COL_FIRST else 0
        return coord[axis]

    out["qkv"], _ = linear_fwd_reduced(x_loc, w["qkv"], red_index("qkv"), peers["qkv"],
                                       b["qkv"], EPI_BIAS)
    out["o"], _ = linear_fwd_reduced(a_loc, w["out"], red_index("out"), peers["out"],
                                     b["out"], EPI_BIAS)
    out["h"], out["pre"] = linear_fwd_reduced(x_loc, w["fc1"], red_index("fc1"),
                                              peers["fc1"], b["fc1"], EPI_BIAS_GELU)
    hin = out["h"] if round_h is None else round_h(out["h"])
    out["z"], _ = linear_fwd_reduced(hin, w["fc2"], red_index("fc2"), peers["fc2"],
                                     b["fc2"], EPI_BIAS)
    return out


def block_fwd_global(block_mode, mesh, coord, X, A, W, B):
    """Unsharded reference of what the device at `coord` must end up holding:
    the blocks of the full layer's outputs selected by the output specs
    (Sec. 3.2.1).  X, A: global [T, h]; W, B: global weights and biases."""
    modes = block_linear_modes(block_mode)
    X = _f64(X)
    A = _f64(A)

    def out_cols(name, Y):
        _, _, ys = linear_specs(modes[name])
        # after the grouped all-reduce the Partial dimension becomes Replicate
        spec = tuple(REPLICATE if p == PARTIAL_SUM else p for p in ys)
        return local_tensor(Y, mesh, coord, spec)

    Yq = matmul(X, W["qkv"]) + _f64(B["qkv"])[None, :]
    Yo = matmul(A, W["out"]) + _f64(B["out"])[None, :]
    pre = matmul(X, W["fc1"]) + _f64(B["fc1"])[None, :]
    H = gelu(pre)
    Z = matmul(H, W["fc2"]) + _f64(B["fc2"])[None, :]
    return dict(qkv=out_cols("qkv", Yq), o=out_cols("out", Yo), h=out_cols("fc1", H),
                pre=out_cols("fc1", pre), z=out_cols("fc2", Z))


def block_bwd_local(block_mode, mesh, coord, x_loc, a_loc, h_loc, pre_loc, w,
                    dz, dqkv, do, peers, round_dpre=None):
    """Backward of one device's share of the block (Sec. 4.2).

    dz, dqkv, do: gradients of the device's reduced output blocks z, qkv, o.
    peers[name]: the other group members' dX partials for the reduction of
    each linear's input gradient, in group order (the backward group of a
    linear is the mesh dimension that split its N).  fc2's reduced input
    gradient is multiplied by GeLU'(pre) to give fc1's dY, which fc1's
    backward reads exactly (fp64, the reference).  `round_dpre` is a
    diagnostic only: a function applied to that dY first (e.g.
    ``round_bf16``, to mimic a 16-bit stored gradient, Sec. 5).
    Returns dict with dx_qkv, da, dh_pre (fc1's dY), dx_fc1 and dw_*/db_*.
    """
    modes = block_linear_modes(block_mode)

    def bwd_index(name):
        # backward reduces over the mesh dimension that is *not* the forward's
        axis = 0 if modes[name] == COL_FIRST else 1
        return coord[axis]

    def reduced_dx(name, dx_own, epi=EPI_NONE, pre=None):
        i = bwd_index(name)
        parts = list(peers[name][:i]) + [dx_own] + list(peers[name][i:])
        return partial_reduce(parts, None, epi, pre)[0]

    res = {}
    dxo, res["dw_fc2"], res["db_fc2"] = linear_bwd(h_loc, w["fc2"], dz)
    res["dh_pre"] = reduced_dx("fc2", dxo, EPI_GELU_BWD, pre_loc)
    dpre = res["dh_pre"] if round_dpre is None else round_dpre(res["dh_pre"])
    dx1, res["dw_fc1"], res["db_fc1"] = linear_bwd(x_loc, w["fc1"], dpre)
    res["dx_fc1"] = reduced_dx("fc1", dx1)
    dxa, res["dw_out"], res["db_out"] = linear_bwd(a_loc, w["out"], do)
    res["da"] = reduced_dx("out", dxa)
    dxq, res["dw_qkv"], res["db_qkv"] = linear_bwd(x_loc, w["qkv"], dqkv)
    res["dx_qkv"] = reduced_dx("qkv", dxq)
    return res


# --------------------------------------------------------------------------
# Sec. 2.1 Formula (mha), Sec. 3.2.1 attention block
# --------------------------------------------------------------------------
def attention_fwd(q, k, v):
    """Causal attention of one head over one sequence: q, k, v [S, d].
    Returns (o [S, d], lse [S]) with lse the natural log of the softmax
    denominator of each row (scores scaled by 1/sqrt(d))."""
    q, k, v = (np.ascontiguousarray(_f64(a)) for a in (q, k, v))
    S, d = q.shape
    o = np.empty((S, d), dtype=np.float64)
    lse = np.empty((S,), dtype=np.float64)
    if S:
        _load().orc_attention_fwd(S, d, _dptr(q), d, _dptr(k), d, _dptr(v), d, _dptr(o), d,
                                  _dptr(lse))
    return o, lse


def attention_bwd(q, k, v, dout):
    """Gradients (dq, dk, dv) of the causal attention above for dO = dout."""
    q, k, v, dout = (np.ascontiguousarray(_f64(a)) for a in (q, k, v, dout))
    S, d = q.shape
    dq, dk, dv = (np.empty((S, d), dtype=np.float64) for _ in range(3))
    if S:
        _load().orc_attention_bwd(S, d, _dptr(q), d, _dptr(k), d, _dptr(v), d, _dptr(dout), d,
                                  _dptr(dq), d, _dptr(dk), d, _dptr(dv), d)
    return dq, dk, dv


def attention_heads(n_qkv_cols, head_dim, scatter_size, scatter_index):
    """The heads of a QKV block a device attends over.  The block holds
    n_qkv_cols / (3 head_dim) whole heads, each as [q | k | v] columns (the
    per-head column order of the QKV weight; the paper does not fix it).
    Sec. 3.2.1 scatters the block over the group that reduced it (it is
    replicated there), so member j of a group of g takes the j-th of g equal
    runs of heads.  Returns (first head, number of heads)."""
    per_block = n_qkv_cols // (3 * head_dim)
    assert per_block * 3 * head_dim == n_qkv_cols and per_block % scatter_size == 0
    hd = per_block // scatter_size
    return scatter_index * hd, hd


def attention_core_local(qkv_loc, batch, seq, head_dim, scatter_size, scatter_index):
    """One device's attention core: its heads of the reduced QKV block
    qkv_loc [batch*seq, 3*h_blk] (token rows sequence-major).  Returns
    (o [batch*seq, Hd*head_dim] with the device's heads in order, lse
    [Hd, batch*seq])."""
    qkv = _f64(qkv_loc)
    T = batch * seq
    h0, hd = attention_heads(qkv.shape[1], head_dim, scatter_size, scatter_index)
    o = np.zeros((T, hd * head_dim))
    lse = np.zeros((hd, T))
    for j in range(hd):
        c = 3 * head_dim * (h0 + j)
        for b in range(batch):
            r = slice(b * seq, (b + 1) * seq)
            q = qkv[r, c:c + head_dim]
            k = qkv[r, c + head_dim:c + 2 * head_dim]
            v = qkv[r, c + 2 * head_dim:c + 3 * head_dim]
            o[r, j * head_dim:(j + 1) * head_dim], lse[j, r] = attention_fwd(q, k, v)
    return o, lse


def attention_core_bwd_local(qkv_loc, dout_dev, batch, seq, head_dim, scatter_size,
                             scatter_index):
    """Gradient of attention_core_local: dout_dev [batch*seq, Hd*head_dim] ->
    d_qkv [batch*seq, Hd*3*head_dim] for the device's heads, each as
    [dq | dk | dv] (the QKV block's column order, restricted to its heads)."""
    qkv = _f64(qkv_loc)
    do = _f64(dout_dev)
    T = batch * seq
    h0, hd = attention_heads(qkv.shape[1], head_dim, scatter_size, scatter_index)
    dqkv = np.zeros((T, hd * 3 * head_dim))
    for j in range(hd):
        c = 3 * head_dim * (h0 + j)
        o3 = 3 * head_dim * j
        for b in range(batch):
            r = slice(b * seq, (b + 1) * seq)
            q = qkv[r, c:c + head_dim]
            k = qkv[r, c + head_dim:c + 2 * head_dim]
            v = qkv[r, c + 2 * head_dim:c + 3 * head_dim]
            dq, dk, dv = attention_bwd(q, k, v, do[r, j * head_dim:(j + 1) * head_dim])
            dqkv[r, o3:o3 + head_dim] = dq
            dqkv[r, o3 + head_dim:o3 + 2 * head_dim] = dk
            dqkv[r, o3 + 2 * head_dim:o3 + 3 * head_dim] = dv
    return dqkv


def attention_block_global(X, W_qkv, b_qkv, W_o, b_o, batch, seq, head_dim):
    """The unsharded attention block of one layer (Sec. 3.2.1 with Sec. 2.1
    Formula (mha) as its core), in fp64: qkv = X W_qkv + b_qkv; every head
    j (columns [3 d j, 3 d (j + 1)) of qkv, [q | k | v]) attends causally
    within each sequence; the heads' outputs side by side form A (head j at
    columns [d j, d (j + 1))); o = A W_o + b_o.  Token rows are
    sequence-major.  Returns dict(qkv, attn=A, o, lse [heads, T])."""
    X = _f64(X)
    qkv = matmul(X, W_qkv) + _f64(b_qkv)[None, :]
    T = batch * seq
    heads = qkv.shape[1] // (3 * head_dim)
    A, lse = attention_core_local(qkv, batch, seq, head_dim, 1, 0)
    assert A.shape == (T, heads * head_dim)
    o = matmul(A, W_o) + _f64(b_o)[None, :]
    return dict(qkv=qkv, attn=A, o=o, lse=lse)


def attention_block_global_bwd(X, W_qkv, W_o, fwd, d_o, batch, seq, head_dim):
    """Gradients of attention_block_global for dL/do = d_o (Sec. 4.2 through
    each product, Formula (mha)'s gradient in the core).  Returns dict with
    d_attn, d_qkv, dx, dw_qkv, db_qkv, dw_out, db_out."""
    d_o = _f64(d_o)
    W_o = _f64(W_o)
    W_qkv = _f64(W_qkv)
    d_attn, dw_out, db_out = linear_bwd(fwd["attn"], W_o, d_o)
    d_qkv = attention_core_bwd_local(fwd["qkv"], d_attn, batch, seq, head_dim, 1, 0)
    dx, dw_qkv, db_qkv = linear_bwd(X, W_qkv, d_qkv)
    return dict(d_attn=d_attn, d_qkv=d_qkv, dx=dx, dw_qkv=dw_qkv, db_qkv=db_qkv, dw_out=dw_out,
                db_out=db_out)
