"""ctypes binding of libatp.so (include/atp.h).

Argument marshalling only: every step of the path runs in the library's
HIP kernels.  Functions keep the C names; tensors are passed as torch
tensors (device pointer + leading dimension), streams as torch streams.
Sizes a C call cannot see (row counts of the buffers) are checked here so
that a short buffer never reaches a kernel.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libatp.so")

ATP_OK = 0
ATP_ERR_INVALID_ARGUMENT = 1
ATP_ERR_SHAPE = 2
ATP_ERR_UNSUPPORTED = 3
ATP_ERR_DEVICE = 4

ATP_ROW_FIRST = 0
ATP_COL_FIRST = 1
ATP_BLOCK_COL = 0
ATP_BLOCK_ROW = 1
ATP_EPI_NONE = 0
ATP_EPI_BIAS = 1
ATP_EPI_BIAS_GELU = 2
ATP_EPI_GELU_BWD = 3
ATP_F32 = 0
ATP_BF16 = 1
ATP_W_KN = 0
ATP_W_NK = 1
ATP_MAX_GROUP = 64
ATP_MAX_CHUNKS = 64

LINEARS = ("qkv", "out", "fc1", "fc2")


class AtpError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{status_string(status)}: {msg}")
        self.status = status


class atp_mesh(ctypes.Structure):
    _fields_ = [("d1", ctypes.c_int32), ("d2", ctypes.c_int32),
                ("i1", ctypes.c_int32), ("i2", ctypes.c_int32)]


class atp_shard(ctypes.Structure):
    _fields_ = [("k_loc", ctypes.c_int64), ("n_loc", ctypes.c_int64),
                ("k_off", ctypes.c_int64), ("n_off", ctypes.c_int64),
                ("red_axis", ctypes.c_int32), ("red_size", ctypes.c_int32),
                ("red_index", ctypes.c_int32), ("bwd_axis", ctypes.c_int32),
                ("bwd_size", ctypes.c_int32), ("bwd_index", ctypes.c_int32)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


_vp = ctypes.c_void_p
_fpp = ctypes.POINTER(ctypes.c_void_p)   # float* const* (host array of device ptrs)


class atp_block_weights(ctypes.Structure):
    _fields_ = [("w", _vp * 4), ("ldw", ctypes.c_int64 * 4), ("b", _vp * 4),
                ("layout", ctypes.c_int32)]


class atp_block_fwd_io(ctypes.Structure):
    _fields_ = [("x_loc", _vp), ("ldx", ctypes.c_int64),
                ("attn_loc", _vp), ("lda", ctypes.c_int64),
                ("partials", _fpp * 4), ("ldp", ctypes.c_int64 * 4),
                ("qkv", _vp), ("ld_qkv", ctypes.c_int64),
                ("o", _vp), ("ld_o", ctypes.c_int64),
                ("h", _vp), ("ld_h", ctypes.c_int64),
                ("pre", _vp),
                ("z", _vp), ("ld_z", ctypes.c_int64),
                ("partial_dtype", ctypes.c_int32)]


class atp_block_bwd_io(ctypes.Structure):
    _fields_ = [("x_loc", _vp), ("ldx", ctypes.c_int64),
                ("attn_loc", _vp), ("lda", ctypes.c_int64),
                ("h", _vp), ("ld_h", ctypes.c_int64),
                ("pre", _vp),
                ("dz", _vp), ("ld_dz", ctypes.c_int64),
                ("dqkv", _vp), ("ld_dqkv", ctypes.c_int64),
                ("d_o", _vp), ("ld_do", ctypes.c_int64),
                ("dx_partials", _fpp * 4), ("ld_dxp", ctypes.c_int64 * 4),
                ("dh_pre", _vp),
                ("dx_qkv", _vp), ("ld_dx_qkv", ctypes.c_int64),
                ("dx_fc1", _vp), ("ld_dx_fc1", ctypes.c_int64),
                ("d_attn", _vp), ("ld_d_attn", ctypes.c_int64),
                ("dw", _vp * 4), ("db", _vp * 4),
                ("partial_dtype", ctypes.c_int32)]


class atp_attn_block_fwd_io(ctypes.Structure):
    _fields_ = [("x_loc", _vp), ("ldx", ctypes.c_int64),
                ("qkv_partials", _fpp), ("ldp_qkv", ctypes.c_int64),
                ("qkv", _vp), ("ld_qkv", ctypes.c_int64),
                ("attn", _vp), ("ld_attn", ctypes.c_int64),
                ("lse", _vp),
                ("o_partials", _fpp), ("ldp_o", ctypes.c_int64),
                ("o", _vp), ("ld_o", ctypes.c_int64),
                ("partial_dtype", ctypes.c_int32)]


class atp_attn_block_bwd_io(ctypes.Structure):
    _fields_ = [("x_loc", _vp), ("ldx", ctypes.c_int64),
                ("qkv", _vp), ("ld_qkv", ctypes.c_int64),
                ("attn", _vp), ("ld_attn", ctypes.c_int64),
                ("lse", _vp),
                ("d_o", _vp), ("ld_do", ctypes.c_int64),
                ("d_attn_partials", _fpp), ("ldp_da", ctypes.c_int64),
                ("d_attn", _vp), ("ld_d_attn", ctypes.c_int64),
                ("delta", _vp),
                ("d_qkv", _vp), ("ld_dqkv", ctypes.c_int64),
                ("dx_partials", _fpp), ("ldp_dx", ctypes.c_int64),
                ("dx", _vp), ("ld_dx", ctypes.c_int64),
                ("dw", _vp * 2), ("db", _vp * 2),
                ("partial_dtype", ctypes.c_int32)]


class atp_kernel_stat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 64), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double), ("flops", ctypes.c_double),
                ("bytes", ctypes.c_double)]


class atp_hcm_layer(ctypes.Structure):
    _fields_ = [("ranks", ctypes.c_int32), ("group_bw", ctypes.c_double),
                ("p2p", ctypes.POINTER(ctypes.c_double))]


class atp_model_dims(ctypes.Structure):
    _fields_ = [("layers", ctypes.c_int64), ("batch", ctypes.c_int64), ("seq", ctypes.c_int64),
                ("hidden", ctypes.c_int64), ("elem_bytes", ctypes.c_int32)]


class atp_mesh_cost(ctypes.Structure):
    _fields_ = [("d1", ctypes.c_int32), ("d2", ctypes.c_int32),
                ("b1_eff", ctypes.c_double), ("b2_eff", ctypes.c_double),
                ("b1", ctypes.c_double), ("b2", ctypes.c_double), ("t_comm", ctypes.c_double)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


EXPORTS = (
    "atp_shard_geometry", "atp_shard_linear_fwd", "atp_chunked_partial_reduce",
    "atp_shard_linear_bwd", "atp_block_workspace_bytes", "atp_block_fwd", "atp_block_bwd",
    "atp_profile_enable", "atp_profile_collect", "atp_status_string", "atp_last_error",
    "atp_version", "atp_tcomm", "atp_hcm_mesh_cost", "atp_plan_mesh", "atp_transpose_bf16",
    "atp_attention_fwd", "atp_attention_bwd", "atp_chunked_partial_reduce_bf16",
    "atp_shard_linear_fwd_fused", "atp_block_workspace_path", "atp_block_geometry",
    "atp_attention_heads", "atp_attention_block_fwd", "atp_attention_block_bwd",
    "atp_attention_bwd_noalloc",
)
ATP_NOALLOC_DELTA_MAX = 1 << 20   # values of atp_attention_bwd_noalloc's scratch

_lib = None


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Load libatp.so.  Raises if it has not been built: there is no fallback."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build the HIP library first "
                          "(python -m paper_2301_08658_amd.build)")
    lib = ctypes.CDLL(path)
    i32, i64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    mp = ctypes.POINTER(atp_mesh)
    lib.atp_shard_geometry.argtypes = [mp, i32, i64, i64, ctypes.POINTER(atp_shard)]
    lib.atp_shard_geometry.restype = i32
    lib.atp_shard_linear_fwd.argtypes = [mp, i32, i64, i64, i64, i32, _vp, i64, _vp, i64, _vp,
                                         i32, _vp, i32, i64, _vp, _vp, _fpp]
    lib.atp_shard_linear_fwd.restype = i32
    lib.atp_chunked_partial_reduce.argtypes = [i32, i64, i64, i32, _fpp, i64, _vp, i32, _vp, _vp,
                                               i32, i64, _vp, _vp, _fpp]
    lib.atp_chunked_partial_reduce.restype = i32
    lib.atp_chunked_partial_reduce_bf16.argtypes = lib.atp_chunked_partial_reduce.argtypes
    lib.atp_chunked_partial_reduce_bf16.restype = i32
    lib.atp_shard_linear_fwd_fused.argtypes = [mp, i32, i64, i64, i64, _vp, i64, _vp, i64, _fpp,
                                               i64, _vp, i32, _vp, i32, i64, _vp, _vp]
    lib.atp_shard_linear_fwd_fused.restype = i32
    lib.atp_shard_linear_bwd.argtypes = [mp, i32, i64, i64, i64, i32, _vp, i64, _vp, i64, _vp, i64,
                                         _vp, i64, _vp, i64, _vp, _vp, _fpp]
    lib.atp_shard_linear_bwd.restype = i32
    lib.atp_block_workspace_bytes.argtypes = [mp, i32, i64, i64, i32, i32]
    lib.atp_block_workspace_bytes.restype = sz
    lib.atp_block_workspace_path.argtypes = [mp, i32, i64, i64, i32, sz, i32]
    lib.atp_block_workspace_path.restype = i32
    lib.atp_block_geometry.argtypes = [mp, i32, i64, ctypes.POINTER(atp_shard)]
    lib.atp_block_geometry.restype = i32
    i32p = ctypes.POINTER(i32)
    lib.atp_attention_heads.argtypes = [mp, i32, i64, i32, i32p, i32p, i32p]
    lib.atp_attention_heads.restype = i32
    lib.atp_attention_block_fwd.argtypes = [mp, i32, i64, i64, i64, i32, i32,
                                            ctypes.POINTER(atp_block_weights),
                                            ctypes.POINTER(atp_attn_block_fwd_io), _vp,
                                            ctypes.c_size_t, _vp, _vp]
    lib.atp_attention_block_fwd.restype = i32
    lib.atp_attention_block_bwd.argtypes = [mp, i32, i64, i64, i64, i32, i32,
                                            ctypes.POINTER(atp_block_weights),
                                            ctypes.POINTER(atp_attn_block_bwd_io), _vp,
                                            ctypes.c_size_t, _vp, _vp]
    lib.atp_attention_block_bwd.restype = i32
    lib.atp_block_fwd.argtypes = [mp, i32, i64, i64, i32, ctypes.POINTER(atp_block_weights),
                                  ctypes.POINTER(atp_block_fwd_io), _vp, sz, _vp, _vp]
    lib.atp_block_fwd.restype = i32
    lib.atp_block_bwd.argtypes = [mp, i32, i64, i64, i32, ctypes.POINTER(atp_block_weights),
                                  ctypes.POINTER(atp_block_bwd_io), _vp, sz, _vp, _vp]
    lib.atp_block_bwd.restype = i32
    lib.atp_profile_enable.argtypes = [i32]
    lib.atp_profile_enable.restype = None
    lib.atp_profile_collect.argtypes = [ctypes.POINTER(atp_kernel_stat), i32]
    lib.atp_profile_collect.restype = i32
    lib.atp_status_string.argtypes = [i32]
    lib.atp_status_string.restype = ctypes.c_char_p
    lib.atp_last_error.argtypes = []
    lib.atp_last_error.restype = ctypes.c_char_p
    lib.atp_version.argtypes = []
    lib.atp_version.restype = ctypes.c_char_p
    lib.atp_transpose_bf16.argtypes = [i64, i64, _vp, i64, _vp, i64, _vp]
    lib.atp_transpose_bf16.restype = i32
    lib.atp_attention_fwd.argtypes = [mp, i32, i64, i64, i64, i32, _vp, i64, _vp, i64, _vp, _vp]
    lib.atp_attention_fwd.restype = i32
    lib.atp_attention_bwd.argtypes = [mp, i32, i64, i64, i64, i32, _vp, i64, _vp, i64, _vp, _vp,
                                      i64, _vp, i64, _vp, _vp]
    lib.atp_attention_bwd.restype = i32
    lib.atp_attention_bwd_noalloc.argtypes = [mp, i32, i64, i64, i64, i32, _vp, i64, _vp, i64,
                                              _vp, _vp, i64, _vp, i64, _vp]
    lib.atp_attention_bwd_noalloc.restype = i32
    hp, dp, cp = (ctypes.POINTER(atp_hcm_layer), ctypes.POINTER(atp_model_dims),
                  ctypes.POINTER(atp_mesh_cost))
    lib.atp_tcomm.argtypes = [dp, i32, i32, ctypes.c_double, ctypes.c_double,
                              ctypes.POINTER(ctypes.c_double)]
    lib.atp_tcomm.restype = i32
    lib.atp_hcm_mesh_cost.argtypes = [hp, i32, dp, i32, i32, cp]
    lib.atp_hcm_mesh_cost.restype = i32
    lib.atp_plan_mesh.argtypes = [hp, i32, dp, cp, cp, i32, ctypes.POINTER(i32)]
    lib.atp_plan_mesh.restype = i32
    _lib = lib
    return lib


def status_string(s: int) -> str:
    return load_library().atp_status_string(int(s)).decode()


def last_error() -> str:
    return load_library().atp_last_error().decode()


def _check(status: int):
    if status != ATP_OK:
        raise AtpError(status, last_error())


# ---------------------------------------------------------------- marshalling
def mesh(d1, d2, i1=0, i2=0) -> atp_mesh:
    return atp_mesh(int(d1), int(d2), int(i1), int(i2))


def _on_device(t: torch.Tensor, name: str):
    """The library reads and writes device memory of the current HIP device."""
    if not t.is_cuda:
        raise ValueError(f"{name}: must be a tensor on the GPU, got one on {t.device}")
    if t.device.index != torch.cuda.current_device():
        raise ValueError(f"{name}: on {t.device}, but the current device is "
                         f"cuda:{torch.cuda.current_device()}")


def _ptr(t: Optional[torch.Tensor], name: str = "tensor") -> Optional[int]:
    if t is None:
        return None
    _on_device(t, name)
    return t.data_ptr()


def _mat(t: Optional[torch.Tensor], rows: int, cols: int, dtype, name: str):
    """(pointer, ld) of a row-major device matrix with at least rows x cols."""
    if t is None:
        return None, 0
    _on_device(t, name)
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if t.dim() != 2 or (t.size(1) > 1 and t.stride(1) != 1):
        raise ValueError(f"{name}: needs a 2-D row-major tensor")
    if t.size(0) < rows or t.size(1) < cols:
        raise ValueError(f"{name}: {tuple(t.shape)} smaller than [{rows}, {cols}]")
    return t.data_ptr(), (t.stride(0) if t.size(0) > 1 else max(t.size(1), cols))


def _vec(t: Optional[torch.Tensor], n: int, dtype, name: str):
    if t is None:
        return None
    _on_device(t, name)
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if t.numel() < n or not t.is_contiguous():
        raise ValueError(f"{name}: needs {n} contiguous elements")
    return t.data_ptr()


def _stream(s) -> Optional[int]:
    if s is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _opt_stream(s) -> Optional[int]:
    """A stream that may be absent (NULL)."""
    return None if s is None else _stream(s)


def _events(evs: Optional[Sequence]) -> Optional[ctypes.Array]:
    if evs is None:
        return None
    return (ctypes.c_void_p * len(evs))(*[e.handle if isinstance(e, HipEvent) else e
                                          for e in evs])


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return ATP_F32
    if t.dtype == torch.bfloat16:
        return ATP_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr_table(ts: Sequence[Optional[torch.Tensor]], rows: int, cols: int, name: str,
               dtype=torch.float32):
    """Host array of device pointers (None entries stay NULL) and their common ld."""
    arr = (ctypes.c_void_p * len(ts))()
    ld = None
    for j, t in enumerate(ts):
        if t is None:
            continue
        p, l = _mat(t, rows, cols, dtype, f"{name}[{j}]")
        arr[j] = p
        if ld is None:
            ld = l
        elif l != ld:
            raise ValueError(f"{name}: all buffers need the same leading dimension")
    return ctypes.cast(arr, _fpp), arr, (ld or cols)


class HipEvent:
    """A raw hipEvent_t (created through the HIP runtime) for chunk signalling."""
    _hip = None

    def __init__(self, timing: bool = False):
        if HipEvent._hip is None:
            HipEvent._hip = ctypes.CDLL("libamdhip64.so")
        h = ctypes.c_void_p()
        flags = 0 if timing else 0x2   # hipEventDisableTiming
        rc = HipEvent._hip.hipEventCreateWithFlags(ctypes.byref(h), ctypes.c_uint(flags))
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")
        self.handle = h.value

    def synchronize(self):
        rc = HipEvent._hip.hipEventSynchronize(ctypes.c_void_p(self.handle))
        if rc != 0:
            raise RuntimeError(f"hipEventSynchronize failed ({rc})")

    def __del__(self):
        if HipEvent._hip is not None and getattr(self, "handle", None):
            HipEvent._hip.hipEventDestroy(ctypes.c_void_p(self.handle))


# ---------------------------------------------------------------- the ABI
def atp_version() -> str:
    return load_library().atp_version().decode()


def atp_shard_geometry(m: atp_mesh, mode: int, k: int, n: int) -> atp_shard:
    out = atp_shard()
    _check(load_library().atp_shard_geometry(ctypes.byref(m), int(mode), int(k), int(n),
                                             ctypes.byref(out)))
    return out


def atp_shard_linear_fwd(m: atp_mesh, mode: int, tokens: int, k: int, n: int, chunks: int,
                         x_loc, w_loc, bias_loc, epi: int, y, preact=None, stream=None,
                         chunk_done=None):
    g = atp_shard_geometry(m, mode, k, n)
    xp, ldx = _mat(x_loc, tokens, g.k_loc, torch.bfloat16, "x_loc")
    wp, ldw = _mat(w_loc, g.k_loc, g.n_loc, torch.bfloat16, "w_loc")
    yp, ldy = _mat(y, tokens, g.n_loc, y.dtype, "y")
    pp, ldp = _mat(preact, tokens, g.n_loc, torch.bfloat16, "preact")
    if preact is not None and ldp != ldy:
        raise ValueError("preact must share y's leading dimension")
    bp = _vec(bias_loc, g.n_loc, torch.bfloat16, "bias_loc")
    _check(load_library().atp_shard_linear_fwd(
        ctypes.byref(m), int(mode), int(tokens), int(k), int(n), int(chunks), xp, ldx, wp, ldw,
        bp, int(epi), yp, _dtype_code(y), ldy, pp, _stream(stream), _events(chunk_done)))


def atp_chunked_partial_reduce(red_size: int, tokens: int, n_loc: int, chunks: int, partials,
                               bias_loc, epi: int, out, preact_in=None, preact_out=None,
                               stream=None, chunk_ready=None):
    if len(partials) != red_size:
        raise ValueError("need exactly red_size partial buffers")
    tab, _keep, ldp = _ptr_table(partials, tokens, n_loc, "partials")
    op, ldo = _mat(out, tokens, n_loc, out.dtype, "out")
    ip, ldi = _mat(preact_in, tokens, n_loc, torch.bfloat16, "preact_in")
    qp, ldq = _mat(preact_out, tokens, n_loc, torch.bfloat16, "preact_out")
    for t, l in ((preact_in, ldi), (preact_out, ldq)):
        if t is not None and l != ldo:
            raise ValueError("pre-activation buffers must share out's leading dimension")
    bp = _vec(bias_loc, n_loc, torch.bfloat16, "bias_loc")
    _check(load_library().atp_chunked_partial_reduce(
        int(red_size), int(tokens), int(n_loc), int(chunks), tab, ldp, bp, int(epi), ip, op,
        _dtype_code(out), ldo, qp, _stream(stream), _events(chunk_ready)))


def atp_chunked_partial_reduce_bf16(red_size: int, tokens: int, n_loc: int, chunks: int,
                                    partials, bias_loc, epi: int, out, preact_in=None,
                                    preact_out=None, stream=None, chunk_ready=None):
    if len(partials) != red_size:
        raise ValueError("need exactly red_size partial buffers")
    tab, _keep, ldp = _ptr_table(partials, tokens, n_loc, "partials", torch.bfloat16)
    op, ldo = _mat(out, tokens, n_loc, out.dtype, "out")
    ip, ldi = _mat(preact_in, tokens, n_loc, torch.bfloat16, "preact_in")
    qp, ldq = _mat(preact_out, tokens, n_loc, torch.bfloat16, "preact_out")
    for t, l in ((preact_in, ldi), (preact_out, ldq)):
        if t is not None and l != ldo:
            raise ValueError("pre-activation buffers must share out's leading dimension")
    bp = _vec(bias_loc, n_loc, torch.bfloat16, "bias_loc")
    _check(load_library().atp_chunked_partial_reduce_bf16(
        int(red_size), int(tokens), int(n_loc), int(chunks), tab, ldp, bp, int(epi), ip, op,
        _dtype_code(out), ldo, qp, _stream(stream), _events(chunk_ready)))


def atp_shard_linear_fwd_fused(m: atp_mesh, mode: int, tokens: int, k: int, n: int, x_loc,
                               w_loc, peers, bias_loc, epi: int, out, preact=None, stream=None):
    """peers: red_size entries, the other members' f32 partials (the own
    entry may be None; it is not read)."""
    g = atp_shard_geometry(m, mode, k, n)
    if len(peers) != g.red_size:
        raise ValueError("need exactly red_size peer entries")
    xp, ldx = _mat(x_loc, tokens, g.k_loc, torch.bfloat16, "x_loc")
    wp, ldw = _mat(w_loc, g.k_loc, g.n_loc, torch.bfloat16, "w_loc")
    tab, _keep, ldp = _ptr_table(peers, tokens, g.n_loc, "peers")
    op, ldo = _mat(out, tokens, g.n_loc, out.dtype, "out")
    pp, ldq = _mat(preact, tokens, g.n_loc, torch.bfloat16, "preact")
    if preact is not None and ldq != ldo:
        raise ValueError("preact must share out's leading dimension")
    bp = _vec(bias_loc, g.n_loc, torch.bfloat16, "bias_loc")
    _check(load_library().atp_shard_linear_fwd_fused(
        ctypes.byref(m), int(mode), int(tokens), int(k), int(n), xp, ldx, wp, ldw,
        tab if g.red_size > 1 else None, ldp, bp, int(epi), op, _dtype_code(out), ldo, pp,
        _stream(stream)))


def atp_shard_linear_bwd(m: atp_mesh, mode: int, tokens: int, k: int, n: int, chunks: int,
                         x_loc, w_loc, dy, dx_partial, dw, db=None, stream=None,
                         dx_chunk_done=None):
    g = atp_shard_geometry(m, mode, k, n)
    xp, ldx = _mat(x_loc, tokens, g.k_loc, torch.bfloat16, "x_loc")
    wp, ldw = _mat(w_loc, g.k_loc, g.n_loc, torch.bfloat16, "w_loc")
    yp, ldy = _mat(dy, tokens, g.n_loc, torch.bfloat16, "dy")
    dxp, lddx = _mat(dx_partial, tokens, g.k_loc, torch.float32, "dx_partial")
    dwp, lddw = _mat(dw, g.k_loc, g.n_loc, torch.float32, "dw")
    dbp = _vec(db, g.n_loc, torch.float32, "db")
    _check(load_library().atp_shard_linear_bwd(
        ctypes.byref(m), int(mode), int(tokens), int(k), int(n), int(chunks), xp, ldx, wp, ldw,
        yp, ldy, dxp, lddx, dwp, lddw, dbp, _stream(stream), _events(dx_chunk_done)))


def block_geometry(m: atp_mesh, block_mode: int, h: int):
    """Shard geometry of the block's four linears (qkv, out, fc1, fc2)."""
    out = (atp_shard * 4)()
    _check(load_library().atp_block_geometry(ctypes.byref(m), int(block_mode), int(h), out))
    return [out[i] for i in range(4)]


def atp_block_workspace_bytes(m: atp_mesh, block_mode: int, tokens: int, h: int,
                              chunks: int, weight_layout: int = ATP_W_KN) -> int:
    return int(load_library().atp_block_workspace_bytes(ctypes.byref(m), int(block_mode),
                                                         int(tokens), int(h), int(chunks),
                                                         int(weight_layout)))


def atp_block_workspace_path(m: atp_mesh, block_mode: int, tokens: int, h: int,
                             weight_layout: int, ws_bytes: int, pass_: int) -> int:
    """1: a block call of the pass (0 fwd, 1 bwd) with ws_bytes of workspace
    takes the transposed-layout path; 0: the direct path; -1: invalid."""
    return int(load_library().atp_block_workspace_path(ctypes.byref(m), int(block_mode),
                                                        int(tokens), int(h), int(weight_layout),
                                                        int(ws_bytes), int(pass_)))


def _weights(G, w: Sequence[torch.Tensor], b: Sequence[torch.Tensor], layout: int):
    """Weights [k_loc, n_loc] (ATP_W_KN) or [n_loc, k_loc] (ATP_W_NK)."""
    W = atp_block_weights()
    W.layout = int(layout)
    for i, g in enumerate(G):
        r, c = (g.k_loc, g.n_loc) if layout == ATP_W_KN else (g.n_loc, g.k_loc)
        p, ld = _mat(w[i], r, c, torch.bfloat16, f"w[{LINEARS[i]}]")
        W.w[i] = p
        W.ldw[i] = ld
        W.b[i] = _vec(b[i], g.n_loc, torch.bfloat16, f"b[{LINEARS[i]}]")
    return W


def _partial_dtype(tables) -> tuple:
    """(ATP dtype code, torch dtype) shared by every partial buffer given."""
    dts = {t.dtype for tab in tables if tab for t in tab if t is not None}
    if len(dts) > 1:
        raise TypeError(f"partial buffers mix dtypes {sorted(map(str, dts))}")
    dt = dts.pop() if dts else torch.float32
    if dt not in (torch.float32, torch.bfloat16):
        raise TypeError(f"partial buffers must be float32 or bfloat16, not {dt}")
    return (ATP_F32 if dt == torch.float32 else ATP_BF16), dt


def _workspace(workspace):
    if workspace is None:
        return None, 0
    _on_device(workspace, "workspace")
    return workspace.data_ptr(), workspace.numel() * workspace.element_size()


def atp_block_fwd(m: atp_mesh, block_mode: int, tokens: int, h: int, chunks: int, w, b,
                  x_loc, attn_loc, partials, qkv, o, h_out, pre, z, workspace=None,
                  compute_stream=None, comm_stream=None, weight_layout: int = ATP_W_KN):
    """partials[i]: list of the red_size buffers of linear i's group (own
    entry written; all float32, or all bfloat16 for 16-bit partials), or
    None for a group of one."""
    G = block_geometry(m, block_mode, h)
    W = _weights(G, w, b, weight_layout)
    io = atp_block_fwd_io()
    io.partial_dtype, pdt = _partial_dtype(partials)
    io.x_loc, io.ldx = _mat(x_loc, tokens, G[0].k_loc, torch.bfloat16, "x_loc")
    io.attn_loc, io.lda = _mat(attn_loc, tokens, G[1].k_loc, torch.bfloat16, "attn_loc")
    keep = []
    for i, g in enumerate(G):
        if g.red_size > 1:
            if len(partials[i]) != g.red_size:
                raise ValueError(f"partials[{LINEARS[i]}] needs {g.red_size} buffers")
            tab, arr, ld = _ptr_table(partials[i], tokens, g.n_loc, f"partials[{LINEARS[i]}]",
                                      pdt)
            io.partials[i] = tab
            io.ldp[i] = ld
            keep.append(arr)
    io.qkv, io.ld_qkv = _mat(qkv, tokens, G[0].n_loc, torch.bfloat16, "qkv")
    io.o, io.ld_o = _mat(o, tokens, G[1].n_loc, torch.bfloat16, "o")
    io.h, io.ld_h = _mat(h_out, tokens, G[2].n_loc, torch.bfloat16, "h")
    pp, ldpre = _mat(pre, tokens, G[2].n_loc, torch.bfloat16, "pre")
    if ldpre != io.ld_h:
        raise ValueError("pre must share h's leading dimension")
    io.pre = pp
    io.z, io.ld_z = _mat(z, tokens, G[3].n_loc, torch.bfloat16, "z")
    wsp, wsb = _workspace(workspace)
    _check(load_library().atp_block_fwd(ctypes.byref(m), int(block_mode), int(tokens), int(h),
                                        int(chunks), ctypes.byref(W), ctypes.byref(io), wsp, wsb,
                                        _stream(compute_stream), _stream(comm_stream)))


def atp_block_bwd(m: atp_mesh, block_mode: int, tokens: int, h: int, chunks: int, w, b,
                  x_loc, attn_loc, h_act, pre, dz, dqkv, d_o, dx_partials, dh_pre, dx_qkv,
                  dx_fc1, d_attn, dw, db, workspace=None, compute_stream=None,
                  comm_stream=None, weight_layout: int = ATP_W_KN):
    """dx_partials[i]: list of the bwd_size buffers of linear i's backward
    group (own entry written; float32 or bfloat16), or None for a group of
    one.  dw[i] has the weight's layout and leading dimension."""
    G = block_geometry(m, block_mode, h)
    W = _weights(G, w, b, weight_layout)
    io = atp_block_bwd_io()
    io.partial_dtype, pdt = _partial_dtype(dx_partials)
    io.x_loc, io.ldx = _mat(x_loc, tokens, G[0].k_loc, torch.bfloat16, "x_loc")
    io.attn_loc, io.lda = _mat(attn_loc, tokens, G[1].k_loc, torch.bfloat16, "attn_loc")
    io.h, io.ld_h = _mat(h_act, tokens, G[2].n_loc, torch.bfloat16, "h")
    pp, ldpre = _mat(pre, tokens, G[2].n_loc, torch.bfloat16, "pre")
    dp, lddp = _mat(dh_pre, tokens, G[2].n_loc, torch.bfloat16, "dh_pre")
    if ldpre != io.ld_h or lddp != io.ld_h:
        raise ValueError("pre and dh_pre must share h's leading dimension")
    io.pre, io.dh_pre = pp, dp
    io.dz, io.ld_dz = _mat(dz, tokens, G[3].n_loc, torch.bfloat16, "dz")
    io.dqkv, io.ld_dqkv = _mat(dqkv, tokens, G[0].n_loc, torch.bfloat16, "dqkv")
    io.d_o, io.ld_do = _mat(d_o, tokens, G[1].n_loc, torch.bfloat16, "d_o")
    keep = []
    for i, g in enumerate(G):
        if g.bwd_size > 1:
            if len(dx_partials[i]) != g.bwd_size:
                raise ValueError(f"dx_partials[{LINEARS[i]}] needs {g.bwd_size} buffers")
            tab, arr, ld = _ptr_table(dx_partials[i], tokens, g.k_loc,
                                      f"dx_partials[{LINEARS[i]}]", pdt)
            io.dx_partials[i] = tab
            io.ld_dxp[i] = ld
            keep.append(arr)
    io.dx_qkv, io.ld_dx_qkv = _mat(dx_qkv, tokens, G[0].k_loc, torch.bfloat16, "dx_qkv")
    io.dx_fc1, io.ld_dx_fc1 = _mat(dx_fc1, tokens, G[2].k_loc, torch.bfloat16, "dx_fc1")
    io.d_attn, io.ld_d_attn = _mat(d_attn, tokens, G[1].k_loc, torch.bfloat16, "d_attn")
    for i, g in enumerate(G):
        r, c = (g.k_loc, g.n_loc) if weight_layout == ATP_W_KN else (g.n_loc, g.k_loc)
        p, ld = _mat(dw[i], r, c, torch.float32, f"dw[{LINEARS[i]}]")
        if ld != W.ldw[i]:
            raise ValueError(f"dw[{LINEARS[i]}] must share the weight's leading dimension")
        io.dw[i] = p
        io.db[i] = _vec(db[i], g.n_loc, torch.float32, f"db[{LINEARS[i]}]") if db else None
    wsp, wsb = _workspace(workspace)
    _check(load_library().atp_block_bwd(ctypes.byref(m), int(block_mode), int(tokens), int(h),
                                        int(chunks), ctypes.byref(W), ctypes.byref(io), wsp, wsb,
                                        _stream(compute_stream), _stream(comm_stream)))


def atp_profile_enable(on=True):
    """on: False/0 off, True/1 per kernel, 2 per kernel and problem shape."""
    load_library().atp_profile_enable(int(on) if not isinstance(on, bool) else (1 if on else 0))


def atp_profile_collect(max_records: int = 32):
    arr = (atp_kernel_stat * max_records)()
    n = load_library().atp_profile_collect(arr, max_records)
    if n < 0:
        raise AtpError(ATP_ERR_DEVICE, last_error())
    return [dict(name=arr[i].name.decode(), launches=arr[i].launches,
                 total_ms=arr[i].total_ms, flops=arr[i].flops, bytes=arr[i].bytes)
            for i in range(n)]


def atp_transpose_bf16(src, dst, stream=None):
    """dst[c, r] = src[r, c]; src [rows, cols] and dst [cols, rows] bf16 views."""
    rows, cols = src.shape
    sp, lds = _mat(src, rows, cols, torch.bfloat16, "src")
    dp_, ldd = _mat(dst, cols, rows, torch.bfloat16, "dst")
    _check(load_library().atp_transpose_bf16(int(rows), int(cols), sp, lds, dp_, ldd,
                                             _stream(stream)))


def attention_heads(m: atp_mesh, block_mode: int, h: int, heads: int):
    """(first head, number of heads) of the device's run of its QKV block's
    heads (block-local indices), and the block's head count."""
    first, count, per_block = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    _check(load_library().atp_attention_heads(ctypes.byref(m), int(block_mode), int(h),
                                              int(heads), ctypes.byref(first),
                                              ctypes.byref(count), ctypes.byref(per_block)))
    return first.value, count.value, per_block.value


def _f32_scratch(t, n: int, name: str):
    """A contiguous float32 buffer of at least n values (checked before any
    other argument, so a short buffer never reaches a kernel)."""
    if t is None:
        return
    if t.dtype != torch.float32 or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous float32 tensor")
    if t.numel() < n:
        raise ValueError(f"{name}: {t.numel()} values, the device's heads need {n}")


def atp_attention_fwd(m: atp_mesh, block_mode: int, batch: int, seq: int, h: int, heads: int,
                      qkv, out, lse, stream=None):
    """The device's attention core: qkv [batch*seq, n_loc] bf16 (its reduced
    QKV block), out [batch*seq, >= n_loc/3] bf16 (the gathered out-proj
    input; the device's columns are written), lse [heads_dev, batch*seq] fp32."""
    T = batch * seq
    _, hd, _ = attention_heads(m, block_mode, h, heads)
    _f32_scratch(lse, hd * T, "lse")
    g = block_geometry(m, block_mode, h)[0]
    qp, ldq = _mat(qkv, T, g.n_loc, torch.bfloat16, "qkv")
    op, ldo = _mat(out, T, g.n_loc // 3, torch.bfloat16, "out")
    _check(load_library().atp_attention_fwd(ctypes.byref(m), int(block_mode), int(batch), int(seq),
                                            int(h), int(heads), qp, ldq, op, ldo,
                                            _ptr(lse, "lse"), _stream(stream)))


def atp_attention_bwd(m: atp_mesh, block_mode: int, batch: int, seq: int, h: int, heads: int,
                      qkv, out, lse, d_out, d_qkv, delta, stream=None):
    """Gradient of atp_attention_fwd: d_qkv (the QKV block's shape) receives
    dq, dk, dv of the device's heads; delta is fp32 scratch [heads_dev*T]."""
    T = batch * seq
    _, hd, _ = attention_heads(m, block_mode, h, heads)
    _f32_scratch(lse, hd * T, "lse")
    _f32_scratch(delta, hd * T, "delta")
    g = block_geometry(m, block_mode, h)[0]
    qp, ldq = _mat(qkv, T, g.n_loc, torch.bfloat16, "qkv")
    op, ldo = _mat(out, T, g.n_loc // 3, torch.bfloat16, "out")
    dop, lddo = _mat(d_out, T, g.n_loc // 3, torch.bfloat16, "d_out")
    dqp, lddq = _mat(d_qkv, T, g.n_loc, torch.bfloat16, "d_qkv")
    _check(load_library().atp_attention_bwd(ctypes.byref(m), int(block_mode), int(batch), int(seq),
                                            int(h), int(heads), qp, ldq, op, ldo,
                                            _ptr(lse, "lse"), dop, lddo, dqp, lddq,
                                            _ptr(delta, "delta"), _stream(stream)))


def atp_attention_bwd_noalloc(m: atp_mesh, block_mode: int, batch: int, seq: int, h: int,
                              heads: int, qkv, out, lse, d_out, d_qkv, stream=None):
    """atp_attention_bwd without caller scratch: delta lives in the library's
    own per-GPU array (for callers that cannot allocate)."""
    T = batch * seq
    _, hd, _ = attention_heads(m, block_mode, h, heads)
    _f32_scratch(lse, hd * T, "lse")
    g = block_geometry(m, block_mode, h)[0]
    qp, ldq = _mat(qkv, T, g.n_loc, torch.bfloat16, "qkv")
    op, ldo = _mat(out, T, g.n_loc // 3, torch.bfloat16, "out")
    dop, lddo = _mat(d_out, T, g.n_loc // 3, torch.bfloat16, "d_out")
    dqp, lddq = _mat(d_qkv, T, g.n_loc, torch.bfloat16, "d_qkv")
    _check(load_library().atp_attention_bwd_noalloc(
        ctypes.byref(m), int(block_mode), int(batch), int(seq), int(h), int(heads), qp, ldq, op,
        ldo, _ptr(lse, "lse"), dop, lddo, dqp, lddq, _stream(stream)))


def _attn_weights(G, w, b, layout: int):
    """Weights of QKV and out-proj (entries 0 and 1) for the attention block."""
    W = atp_block_weights()
    W.layout = int(layout)
    for i in range(2):
        g = G[i]
        r, c = (g.k_loc, g.n_loc) if layout == ATP_W_KN else (g.n_loc, g.k_loc)
        W.w[i], W.ldw[i] = _mat(w[i], r, c, torch.bfloat16, f"w[{LINEARS[i]}]")
        W.b[i] = _vec(b[i], g.n_loc, torch.bfloat16, f"b[{LINEARS[i]}]")
    return W


def atp_attention_block_fwd(m: atp_mesh, block_mode: int, batch: int, seq: int, h: int,
                            heads: int, chunks: int, w, b, x_loc, qkv_partials, qkv, attn, lse,
                            o_partials, o, workspace=None, compute_stream=None, comm_stream=None,
                            weight_layout: int = ATP_W_KN):
    """The device's attention block: QKV -> its heads' attention -> out-proj.
    w, b: [qkv, out] weights and biases; qkv_partials / o_partials: the
    groups' buffers (own entry written) or None for a group of one; attn: the
    gathered out-proj input, whose other members' columns must be filled;
    workspace: an optional uint8 device buffer (atp_block_workspace_bytes
    covers it)."""
    T = batch * seq
    G = block_geometry(m, block_mode, h)
    _, hd, _ = attention_heads(m, block_mode, h, heads)
    _f32_scratch(lse, hd * T, "lse")
    W = _attn_weights(G, w, b, weight_layout)
    io = atp_attn_block_fwd_io()
    io.partial_dtype, pdt = _partial_dtype([qkv_partials, o_partials])
    io.x_loc, io.ldx = _mat(x_loc, T, G[0].k_loc, torch.bfloat16, "x_loc")
    keep = []
    for name, parts, g, attr in (("qkv_partials", qkv_partials, G[0], "qkv"),
                                 ("o_partials", o_partials, G[1], "o")):
        if g.red_size > 1:
            if len(parts) != g.red_size:
                raise ValueError(f"{name} needs {g.red_size} buffers")
            tab, arr, ld = _ptr_table(parts, T, g.n_loc, name, pdt)
            setattr(io, name, tab)
            setattr(io, "ldp_" + attr, ld)
            keep.append(arr)
    io.qkv, io.ld_qkv = _mat(qkv, T, G[0].n_loc, torch.bfloat16, "qkv")
    io.attn, io.ld_attn = _mat(attn, T, G[1].k_loc, torch.bfloat16, "attn")
    io.lse = _ptr(lse, "lse")
    io.o, io.ld_o = _mat(o, T, G[1].n_loc, torch.bfloat16, "o")
    wsp, wsb = _workspace(workspace)
    _check(load_library().atp_attention_block_fwd(
        ctypes.byref(m), int(block_mode), int(batch), int(seq), int(h), int(heads), int(chunks),
        ctypes.byref(W), ctypes.byref(io), wsp, wsb, _stream(compute_stream),
        _stream(comm_stream)))


def atp_attention_block_bwd(m: atp_mesh, block_mode: int, batch: int, seq: int, h: int,
                            heads: int, chunks: int, w, b, x_loc, qkv, attn, lse, d_o,
                            d_attn_partials, d_attn, delta, d_qkv, dx_partials, dx, dw, db,
                            workspace=None, compute_stream=None, comm_stream=None,
                            weight_layout: int = ATP_W_KN):
    """Backward of atp_attention_block_fwd.  d_qkv: the QKV block's
    gradient, whose other members' columns must be filled; dw, db: [qkv, out]
    (dw in the weights' layout, db entries may be None); workspace: an
    optional uint8 device buffer (atp_block_workspace_bytes covers it)."""
    T = batch * seq
    G = block_geometry(m, block_mode, h)
    _, hd, _ = attention_heads(m, block_mode, h, heads)
    _f32_scratch(lse, hd * T, "lse")
    _f32_scratch(delta, hd * T, "delta")
    W = _attn_weights(G, w, b, weight_layout)
    io = atp_attn_block_bwd_io()
    io.partial_dtype, pdt = _partial_dtype([d_attn_partials, dx_partials])
    io.x_loc, io.ldx = _mat(x_loc, T, G[0].k_loc, torch.bfloat16, "x_loc")
    io.qkv, io.ld_qkv = _mat(qkv, T, G[0].n_loc, torch.bfloat16, "qkv")
    io.attn, io.ld_attn = _mat(attn, T, G[1].k_loc, torch.bfloat16, "attn")
    io.lse = _ptr(lse, "lse")
    io.d_o, io.ld_do = _mat(d_o, T, G[1].n_loc, torch.bfloat16, "d_o")
    keep = []
    for name, parts, g, ldname in (("d_attn_partials", d_attn_partials, G[1], "ldp_da"),
                                   ("dx_partials", dx_partials, G[0], "ldp_dx")):
        if g.bwd_size > 1:
            if len(parts) != g.bwd_size:
                raise ValueError(f"{name} needs {g.bwd_size} buffers")
            tab, arr, ld = _ptr_table(parts, T, g.k_loc, name, pdt)
            setattr(io, name, tab)
            setattr(io, ldname, ld)
            keep.append(arr)
    io.d_attn, io.ld_d_attn = _mat(d_attn, T, G[1].k_loc, torch.bfloat16, "d_attn")
    io.delta = _ptr(delta, "delta")
    io.d_qkv, io.ld_dqkv = _mat(d_qkv, T, G[0].n_loc, torch.bfloat16, "d_qkv")
    io.dx, io.ld_dx = _mat(dx, T, G[0].k_loc, torch.bfloat16, "dx")
    for i in range(2):
        g = G[i]
        r, c = (g.k_loc, g.n_loc) if weight_layout == ATP_W_KN else (g.n_loc, g.k_loc)
        p, ld = _mat(dw[i], r, c, torch.float32, f"dw[{LINEARS[i]}]")
        if ld != W.ldw[i]:
            raise ValueError(f"dw[{LINEARS[i]}] must share the weight's leading dimension")
        io.dw[i] = p
        io.db[i] = _vec(db[i], g.n_loc, torch.float32, f"db[{LINEARS[i]}]") if db else None
    wsp, wsb = _workspace(workspace)
    _check(load_library().atp_attention_block_bwd(
        ctypes.byref(m), int(block_mode), int(batch), int(seq), int(h), int(heads), int(chunks),
        ctypes.byref(W), ctypes.byref(io), wsp, wsb, _stream(compute_stream),
        _stream(comm_stream)))


# ---------------------------------------------------------------------------
# Mesh planner (host only)
# ---------------------------------------------------------------------------
class Hcm:
    """A hierarchical communication matrix: `layers` is a list of
    (ranks, group_bw, p2p) outermost first, p2p a ranks x ranks nested list of
    GB/s or None (every pair at group_bw)."""

    def __init__(self, layers):
        self._keep = []
        arr = (atp_hcm_layer * len(layers))()
        for j, (ranks, group_bw, p2p) in enumerate(layers):
            arr[j].ranks = int(ranks)
            arr[j].group_bw = float(group_bw)
            if p2p is None:
                arr[j].p2p = None
            else:
                flat = (ctypes.c_double * (int(ranks) * int(ranks)))(
                    *[float(x) for row in p2p for x in row])
                self._keep.append(flat)
                arr[j].p2p = ctypes.cast(flat, ctypes.POINTER(ctypes.c_double))
        self.layers = arr
        self.n = len(layers)


def hcm_mi355x_xgmi(gpus: int = 8, link_gbs: float = 153.0) -> Hcm:
    """One MI355X node: `gpus` GPUs, every pair joined by one xGMI link of
    `link_gbs` GB/s, so a GPU's group bandwidth is (gpus - 1) links."""
    p2p = [[0.0 if u == v else link_gbs for v in range(gpus)] for u in range(gpus)]
    return Hcm([(gpus, (gpus - 1) * link_gbs, p2p)])


def model_dims(layers: int, batch: int, seq: int, hidden: int, elem_bytes: int = 2):
    return atp_model_dims(int(layers), int(batch), int(seq), int(hidden), int(elem_bytes))


def atp_tcomm(dims: atp_model_dims, d1: int, d2: int, b1: float, b2: float) -> float:
    t = ctypes.c_double()
    _check(load_library().atp_tcomm(ctypes.byref(dims), int(d1), int(d2), float(b1), float(b2),
                                    ctypes.byref(t)))
    return t.value


def atp_hcm_mesh_cost(hcm: Hcm, dims: atp_model_dims, d1: int, d2: int) -> dict:
    c = atp_mesh_cost()
    _check(load_library().atp_hcm_mesh_cost(hcm.layers, hcm.n, ctypes.byref(dims), int(d1),
                                            int(d2), ctypes.byref(c)))
    return c.as_dict()


def atp_plan_mesh(hcm: Hcm, dims: atp_model_dims, max_costs: int = 256):
    """(best mesh cost, costs of every candidate mesh, largest d1 first)."""
    best = atp_mesh_cost()
    arr = (atp_mesh_cost * max_costs)()
    n = ctypes.c_int32()
    _check(load_library().atp_plan_mesh(hcm.layers, hcm.n, ctypes.byref(dims), ctypes.byref(best),
                                        arr, int(max_costs), ctypes.byref(n)))
    return best.as_dict(), [arr[i].as_dict() for i in range(n.value)]
