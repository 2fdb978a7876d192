"""Host-side checks of the C ABI that need no GPU: the library loads and
exports every symbol include/atp.h declares, the shard geometry agrees with
the oracle's spec-derived geometry (Sec. 3.2), and every argument error is
reported before any device work (the pointers used here are never
dereferenced: each call fails validation first)."""
import ctypes
import itertools
import os
import re

import pytest

import oracle as O
import paper_2301_08658_amd as atp
from paper_2301_08658_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x10000          # 16-byte aligned, never dereferenced
MISALIGNED = 0x10004


def _declared_symbols():
    txt = open(os.path.join(ROOT, "include", "atp.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(atp_[a-z_0-9]+)\s*\(", txt)))


def test_library_exports_every_declared_symbol():
    lib = atp.load_library()
    decl = _declared_symbols()
    assert len(decl) >= 10
    for name in decl:
        assert hasattr(lib, name), name
    assert set(decl) == set(B.EXPORTS)
    assert "gfx950" in atp.atp_version()


@pytest.mark.parametrize("mesh", [(1, 1), (2, 2), (2, 4), (4, 2), (8, 1), (1, 8), (3, 2)])
@pytest.mark.parametrize("mode", [0, 1])
def test_geometry_matches_oracle(mesh, mode):
    d1, d2 = mesh
    K, N = 48 * 8, 96 * 8
    for i1, i2 in itertools.product(range(d1), range(d2)):
        g = atp.atp_shard_geometry(atp.mesh(d1, d2, i1, i2), mode, K, N)
        o = O.shard_geometry(mesh, (i1, i2), mode, K, N)
        assert (g.k_off, g.k_off + g.k_loc) == (o["k_lo"], o["k_hi"])
        assert (g.n_off, g.n_off + g.n_loc) == (o["n_lo"], o["n_hi"])
        assert (g.red_axis, g.red_size, g.red_index) == (o["red_axis"], o["red_size"],
                                                          o["red_index"])
        # backward reduces over the other mesh axis (the one that split N)
        other = 1 - o["red_axis"]
        assert (g.bwd_axis, g.bwd_size, g.bwd_index) == (other, mesh[other], (i1, i2)[other])


def _status(fn, *args):
    lib = atp.load_library()
    return getattr(lib, fn)(*args), atp.binding.last_error()


def test_geometry_errors():
    lib = atp.load_library()
    out = B.atp_shard()
    m = atp.mesh(2, 4, 1, 3)
    assert lib.atp_shard_geometry(None, 0, 8, 8, ctypes.byref(out)) == B.ATP_ERR_INVALID_ARGUMENT
    assert lib.atp_shard_geometry(ctypes.byref(m), 0, 8, 8, None) == B.ATP_ERR_INVALID_ARGUMENT
    assert lib.atp_shard_geometry(ctypes.byref(m), 2, 8, 8, ctypes.byref(out)) == \
        B.ATP_ERR_INVALID_ARGUMENT
    assert lib.atp_shard_geometry(ctypes.byref(m), 0, 7, 8, ctypes.byref(out)) == B.ATP_ERR_SHAPE
    assert lib.atp_shard_geometry(ctypes.byref(m), 0, 8, 6, ctypes.byref(out)) == B.ATP_ERR_SHAPE
    bad = atp.mesh(2, 4, 2, 0)
    assert lib.atp_shard_geometry(ctypes.byref(bad), 0, 8, 8, ctypes.byref(out)) == \
        B.ATP_ERR_INVALID_ARGUMENT
    assert "outside" in atp.binding.last_error()
    z = atp.mesh(0, 4, 0, 0)
    assert lib.atp_shard_geometry(ctypes.byref(z), 0, 8, 8, ctypes.byref(out)) == \
        B.ATP_ERR_INVALID_ARGUMENT


def _fwd(m, mode=0, tokens=64, k=256, n=256, chunks=2, x=FAKE, ldx=None, w=FAKE, ldw=None,
         bias=None, epi=0, y=FAKE, ydt=0, ldy=None, pre=None):
    g = atp.atp_shard_geometry(m, mode, 256, 256)
    lib = atp.load_library()
    return lib.atp_shard_linear_fwd(ctypes.byref(m), mode, tokens, k, n, chunks, x,
                                    ldx or g.k_loc, w, ldw or g.n_loc, bias, epi, y, ydt,
                                    ldy or g.n_loc, pre, None, None)


def test_linear_fwd_validation():
    m = atp.mesh(2, 2, 1, 0)
    assert _fwd(m, chunks=3) == B.ATP_ERR_SHAPE                 # 64 % 3
    assert _fwd(m, chunks=0) == B.ATP_ERR_INVALID_ARGUMENT
    assert _fwd(m, chunks=B.ATP_MAX_CHUNKS + 1, tokens=0) == B.ATP_ERR_INVALID_ARGUMENT
    assert _fwd(m, tokens=-1) == B.ATP_ERR_INVALID_ARGUMENT
    assert _fwd(m, x=None) == B.ATP_ERR_INVALID_ARGUMENT
    assert _fwd(m, x=MISALIGNED) == B.ATP_ERR_UNSUPPORTED
    assert _fwd(m, ldx=64) == B.ATP_ERR_INVALID_ARGUMENT         # ld < k_loc = 128
    assert _fwd(m, ldw=132) == B.ATP_ERR_UNSUPPORTED             # ld not a multiple of 8
    assert _fwd(m, k=255) == B.ATP_ERR_SHAPE
    # a partial output (group of 2) cannot take the bias / GeLU (f32 or bf16)
    assert _fwd(m, epi=1, bias=FAKE) == B.ATP_ERR_INVALID_ARGUMENT
    assert "Partial" in atp.binding.last_error()
    assert _fwd(m, ydt=1, epi=2, bias=FAKE) == B.ATP_ERR_INVALID_ARGUMENT
    # group of one: BIAS needs the bias vector; GELU_BWD is not a forward epilogue
    m1 = atp.mesh(1, 1, 0, 0)
    assert _fwd(m1, epi=1, bias=None) == B.ATP_ERR_INVALID_ARGUMENT
    assert _fwd(m1, epi=3) == B.ATP_ERR_INVALID_ARGUMENT
    assert _fwd(m1, epi=0, pre=FAKE) == B.ATP_ERR_INVALID_ARGUMENT   # preact only with GeLU
    assert _fwd(m1, ydt=7) == B.ATP_ERR_INVALID_ARGUMENT


def _red(red_size=2, tokens=64, n=256, chunks=2, parts=(FAKE, FAKE), ldp=256, bias=None,
         epi=0, pin=None, out=FAKE, odt=0, ldo=256, pout=None):
    lib = atp.load_library()
    arr = (ctypes.c_void_p * max(1, len(parts)))(*parts) if parts is not None else None
    tab = ctypes.cast(arr, B._fpp) if arr is not None else None
    return lib.atp_chunked_partial_reduce(red_size, tokens, n, chunks, tab, ldp, bias, epi, pin,
                                          out, odt, ldo, pout, None, None)


def test_reduce_validation():
    assert _red(red_size=0) == B.ATP_ERR_INVALID_ARGUMENT
    assert _red(red_size=B.ATP_MAX_GROUP + 1) == B.ATP_ERR_UNSUPPORTED
    assert _red(parts=None) == B.ATP_ERR_INVALID_ARGUMENT
    assert _red(parts=(FAKE, 0)) == B.ATP_ERR_INVALID_ARGUMENT
    assert "partials[1]" in atp.binding.last_error()
    assert _red(parts=(FAKE, MISALIGNED)) == B.ATP_ERR_UNSUPPORTED
    assert _red(chunks=5) == B.ATP_ERR_SHAPE
    assert _red(n=250, ldp=256, ldo=256) == B.ATP_ERR_UNSUPPORTED
    assert _red(ldp=128) == B.ATP_ERR_INVALID_ARGUMENT
    assert _red(epi=1) == B.ATP_ERR_INVALID_ARGUMENT               # bias missing
    assert _red(epi=3) == B.ATP_ERR_INVALID_ARGUMENT               # preact_in missing
    assert _red(epi=9) == B.ATP_ERR_INVALID_ARGUMENT
    assert _red(epi=1, bias=FAKE, pout=FAKE) == B.ATP_ERR_INVALID_ARGUMENT
    assert _red(odt=5) == B.ATP_ERR_INVALID_ARGUMENT


def test_reduce_bf16_validation():
    lib = atp.load_library()

    def red16(red_size=2, parts=(FAKE, FAKE), epi=0, bias=None):
        arr = (ctypes.c_void_p * max(1, len(parts)))(*parts)
        return lib.atp_chunked_partial_reduce_bf16(red_size, 64, 256, 2, ctypes.cast(arr, B._fpp),
                                                   256, bias, epi, None, FAKE, 1, 256, None,
                                                   None, None)
    assert red16(red_size=0) == B.ATP_ERR_INVALID_ARGUMENT
    assert red16(parts=(FAKE, 0)) == B.ATP_ERR_INVALID_ARGUMENT
    assert "partials[1]" in atp.binding.last_error()
    assert red16(parts=(FAKE, MISALIGNED)) == B.ATP_ERR_UNSUPPORTED
    assert red16(epi=1) == B.ATP_ERR_INVALID_ARGUMENT               # bias missing


def test_fused_linear_validation():
    lib = atp.load_library()

    def fused(m, tokens=64, k=256, n=512, peers=(FAKE, None), epi=0, bias=None, pre=None,
              odt=1):
        g = atp.atp_shard_geometry(m, 0, k, n)
        arr = (ctypes.c_void_p * max(1, len(peers)))(*[p or 0 for p in peers]) \
            if peers is not None else None
        tab = ctypes.cast(arr, B._fpp) if arr is not None else None
        return lib.atp_shard_linear_fwd_fused(ctypes.byref(m), 0, tokens, k, n, FAKE, g.k_loc,
                                              FAKE, g.n_loc, tab, g.n_loc, bias, epi, FAKE, odt,
                                              g.n_loc, pre, None)
    m = atp.mesh(2, 2, 1, 0)                  # row-first: group over d1, own index 1
    assert fused(m, epi=3) == B.ATP_ERR_INVALID_ARGUMENT            # GELU_BWD
    assert fused(m, peers=None) == B.ATP_ERR_INVALID_ARGUMENT
    assert fused(m, peers=(None, FAKE)) == B.ATP_ERR_INVALID_ARGUMENT
    assert "peers[0]" in atp.binding.last_error()
    assert fused(m, tokens=-1) == B.ATP_ERR_INVALID_ARGUMENT
    assert fused(m, epi=1) == B.ATP_ERR_INVALID_ARGUMENT            # bias missing
    assert fused(m, pre=FAKE) == B.ATP_ERR_INVALID_ARGUMENT         # preact only with GeLU
    assert fused(m, odt=4) == B.ATP_ERR_INVALID_ARGUMENT
    assert fused(atp.mesh(16, 1, 0, 0), k=4096, peers=(FAKE,) * 16) == B.ATP_ERR_UNSUPPORTED


def test_linear_bwd_validation():
    lib = atp.load_library()
    m = atp.mesh(2, 4, 1, 1)
    g = atp.atp_shard_geometry(m, 1, 256, 512)

    def call(**kw):
        a = dict(x=FAKE, ldx=g.k_loc, w=FAKE, ldw=g.n_loc, dy=FAKE, lddy=g.n_loc, dx=FAKE,
                 lddx=g.k_loc, dw=FAKE, lddw=g.n_loc, db=None, tokens=64, chunks=4)
        a.update(kw)
        return lib.atp_shard_linear_bwd(ctypes.byref(m), 1, a["tokens"], 256, 512, a["chunks"],
                                        a["x"], a["ldx"], a["w"], a["ldw"], a["dy"], a["lddy"],
                                        a["dx"], a["lddx"], a["dw"], a["lddw"], a["db"], None,
                                        None)
    assert call(dy=None) == B.ATP_ERR_INVALID_ARGUMENT
    assert call(dx=MISALIGNED) == B.ATP_ERR_UNSUPPORTED
    assert call(lddw=8) == B.ATP_ERR_INVALID_ARGUMENT
    assert call(chunks=3) == B.ATP_ERR_SHAPE
    assert call(db=MISALIGNED) == B.ATP_ERR_UNSUPPORTED


def test_block_validation():
    lib = atp.load_library()
    h, T = 512, 256
    m = atp.mesh(2, 2, 0, 1)
    G = atp.block_geometry(m, B.ATP_BLOCK_COL, h)
    W = B.atp_block_weights()
    for i, g in enumerate(G):
        W.w[i] = FAKE
        W.ldw[i] = g.n_loc
        W.b[i] = FAKE
    io = B.atp_block_fwd_io()
    io.x_loc, io.ldx = FAKE, G[0].k_loc
    io.attn_loc, io.lda = FAKE, G[1].k_loc
    io.qkv, io.ld_qkv = FAKE, G[0].n_loc
    io.o, io.ld_o = FAKE, G[1].n_loc
    io.h, io.ld_h = FAKE, G[2].n_loc
    io.pre = FAKE
    io.z, io.ld_z = FAKE, G[3].n_loc
    keep = []
    for i, g in enumerate(G):
        arr = (ctypes.c_void_p * g.red_size)(*([FAKE] * g.red_size))
        keep.append(arr)
        io.partials[i] = ctypes.cast(arr, B._fpp)
        io.ldp[i] = g.n_loc

    def call(mm=m, bm=0, tokens=T, hh=h, chunks=2):
        return lib.atp_block_fwd(ctypes.byref(mm), bm, tokens, hh, chunks, ctypes.byref(W),
                                 ctypes.byref(io), None, 0, None, None)
    assert call(bm=5) == B.ATP_ERR_INVALID_ARGUMENT
    assert call(hh=500) == B.ATP_ERR_UNSUPPORTED or call(hh=500) == B.ATP_ERR_SHAPE
    assert call(chunks=3) == B.ATP_ERR_SHAPE
    assert call(mm=atp.mesh(2, 2, 2, 0)) == B.ATP_ERR_INVALID_ARGUMENT
    io.partials[3] = None
    assert call() == B.ATP_ERR_INVALID_ARGUMENT
    assert "partials[fc2]" in atp.binding.last_error()
    io.partials[3] = ctypes.cast(keep[3], B._fpp)
    W.b[2] = None
    assert call() == B.ATP_ERR_INVALID_ARGUMENT
    W.b[2] = FAKE
    io.ld_h = G[2].n_loc - 8
    assert call() == B.ATP_ERR_INVALID_ARGUMENT
    assert lib.atp_block_workspace_bytes(ctypes.byref(m), 0, T, h, 2, 0) > 0


def test_status_strings():
    assert atp.binding.status_string(0) == "ATP_OK"
    assert atp.binding.status_string(2) == "ATP_ERR_SHAPE"
    assert atp.binding.status_string(99) == "ATP_ERR_UNKNOWN"


def test_block_workspace_bytes_formula():
    # forward: at most W^T of the four shards (a linear whose products stream
    # the weight as stored keeps no copy); backward: X^T of x, attention block, H
    # and dY^T of the four linears over the tokens; every row of a copy padded
    # by 64 values (128 bytes); pieces rounded to 256 B.
    # Each side adds the fp32 split-K slabs of its chunk products, at most
    # 512 tiles of 256 x 160 fp32 values, sized for the largest plan over
    # every chunk count (a 64-chunk split of the 8 x 1 wide layer splits, 8
    # chunks do not); no slabs without tokens
    r = lambda b: (b + 255) // 256 * 256  # noqa: E731
    slab_max = 512 * 256 * 160 * 4
    for (d1, d2), mode, T, h, splits in [((8, 1), 0, 4096, 20480, True),
                                         ((2, 4), 1, 8192, 4096, True),
                                         ((2, 2), 0, 132, 512, True), ((1, 1), 0, 0, 256, False)]:
        m = B.mesh(d1, d2, 0, 0)
        G = B.block_geometry(m, mode, h)
        fwd = sum(r((g.k_loc + 64) * g.n_loc * 2) for g in G)   # every W^T: an upper bound
        tp = T + 64
        colpart = ((T + 63) // 64) * max(g.n_loc for g in G) * 4   # fp32 column partials for db
        bwd = (r(G[0].k_loc * tp * 2) + r(G[1].k_loc * tp * 2) + r(G[3].k_loc * tp * 2) +
               sum(r(g.n_loc * tp * 2) for g in G) + r(colpart))
        sizes = {B.atp_block_workspace_bytes(m, mode, T, h, c) for c in (1, 2, 4)}
        assert len(sizes) == 1, sizes          # the chunk count does not change it
        ws = sizes.pop()
        assert ws % 256 == 0
        if splits:
            assert bwd < ws <= max(fwd, bwd) + slab_max
        else:
            assert bwd <= ws <= max(fwd, bwd)
    # invalid arguments give 0
    assert B.atp_block_workspace_bytes(B.mesh(2, 2, 0, 0), 7, 128, 512, 1) == 0
    assert B.atp_block_workspace_bytes(B.mesh(2, 2, 0, 0), 0, 128, 500, 1) == 0


def test_block_workspace_path_decides_the_capture_refusal():
    """atp_block_workspace_path is the decision the block calls take: the
    transposed-layout path needs the pass's whole workspace (and, for the
    backward, tokens % 8 == 0); everything else is the direct path, which the
    calls refuse under HIP graph capture."""
    m = B.mesh(2, 2, 1, 0)
    h = 512
    for layout in (B.ATP_W_KN, B.ATP_W_NK):
        for T in (256, 132):
            full = B.atp_block_workspace_bytes(m, 0, T, h, 2, layout)
            assert full > 0 and full % 256 == 0
            for p in (0, 1):
                path = lambda n: B.atp_block_workspace_path(m, 0, T, h, layout, n, p)  # noqa
                ok_tokens = p == 0 or T % 8 == 0
                assert path(full) == (1 if ok_tokens else 0)
                assert path(0) == 0                      # no workspace: direct
                if ok_tokens:
                    need = _least_size(m, 0, T, h, layout, p, full)
                    assert need % 256 == 0 and path(need - 1) == 0 and path(need) == 1
    assert B.atp_block_workspace_path(m, 0, 256, h, 7, 1 << 20, 0) == -1      # bad layout
    assert B.atp_block_workspace_path(m, 0, 256, h, 0, 1 << 20, 2) == -1      # bad pass
    assert B.atp_block_workspace_path(B.mesh(2, 2, 2, 0), 0, 256, h, 0, 1, 0) == -1


def _least_size(m, mode, T, h, layout, pass_, hi):
    """The least workspace size that takes the pass's transposed-layout path
    (binary search over the library's own decision; 0 if even `hi` does not)."""
    path = lambda n: B.atp_block_workspace_path(m, mode, T, h, layout, n, pass_)  # noqa: E731
    if path(hi) != 1:
        return 0
    lo = 0                      # path(lo) == 0 (no workspace is the direct path)
    while hi - lo > 1:
        mid = (lo + hi) // 2
        if path(mid) == 1:
            hi = mid
        else:
            lo = mid
    return hi


def test_block_workspace_weight_layouts():
    """Weights stored [n][k] need no W^T in the forward, and one [k][n] copy
    of the largest weight (rows padded by 64 values) in the backward.  Weights
    stored [k][n] add the W^T copies of some of the linears to the forward:
    those whose products, at some chunk count, are split over k or do not
    run on the 256 x 256 tiles.  On the wide 8 x 1 layer the two unchunked
    linears (QKV, fc1: one 4096-row product each) read W as stored, while
    out-proj and fc2 split at 64 chunks and keep their copies."""
    r = lambda b: (b + 255) // 256 * 256  # noqa: E731
    for (d1, d2), mode, T, h in [((8, 1), 0, 4096, 20480), ((2, 4), 1, 8192, 4096),
                                 ((2, 2), 0, 256, 512)]:
        m = B.mesh(d1, d2, 0, 0)
        G = B.block_geometry(m, mode, h)
        kn = B.atp_block_workspace_bytes(m, mode, T, h, 1, B.ATP_W_KN)
        nk = B.atp_block_workspace_bytes(m, mode, T, h, 1, B.ATP_W_NK)
        wkn = r(max(g.k_loc * (g.n_loc + 64) * 2 for g in G))
        wt = [r((g.k_loc + 64) * g.n_loc * 2) for g in G]
        assert (_least_size(m, mode, T, h, B.ATP_W_NK, 1, nk) -
                _least_size(m, mode, T, h, B.ATP_W_KN, 1, kn)) == wkn
        extra = (_least_size(m, mode, T, h, B.ATP_W_KN, 0, kn) -
                 _least_size(m, mode, T, h, B.ATP_W_NK, 0, nk))
        subsets = {sum(w for i, w in enumerate(wt) if mask >> i & 1) for mask in range(16)}
        assert extra in subsets, (extra, wt)
        if (d1, d2) == (8, 1):
            assert extra == wt[1] + wt[3]
    assert B.atp_block_workspace_bytes(B.mesh(2, 2, 0, 0), 0, 128, 512, 1, 5) == 0


def test_block_geometry_export_matches_per_linear_geometry():
    lib = atp.load_library()
    for (d1, d2) in [(2, 2), (2, 4), (4, 2), (8, 1), (1, 8)]:
        for i1, i2 in itertools.product(range(d1), range(d2)):
            m = atp.mesh(d1, d2, i1, i2)
            for bm, modes in ((B.ATP_BLOCK_COL, (1, 0, 1, 0)), (B.ATP_BLOCK_ROW, (0, 1, 0, 1))):
                G = B.block_geometry(m, bm, 1024)
                for g, md, (k, n) in zip(G, modes, ((1024, 3072), (1024, 1024), (1024, 4096),
                                                    (4096, 1024))):
                    assert g.as_dict() == atp.atp_shard_geometry(m, md, k, n).as_dict()
    out = (B.atp_shard * 4)()
    m = atp.mesh(2, 2, 0, 0)
    assert lib.atp_block_geometry(ctypes.byref(m), 0, 1024, None) == B.ATP_ERR_INVALID_ARGUMENT
    assert lib.atp_block_geometry(ctypes.byref(m), 3, 1024, out) == B.ATP_ERR_INVALID_ARGUMENT
    assert lib.atp_block_geometry(ctypes.byref(m), 0, 1001, out) == B.ATP_ERR_SHAPE
    assert lib.atp_block_geometry(ctypes.byref(m), 0, 1000, out) == B.ATP_ERR_UNSUPPORTED


def test_attention_heads_export_matches_oracle():
    """The device's run of heads equals the oracle's scatter of the QKV
    block's heads over its reduction group (Sec. 3.2.1)."""
    h, heads = 2048, 16
    for (d1, d2) in [(2, 2), (2, 4), (4, 2), (8, 1), (1, 4)]:
        for bm in (B.ATP_BLOCK_COL, B.ATP_BLOCK_ROW):
            for i1, i2 in itertools.product(range(d1), range(d2)):
                m = atp.mesh(d1, d2, i1, i2)
                g = B.block_geometry(m, bm, h)[0]
                first, count, per_block = B.attention_heads(m, bm, h, heads)
                assert per_block * 3 * 128 == g.n_loc
                lo, n = O.attention_heads(g.n_loc, 128, g.red_size, g.red_index)
                assert (first, count) == (lo, n)
    lib = atp.load_library()
    m = atp.mesh(2, 2, 0, 0)
    i = ctypes.c_int32()
    assert lib.atp_attention_heads(ctypes.byref(m), 0, 2048, 16, None, ctypes.byref(i),
                                   ctypes.byref(i)) == B.ATP_ERR_INVALID_ARGUMENT
    assert lib.atp_attention_heads(ctypes.byref(m), 0, 2048, 15, ctypes.byref(i), ctypes.byref(i),
                                   ctypes.byref(i)) == B.ATP_ERR_SHAPE
    assert lib.atp_attention_heads(ctypes.byref(m), 0, 2048, 32, ctypes.byref(i), ctypes.byref(i),
                                   ctypes.byref(i)) == B.ATP_ERR_UNSUPPORTED   # head dim 64


def test_block_option_validation():
    """An unknown weight layout or partial dtype is refused before any work."""
    lib = atp.load_library()
    h, T = 512, 256
    m = atp.mesh(2, 2, 0, 1)
    G = atp.block_geometry(m, B.ATP_BLOCK_COL, h)
    W = B.atp_block_weights()
    for i, g in enumerate(G):
        W.w[i], W.ldw[i], W.b[i] = FAKE, g.n_loc, FAKE
    io = B.atp_block_fwd_io()
    io.x_loc, io.ldx = FAKE, G[0].k_loc
    io.attn_loc, io.lda = FAKE, G[1].k_loc
    io.qkv, io.ld_qkv = FAKE, G[0].n_loc
    io.o, io.ld_o = FAKE, G[1].n_loc
    io.h, io.ld_h = FAKE, G[2].n_loc
    io.pre = FAKE
    io.z, io.ld_z = FAKE, G[3].n_loc

    def call():
        return lib.atp_block_fwd(ctypes.byref(m), 0, T, h, 2, ctypes.byref(W), ctypes.byref(io),
                                 None, 0, None, None)
    W.layout = 2
    assert call() == B.ATP_ERR_INVALID_ARGUMENT and "layout" in atp.binding.last_error()
    W.layout = B.ATP_W_NK          # [n][k] weights: ld 128 < k_loc 256
    assert call() == B.ATP_ERR_INVALID_ARGUMENT and "w[" in atp.binding.last_error()
    W.layout = B.ATP_W_KN
    io.partial_dtype = 3
    assert call() == B.ATP_ERR_INVALID_ARGUMENT and "partial_dtype" in atp.binding.last_error()


def test_binding_refuses_host_tensors_and_short_scratch():
    """A host tensor, or an lse / delta buffer smaller than the device's
    heads need, is refused by the binding before the library is called."""
    import torch
    m = atp.mesh(2, 2, 0, 0)
    T, h, heads = 256, 1024, 8
    _, hd, _ = atp.attention_heads(m, 0, h, heads)
    g = atp.block_geometry(m, 0, h)[0]
    qkv = torch.zeros((T, g.n_loc), dtype=torch.bfloat16)
    out = torch.zeros((T, g.n_loc // 3), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="lse"):
        atp.atp_attention_fwd(m, 0, 1, T, h, heads, qkv, out,
                              torch.zeros(hd * T - 1, dtype=torch.float32))
    with pytest.raises(ValueError, match="delta"):
        atp.atp_attention_bwd(m, 0, 1, T, h, heads, qkv, out,
                              torch.zeros(hd * T, dtype=torch.float32), out, qkv,
                              torch.zeros(hd * T - 8, dtype=torch.float32))
    with pytest.raises(ValueError, match="on the GPU"):
        atp.atp_attention_fwd(m, 0, 1, T, h, heads, qkv, out,
                              torch.zeros(hd * T, dtype=torch.float32))
    with pytest.raises(ValueError, match="on the GPU"):
        atp.atp_transpose_bf16(qkv, torch.zeros((g.n_loc, T), dtype=torch.bfloat16))
    with pytest.raises(ValueError, match="on the GPU"):
        atp.atp_chunked_partial_reduce(1, T, 8, 1, [torch.zeros((T, 8))], None, 0,
                                       torch.zeros((T, 8)))


def test_binding_partial_dtype_of_tables():
    import torch
    f, h = torch.zeros(2), torch.zeros(2, dtype=torch.bfloat16)
    assert B._partial_dtype([None, [f, None, f]]) == (B.ATP_F32, torch.float32)
    assert B._partial_dtype([[h], None]) == (B.ATP_BF16, torch.bfloat16)
    assert B._partial_dtype([None, None]) == (B.ATP_F32, torch.float32)
    with pytest.raises(TypeError):
        B._partial_dtype([[f], [h]])
    with pytest.raises(TypeError):
        B._partial_dtype([[torch.zeros(2, dtype=torch.float16)]])


def test_noalloc_attention_bwd_refuses_beyond_its_scratch():
    """More delta values than the library's scratch holds is refused before
    any device work (the pointers are never dereferenced)."""
    lib = atp.load_library()
    m = atp.mesh(1, 1, 0, 0)
    h, heads = 4096, 32                      # 32 heads on the device
    seq = B.ATP_NOALLOC_DELTA_MAX // heads + 1
    g = atp.block_geometry(m, 0, h)[0]
    st = lib.atp_attention_bwd_noalloc(ctypes.byref(m), 0, 1, seq, h, heads, FAKE, g.n_loc, FAKE,
                                       g.n_loc // 3, FAKE, FAKE, g.n_loc // 3, FAKE, g.n_loc, None)
    assert st == B.ATP_ERR_UNSUPPORTED
    assert "scratch" in atp.binding.last_error()


def test_attention_refuses_overlapping_buffers():
    """The attention core refuses an output that shares memory with an input
    (not only an identical pointer) before any device work; the addresses
    are never dereferenced."""
    lib = atp.load_library()
    m = atp.mesh(1, 1, 0, 0)
    T, h, heads = 256, 1024, 8
    g = atp.block_geometry(m, 0, h)[0]
    nq, no = g.n_loc, g.n_loc // 3
    inside = FAKE + 2 * (T // 2) * nq           # a row in the middle of qkv (bf16)
    past = FAKE + 2 * T * nq                    # the first byte after qkv
    fwd = lambda out: lib.atp_attention_fwd(ctypes.byref(m), 0, 1, T, h, heads,  # noqa: E731
                                            FAKE, nq, out, no, FAKE, None)
    assert fwd(inside) == B.ATP_ERR_INVALID_ARGUMENT
    assert "overlap" in atp.binding.last_error()
    far = 0x40000000                            # disjoint from qkv; d_qkv below overlaps it
    bwd = lambda dqkv: lib.atp_attention_bwd(  # noqa: E731
        ctypes.byref(m), 0, 1, T, h, heads, FAKE, nq, far, no, FAKE, past, no, dqkv, nq,
        FAKE, None)
    for dqkv in (FAKE + 16 * nq, far - 16 * nq, past + 32):
        assert bwd(dqkv) == B.ATP_ERR_INVALID_ARGUMENT, hex(dqkv)
        assert "overlap" in atp.binding.last_error()


def test_attention_block_bwd_refuses_misaligned_workspace():
    """A workspace that is not 256-byte aligned is refused before any work;
    every buffer address is distinct and never dereferenced (mesh 1 x 1: no
    reduction tables)."""
    lib = atp.load_library()
    m = atp.mesh(1, 1, 0, 0)
    h, heads, batch, seq = 1024, 8, 1, 256
    T = batch * seq
    gq, go = atp.block_geometry(m, B.ATP_BLOCK_COL, h)[:2]
    addr = iter(range(1 << 36, 1 << 42, 1 << 36))   # far apart: no two buffers overlap
    W = B.atp_block_weights()
    W.layout = B.ATP_W_KN
    for i, g in enumerate((gq, go)):
        W.w[i], W.ldw[i], W.b[i] = next(addr), g.n_loc, next(addr)
    io = B.atp_attn_block_bwd_io()
    io.x_loc, io.ldx = next(addr), gq.k_loc
    io.qkv, io.ld_qkv = next(addr), gq.n_loc
    io.attn, io.ld_attn = next(addr), go.k_loc
    io.lse = next(addr)
    io.d_o, io.ld_do = next(addr), go.n_loc
    io.d_attn, io.ld_d_attn = next(addr), go.k_loc
    io.delta = next(addr)
    io.d_qkv, io.ld_dqkv = next(addr), gq.n_loc
    io.dx, io.ld_dx = next(addr), gq.k_loc
    for i in range(2):
        io.dw[i], io.db[i] = next(addr), next(addr)
    ws = next(addr)
    st = lib.atp_attention_block_bwd(ctypes.byref(m), 0, batch, seq, h, heads, 1, ctypes.byref(W),
                                     ctypes.byref(io), ws + 16, 1 << 30, None, None)
    assert st == B.ATP_ERR_INVALID_ARGUMENT
    assert "workspace" in atp.binding.last_error()
