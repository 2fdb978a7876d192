"""The attention core of one device (Sec. 2.1 Formula (mha), causal; the
attention block of Sec. 3.2.1) against the oracle on the same seeded QKV
block: the device's run of heads, its output columns of the gathered
out-proj input (the other members' columns untouched) and the row
log-sum-exps, over meshes, block modes, coordinates, ragged sequence
lengths and several sequences."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2301_08658_amd as atp
import synth_inputs as S
from bounds import attention_prob_bounds, delta_bounds
from helpers import DEV, assert_close, block_mode_code, to64

pytestmark = pytest.mark.gpu
HD = 128


def _run(mode, mesh, coord, batch, seq, h, seed, sigma=1.0):
    m = atp.mesh(mesh[0], mesh[1], coord[0], coord[1])
    bm = block_mode_code(mode)
    heads = h // HD
    g = atp.block_geometry(m, bm, h)[0]
    T = batch * seq
    qkv = S.randn_bf16((T, g.n_loc), sigma, seed, 301).to(DEV)
    first, hd, per_block = atp.attention_heads(m, bm, h, heads)
    out = torch.full((T, g.n_loc // 3), -7.0, dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((hd, T), dtype=torch.float32, device=DEV)
    atp.atp_attention_fwd(m, bm, batch, seq, h, heads, qkv, out, lse)
    torch.cuda.synchronize()
    ref_o, ref_lse = O.attention_core_local(qkv.cpu(), batch, seq, HD, g.red_size, g.red_index)
    return out, lse, ref_o, ref_lse, first, hd


@pytest.mark.parametrize("mode,mesh,coord,batch,seq,h", [
    ("col", (2, 2), (1, 0), 1, 64, 512),
    ("col", (2, 2), (0, 1), 2, 100, 512),      # ragged tile
    ("row", (2, 2), (1, 1), 3, 130, 512),
    ("col", (1, 1), (0, 0), 2, 1, 512),        # one token
    ("col", (2, 4), (1, 2), 2, 257, 4096),     # GPT h=4096 heads, 4 per device
    ("row", (4, 2), (3, 1), 1, 192, 4096),
    ("col", (8, 1), (5, 0), 1, 320, 4096),     # Megatron's mesh: whole block per device
])
def test_attention_fwd_matches_oracle(mode, mesh, coord, batch, seq, h):
    print(f"attention {mode} {mesh} {coord} b={batch} s={seq} h={h}", flush=True)
    out, lse, ref_o, ref_lse, first, hd = _run(mode, mesh, coord, batch, seq, h, seed=51)
    cols = slice(first * HD, (first + hd) * HD)
    assert_close(out[:, cols], ref_o, "attention output")
    np.testing.assert_allclose(to64(lse), ref_lse, rtol=0, atol=2e-3)
    rest = torch.ones(out.shape[1], dtype=torch.bool)
    rest[cols] = False
    assert torch.all(out[:, rest.to(DEV)] == -7.0), "columns of other group members written"


def test_attention_fwd_full_gpt_sequence():
    """Four 2048-token sequences of the GPT h=4096 layer on the 2 x 4 mesh."""
    out, lse, ref_o, ref_lse, first, hd = _run("col", (2, 4), (0, 3), 4, 2048, 4096, seed=52)
    cols = slice(first * HD, (first + hd) * HD)
    assert_close(out[:, cols], ref_o, "attention output")
    np.testing.assert_allclose(to64(lse), ref_lse, rtol=0, atol=2e-3)


def test_attention_fwd_128_row_tiles_ragged():
    """Enough heads and sequences for 128-row query tiles (two workgroups per
    CU): four 130-token sequences, 64 heads, so each second tile holds two
    live rows."""
    batch, seq, h = 4, 130, 8192
    assert ((seq + 127) // 128) * batch * (h // HD) >= 512
    out, lse, ref_o, ref_lse, first, hd = _run("col", (1, 1), (0, 0), batch, seq, h, seed=54)
    cols = slice(first * HD, (first + hd) * HD)
    assert_close(out[:, cols], ref_o, "attention output")
    np.testing.assert_allclose(to64(lse), ref_lse, rtol=0, atol=2e-3)


@pytest.mark.parametrize("batch,seq,h", [
    (2, 300, 512),      # 64-row tiles, key range split between two wave groups
    (4, 130, 8192),     # 128-row tiles, two workgroups per CU
])
def test_attention_fwd_sharp_scores(batch, seq, h):
    """Queries scaled by 4 (exact in bf16): score rows with a standard
    deviation of ~5.8 in base 2, so row maxima pass the running reference
    point at irregular key steps and the softmax is close to one-hot (the
    forward's conditional rescale).  Values keep std 1."""
    m = atp.mesh(1, 1, 0, 0)
    heads = h // HD
    g = atp.block_geometry(m, atp.ATP_BLOCK_COL, h)[0]
    T = batch * seq
    qkv = S.randn_bf16((T, g.n_loc), 1.0, 56, 304)
    for hh in range(heads):
        qkv[:, hh * 3 * HD:hh * 3 * HD + HD] *= 4
    ref_o, ref_lse = O.attention_core_local(qkv, batch, seq, HD, g.red_size, g.red_index)
    qkv = qkv.to(DEV)
    out = torch.empty((T, h), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((heads, T), dtype=torch.float32, device=DEV)
    atp.atp_attention_fwd(m, atp.ATP_BLOCK_COL, batch, seq, h, heads, qkv, out, lse)
    torch.cuda.synchronize()
    assert_close(out, ref_o, "attention output")
    np.testing.assert_allclose(to64(lse), ref_lse, rtol=0, atol=2e-3)


def test_attention_fwd_growing_scores():
    """q = 1 and key j = j/16 in every dimension: the score of key j is
    8 j / sqrt(128), about 1.02 j in base 2, so every key step raises each
    row's maximum by ~65 and the output is rescaled at every step; weights
    fall off geometrically behind the diagonal."""
    m = atp.mesh(1, 1, 0, 0)
    h, seq, heads = 512, 300, 4
    g = atp.block_geometry(m, atp.ATP_BLOCK_COL, h)[0]
    qkv = S.randn_bf16((seq, g.n_loc), 1.0, 57, 303)
    ramp = (torch.arange(seq, dtype=torch.float32) / 16).to(torch.bfloat16)
    for hh in range(heads):
        qkv[:, hh * 3 * HD:hh * 3 * HD + HD] = 1
        qkv[:, hh * 3 * HD + HD:hh * 3 * HD + 2 * HD] = ramp[:, None]
    ref_o, ref_lse = O.attention_core_local(qkv, 1, seq, HD, g.red_size, g.red_index)
    qkv = qkv.to(DEV)
    out = torch.empty((seq, h), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((heads, seq), dtype=torch.float32, device=DEV)
    atp.atp_attention_fwd(m, atp.ATP_BLOCK_COL, 1, seq, h, heads, qkv, out, lse)
    torch.cuda.synchronize()
    assert_close(out, ref_o, "attention output")
    np.testing.assert_allclose(to64(lse), ref_lse, rtol=1e-6, atol=2e-3)


def test_attention_fwd_wide_share_sampled():
    """The benchmark's attention share (h = 20480 on the 8 x 1 mesh: 20 heads
    per device, two 2048-token sequences; 128-row tiles) against the oracle
    on sampled (sequence, head) pairs, each computed alone."""
    m = atp.mesh(8, 1, 3, 0)
    h, batch, seq = 20480, 2, 2048
    g = atp.block_geometry(m, atp.ATP_BLOCK_COL, h)[0]
    first, hd, _ = atp.attention_heads(m, atp.ATP_BLOCK_COL, h, h // HD)
    assert (first, hd) == (0, 20)
    T = batch * seq
    qkv = S.randn_bf16((T, g.n_loc), 1.0, 55, 308).to(DEV)
    out = torch.empty((T, g.n_loc // 3), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((hd, T), dtype=torch.float32, device=DEV)
    atp.atp_attention_fwd(m, atp.ATP_BLOCK_COL, batch, seq, h, h // HD, qkv, out, lse)
    torch.cuda.synchronize()
    q = qkv.cpu()
    for b, hh in ((1, 0), (0, 11), (1, 19)):
        rows = slice(b * seq, (b + 1) * seq)
        c = 3 * HD * hh
        ref_o, ref_lse = O.attention_fwd(q[rows, c:c + HD], q[rows, c + HD:c + 2 * HD],
                                         q[rows, c + 2 * HD:c + 3 * HD])
        assert_close(out[rows, hh * HD:(hh + 1) * HD], ref_o, f"sequence {b} head {hh}")
        np.testing.assert_allclose(to64(lse[hh, rows]), ref_lse, rtol=0, atol=2e-3)


def test_attention_fwd_uniform_queries_give_prefix_means():
    """q = 0: every row averages the values of its prefix (closed form)."""
    m = atp.mesh(1, 1, 0, 0)
    h, seq = 512, 150
    g = atp.block_geometry(m, atp.ATP_BLOCK_COL, h)[0]
    qkv = S.randn_bf16((seq, g.n_loc), 1.0, 53, 302).to(DEV)
    for hh in range(4):
        qkv[:, hh * 3 * HD:hh * 3 * HD + HD] = 0
    out = torch.empty((seq, h), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((4, seq), dtype=torch.float32, device=DEV)
    atp.atp_attention_fwd(m, atp.ATP_BLOCK_COL, 1, seq, h, 4, qkv, out, lse)
    torch.cuda.synchronize()
    q = to64(qkv)
    for hh in range(4):
        v = q[:, hh * 3 * HD + 2 * HD:hh * 3 * HD + 3 * HD]
        prefix = np.cumsum(v, axis=0) / np.arange(1, seq + 1)[:, None]
        assert_close(out[:, hh * HD:(hh + 1) * HD], prefix, f"head {hh}")
    np.testing.assert_allclose(to64(lse), np.log(np.arange(1, seq + 1))[None, :].repeat(4, 0),
                               rtol=0, atol=1e-5)


def test_attention_fwd_empty_and_errors():
    m = atp.mesh(2, 2, 0, 0)
    z = torch.empty((0, 768), dtype=torch.bfloat16, device=DEV)
    atp.atp_attention_fwd(m, atp.ATP_BLOCK_COL, 0, 64, 512, 4, z,
                          torch.empty((0, 256), dtype=torch.bfloat16, device=DEV), None)
    qkv = torch.zeros((64, 768), dtype=torch.bfloat16, device=DEV)
    out = torch.zeros((64, 256), dtype=torch.bfloat16, device=DEV)
    lse = torch.zeros((2, 64), dtype=torch.float32, device=DEV)
    with pytest.raises(atp.AtpError):       # head dimension 64 is not built
        atp.atp_attention_fwd(m, atp.ATP_BLOCK_COL, 1, 64, 512, 8, qkv, out, lse)


@pytest.mark.parametrize("mode,mesh,coord,batch,seq,h", [
    ("col", (2, 2), (1, 0), 1, 64, 512),
    ("col", (2, 2), (0, 1), 2, 100, 512),      # ragged tile
    ("row", (2, 2), (1, 1), 3, 130, 512),
    ("col", (1, 1), (0, 0), 2, 1, 512),        # one token
    ("col", (2, 4), (1, 2), 2, 257, 4096),
    ("row", (4, 2), (3, 1), 1, 192, 4096),
    ("col", (1, 1), (0, 0), 4, 260, 8192),     # 1280 tiles: loops not split
])
def test_attention_bwd_matches_oracle(mode, mesh, coord, batch, seq, h):
    print(f"attention bwd {mode} {mesh} {coord} b={batch} s={seq} h={h}", flush=True)
    m = atp.mesh(mesh[0], mesh[1], coord[0], coord[1])
    bm = block_mode_code(mode)
    heads = h // HD
    g = atp.block_geometry(m, bm, h)[0]
    T = batch * seq
    qkv = S.randn_bf16((T, g.n_loc), 1.0, 61, 303).to(DEV)
    first, hd, per_block = atp.attention_heads(m, bm, h, heads)
    out = torch.zeros((T, g.n_loc // 3), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((hd, T), dtype=torch.float32, device=DEV)
    atp.atp_attention_fwd(m, bm, batch, seq, h, heads, qkv, out, lse)
    d_out = S.randn_bf16((T, g.n_loc // 3), 1.0, 61, 304).to(DEV)
    d_qkv = torch.full((T, g.n_loc), -5.0, dtype=torch.bfloat16, device=DEV)
    delta = torch.empty((hd * T,), dtype=torch.float32, device=DEV)
    atp.atp_attention_bwd(m, bm, batch, seq, h, heads, qkv, out, lse, d_out, d_qkv, delta)
    torch.cuda.synchronize()
    cols = slice(first * HD, (first + hd) * HD)
    ref = O.attention_core_bwd_local(qkv.cpu(), d_out[:, cols].cpu(), batch, seq, HD,
                                     g.red_size, g.red_index)
    mine = slice(first * 3 * HD, (first + hd) * 3 * HD)
    got = d_qkv[:, mine]
    # error terms of dQ and dK from delta over the stored bf16 output
    extra = np.zeros((T, 3 * HD * hd))
    qc, dc = qkv.cpu(), d_out.cpu()
    for bb in range(batch):
        rows = slice(bb * seq, (bb + 1) * seq)
        for j in range(hd):
            c = 3 * HD * (first + j)
            bq, bk = delta_bounds(qc[rows, c:c + HD], qc[rows, c + HD:c + 2 * HD],
                                  qc[rows, c + 2 * HD:c + 3 * HD],
                                  dc[rows, (first + j) * HD:(first + j + 1) * HD])
            extra[rows, 3 * HD * j:3 * HD * j + HD] = bq
            extra[rows, 3 * HD * j + HD:3 * HD * j + 2 * HD] = bk
    for part, nm in ((0, "dq"), (1, "dk"), (2, "dv")):
        sel = np.concatenate([np.arange(j * 3 * HD + part * HD, j * 3 * HD + (part + 1) * HD)
                              for j in range(hd)])
        assert_close(got[:, torch.as_tensor(sel, device=DEV)], ref[:, sel], nm,
                     extra=extra[:, sel])
    rest = torch.ones(g.n_loc, dtype=torch.bool)
    rest[mine] = False
    assert torch.all(d_qkv[:, rest.to(DEV)] == -5.0), "columns of other group members written"


@pytest.mark.parametrize("batch,seq,h", [
    (2, 300, 512),      # loops split between two wave groups
    (4, 260, 8192),     # 1280 tiles: loops not split, 128-row dQ tiles
])
def test_attention_bwd_sharp_scores(batch, seq, h):
    """The backward on queries scaled by 4 (exact in bf16; values and dO keep
    std 1): near one-hot rows put P close to 1 for many queries of one key,
    so the bf16 P and dS of the second products carry errors beyond the
    generic tolerance; their derived terms (bounds.attention_prob_bounds)
    join the delta terms."""
    m = atp.mesh(1, 1, 0, 0)
    heads = h // HD
    g = atp.block_geometry(m, atp.ATP_BLOCK_COL, h)[0]
    T = batch * seq
    qkv = S.randn_bf16((T, g.n_loc), 1.0, 64, 311)
    for hh in range(heads):
        qkv[:, hh * 3 * HD:hh * 3 * HD + HD] *= 4
    d_out = S.randn_bf16((T, h), 1.0, 64, 312)
    ref = O.attention_core_bwd_local(qkv, d_out, batch, seq, HD, g.red_size, g.red_index)
    extra = np.zeros((T, 3 * h))
    for bb in range(batch):
        rows = slice(bb * seq, (bb + 1) * seq)
        for j in range(heads):
            c = 3 * HD * j
            args = (qkv[rows, c:c + HD], qkv[rows, c + HD:c + 2 * HD],
                    qkv[rows, c + 2 * HD:c + 3 * HD], d_out[rows, j * HD:(j + 1) * HD])
            bq, bk = delta_bounds(*args)
            pq, pk, pv = attention_prob_bounds(*args)
            extra[rows, c:c + HD] = bq + pq
            extra[rows, c + HD:c + 2 * HD] = bk + pk
            extra[rows, c + 2 * HD:c + 3 * HD] = pv
    qkv, d_out = qkv.to(DEV), d_out.to(DEV)
    out = torch.empty((T, h), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((heads, T), dtype=torch.float32, device=DEV)
    atp.atp_attention_fwd(m, atp.ATP_BLOCK_COL, batch, seq, h, heads, qkv, out, lse)
    d_qkv = torch.full((T, 3 * h), -5.0, dtype=torch.bfloat16, device=DEV)
    delta = torch.empty((heads * T,), dtype=torch.float32, device=DEV)
    atp.atp_attention_bwd(m, atp.ATP_BLOCK_COL, batch, seq, h, heads, qkv, out, lse, d_out,
                          d_qkv, delta)
    torch.cuda.synchronize()
    for part, nm in ((0, "dq"), (1, "dk"), (2, "dv")):
        sel = np.concatenate([np.arange(j * 3 * HD + part * HD, j * 3 * HD + (part + 1) * HD)
                              for j in range(heads)])
        assert_close(d_qkv[:, torch.as_tensor(sel, device=DEV)], ref[:, sel], nm,
                     extra=extra[:, sel])


def test_attention_bwd_wide_share_sampled():
    """The benchmark's attention share backward (h = 20480 on 8 x 1: 20 heads,
    two 2048-token sequences) against the oracle on one (sequence, head)."""
    m = atp.mesh(8, 1, 6, 0)
    h, batch, seq, heads = 20480, 2, 2048, 160
    g = atp.block_geometry(m, atp.ATP_BLOCK_COL, h)[0]
    first, hd, _ = atp.attention_heads(m, atp.ATP_BLOCK_COL, h, heads)
    T = batch * seq
    qkv = S.randn_bf16((T, g.n_loc), 1.0, 63, 309).to(DEV)
    out = torch.empty((T, g.n_loc // 3), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((hd, T), dtype=torch.float32, device=DEV)
    atp.atp_attention_fwd(m, atp.ATP_BLOCK_COL, batch, seq, h, heads, qkv, out, lse)
    d_out = S.randn_bf16((T, g.n_loc // 3), 1.0, 63, 310).to(DEV)
    d_qkv = torch.empty((T, g.n_loc), dtype=torch.bfloat16, device=DEV)
    delta = torch.empty((hd * T,), dtype=torch.float32, device=DEV)
    atp.atp_attention_bwd(m, atp.ATP_BLOCK_COL, batch, seq, h, heads, qkv, out, lse, d_out,
                          d_qkv, delta)
    torch.cuda.synchronize()
    b, hh = 1, 13
    rows = slice(b * seq, (b + 1) * seq)
    c = 3 * HD * hh
    q = qkv[rows].cpu()
    args = (q[:, c:c + HD], q[:, c + HD:c + 2 * HD], q[:, c + 2 * HD:c + 3 * HD],
            d_out[rows, hh * HD:(hh + 1) * HD].cpu())
    dq, dk, dv = O.attention_bwd(*args)
    bq, bk = delta_bounds(*args)
    for part, ref, nm, ex in ((0, dq, "dq", bq), (1, dk, "dk", bk), (2, dv, "dv", None)):
        assert_close(d_qkv[rows, c + part * HD:c + (part + 1) * HD], ref, nm, extra=ex)


def test_attention_bwd_deterministic():
    m = atp.mesh(2, 4, 1, 1)
    h, batch, seq = 4096, 2, 300
    g = atp.block_geometry(m, atp.ATP_BLOCK_COL, h)[0]
    T = batch * seq
    qkv = S.randn_bf16((T, g.n_loc), 1.0, 62, 305).to(DEV)
    first, hd, _ = atp.attention_heads(m, atp.ATP_BLOCK_COL, h, 32)
    out = torch.zeros((T, g.n_loc // 3), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((hd, T), dtype=torch.float32, device=DEV)
    atp.atp_attention_fwd(m, atp.ATP_BLOCK_COL, batch, seq, h, 32, qkv, out, lse)
    d_out = S.randn_bf16((T, g.n_loc // 3), 1.0, 62, 306).to(DEV)
    res = []
    for _ in range(2):
        d_qkv = torch.zeros((T, g.n_loc), dtype=torch.bfloat16, device=DEV)
        delta = torch.empty((hd * T,), dtype=torch.float32, device=DEV)
        atp.atp_attention_bwd(m, atp.ATP_BLOCK_COL, batch, seq, h, 32, qkv, out, lse, d_out,
                              d_qkv, delta)
        res.append(d_qkv)
    torch.cuda.synchronize()
    assert torch.equal(res[0], res[1])


@pytest.mark.parametrize("mode,mesh", [("col", (2, 2)), ("row", (2, 4)), ("col", (4, 2)),
                                       ("col", (8, 1))])
def test_attention_block_scatter_gather_equals_unsharded(mode, mesh):
    """Every coordinate of the mesh: the members of each scatter group write
    their heads into one shared buffer (the all-gather); it equals the
    attention of the unsharded layer restricted to the block's heads, and
    the group's lse rows are the unsharded ones."""
    h, batch, seq = 1024, 2, 96
    heads = h // HD
    T = batch * seq
    bm = block_mode_code(mode)
    qkv_full = S.randn_bf16((T, 3 * h), 1.0, 71, 307)          # unsharded QKV output
    ref_full, ref_lse = O.attention_core_local(qkv_full, batch, seq, HD, 1, 0)
    d1, d2 = mesh
    gathered = {}
    for i1 in range(d1):
        for i2 in range(d2):
            m = atp.mesh(d1, d2, i1, i2)
            g = atp.block_geometry(m, bm, h)[0]
            blk = qkv_full[:, g.n_off:g.n_off + g.n_loc].contiguous().to(DEV)
            key = g.n_off                       # the group sharing this block
            if key not in gathered:
                gathered[key] = (torch.full((T, g.n_loc // 3), -9.0, dtype=torch.bfloat16,
                                            device=DEV), [], g)
            first, hd, _ = atp.attention_heads(m, bm, h, heads)
            lse = torch.empty((hd, T), dtype=torch.float32, device=DEV)
            atp.atp_attention_fwd(m, bm, batch, seq, h, heads, blk, gathered[key][0], lse)
            gathered[key][1].append((first, lse))
    torch.cuda.synchronize()
    assert len(gathered) * next(iter(gathered.values()))[2].red_size == d1 * d2
    for n_off, (buf, lses, g) in gathered.items():
        h0 = n_off // (3 * HD)                  # the block's first head in the layer
        cols = slice(h0 * HD, h0 * HD + g.n_loc // 3)
        assert_close(buf, ref_full[:, cols], f"block at column {n_off}")
        for first, lse in lses:
            hd = lse.shape[0]
            np.testing.assert_allclose(to64(lse), ref_lse[h0 + first:h0 + first + hd],
                                       rtol=0, atol=2e-3)
