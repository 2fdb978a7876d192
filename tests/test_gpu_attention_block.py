"""The attention block of one device, chained (Sec. 3.2.1 with Formula (mha)
as its core): QKV -> scatter of the reduced QKV block's heads over the group
that reduced it -> causal attention core -> all-gather -> out-proj, and the
backward through the same chain (Sec. 4.2).

Every coordinate of the mesh runs on the one GPU.  The peers' data each
device needs (their Partial(SUM) blocks, their heads' attention outputs for
the all-gather, their heads' d_qkv columns) are computed first with the
single-step calls, then every device makes the chained call.  Checked:

* every output against the unsharded attention block of the strict fp64
  oracle (the spec invariant for this block), the device's blocks
  selected by the output specs;
* the chained call gives the bits of the single-step sequence;
* members of each reduction group hold identical bits;
* the columns of the gathered buffers owned by other members are left as
  they were (the call writes its own heads' columns only).

Tolerance: the stated 1e-2 (|ref| + 1) elementwise and 5e-3 Frobenius.  The
attention output adds its first-order response to the bf16 QKV block it
reads (bounds.attention_qkv_sensitivity), and o and out-proj's dW the
rounding of that bf16 output carried through their products.  The
attention backward's dq, dk add the term of its delta over the stored bf16
output (bounds.delta_bounds) and every d_qkv column the exact linear
response to the bf16 d_attn it reads (bounds.attention_dout_sensitivity);
QKV's dX, dW add those and the bf16 rounding of d_qkv carried through their
products, and db the same terms for the token sums, taken from the linear
maps (sum_u dV_u = sum_t dO_t carries d_attn's rounding one to one)."""
import itertools

import numpy as np
import pytest
import torch

import bounds
import oracle as O
import paper_2301_08658_amd as atp
import synth_inputs as S
from helpers import DEV, assert_close, block_mode_code, group_table, to64

pytestmark = pytest.mark.gpu
HD = 128


def _bits(t):
    return t.contiguous().view(torch.int16 if t.element_size() == 2 else torch.int32)


def _group(c, axis, size):
    """Coordinates of the group along `axis` that contains c, in group order."""
    return [tuple(c[:axis]) + (j,) + tuple(c[axis + 1:]) for j in range(size)]


def _key(c, axis):
    """Identifies the group along `axis` (the coordinate on the other axis)."""
    return c[1 - axis]


@pytest.mark.parametrize("mode,mesh,seq", [("col", (2, 2), 128), ("col", (2, 4), 128),
                                           ("col", (4, 2), 128), ("col", (8, 1), 128),
                                           ("row", (2, 2), 128),
                                           ("col", (2, 2), 200)])   # ragged key / query tiles
def test_attention_block_every_coordinate(mode, mesh, seq):
    d1, d2 = mesh
    h, heads, batch, chunks = 1024, 8, 2, 2
    T = batch * seq
    bm = block_mode_code(mode)
    print(f"attention block {mode} {mesh} seq {seq}", flush=True)
    X = S.randn_bf16((T, h), 1.0, 81, 1)
    Wq = S.randn_bf16((h, 3 * h), 0.02, 81, 2)
    bq = S.randn_bf16((3 * h,), 0.02, 81, 3)
    Wo = S.randn_bf16((h, h), 0.02, 81, 4)
    bo = S.randn_bf16((h,), 0.02, 81, 5)
    dO = S.randn_bf16((T, h), 1.0, 81, 6)
    coords = list(itertools.product(range(d1), range(d2)))
    bf = lambda r, c_: torch.empty((r, c_), dtype=torch.bfloat16, device=DEV)  # noqa: E731
    nan = lambda r, c_, dt=torch.float32: torch.full((r, c_), float("nan"), dtype=dt,  # noqa
                                                     device=DEV)
    L = {}
    for c in coords:
        m = atp.mesh(d1, d2, *c)
        gq, go = atp.block_geometry(m, bm, h)[:2]
        first, hd, _ = atp.attention_heads(m, bm, h, heads)
        L[c] = dict(m=m, gq=gq, go=go, first=first, hd=hd,
                    x=X[:, gq.k_off:gq.k_off + gq.k_loc].contiguous().to(DEV),
                    wq=Wq[gq.k_off:gq.k_off + gq.k_loc, gq.n_off:gq.n_off + gq.n_loc]
                    .contiguous().to(DEV),
                    bq=bq[gq.n_off:gq.n_off + gq.n_loc].contiguous().to(DEV),
                    wo=Wo[go.k_off:go.k_off + go.k_loc, go.n_off:go.n_off + go.n_loc]
                    .contiguous().to(DEV),
                    bo=bo[go.n_off:go.n_off + go.n_loc].contiguous().to(DEV),
                    do=dO[:, go.n_off:go.n_off + go.n_loc].contiguous().to(DEV))
        assert gq.n_off == 3 * go.k_off and gq.n_loc == 3 * go.k_loc
    g0q, g0o = L[coords[0]]["gq"], L[coords[0]]["go"]
    qax, oax = g0q.red_axis, g0o.red_axis          # scatter group = QKV's group
    qbax, obax = g0q.bwd_axis, g0o.bwd_axis
    mode_of = lambda g: atp.ATP_COL_FIRST if g.red_axis == 1 else atp.ATP_ROW_FIRST  # noqa

    # ---- the peers' data, from the single-step calls
    Pq, Qred, lse, Po = {}, {}, {}, {}
    for c in coords:
        l_ = L[c]
        Pq[c] = torch.empty((T, l_["gq"].n_loc), device=DEV)
        atp.atp_shard_linear_fwd(l_["m"], mode_of(l_["gq"]), T, h, 3 * h, chunks, l_["x"],
                                 l_["wq"], None, 0, Pq[c])
    Ag = {}
    for c in coords:
        l_, gq = L[c], L[c]["gq"]
        Qred[c] = bf(T, gq.n_loc)
        atp.atp_chunked_partial_reduce(gq.red_size, T, gq.n_loc, chunks,
                                       [Pq[p] for p in _group(c, qax, gq.red_size)], l_["bq"],
                                       atp.ATP_EPI_BIAS, Qred[c])
        k = _key(c, qax)
        if k not in Ag:
            Ag[k] = torch.full((T, l_["go"].k_loc), -9.0, dtype=torch.bfloat16, device=DEV)
        lse[c] = torch.empty((l_["hd"], T), device=DEV)
        atp.atp_attention_fwd(l_["m"], bm, batch, seq, h, heads, Qred[c], Ag[k], lse[c])
    for c in coords:
        l_ = L[c]
        Po[c] = torch.empty((T, l_["go"].n_loc), device=DEV)
        atp.atp_shard_linear_fwd(l_["m"], mode_of(l_["go"]), T, h, h, chunks, Ag[_key(c, qax)],
                                 l_["wo"], None, 0, Po[c])
    torch.cuda.synchronize()

    # ---- the chained forward on every device
    F = {}
    for c in coords:
        l_, gq, go = L[c], L[c]["gq"], L[c]["go"]
        own_q = nan(T, gq.n_loc) if gq.red_size > 1 else None
        own_o = nan(T, go.n_loc) if go.red_size > 1 else None
        qtab = [own_q if p == c else Pq[p] for p in _group(c, qax, gq.red_size)]
        otab = [own_o if p == c else Po[p] for p in _group(c, oax, go.red_size)]
        attn = Ag[_key(c, qax)].clone()
        cols = slice(l_["first"] * HD, (l_["first"] + l_["hd"]) * HD)
        attn[:, cols] = float("nan")
        out = dict(qkv=nan(T, gq.n_loc, torch.bfloat16), attn=attn,
                   lse=torch.full((l_["hd"], T), float("nan"), device=DEV),
                   o=nan(T, go.n_loc, torch.bfloat16))
        atp.atp_attention_block_fwd(l_["m"], bm, batch, seq, h, heads, chunks,
                                    [l_["wq"], l_["wo"]], [l_["bq"], l_["bo"]], l_["x"],
                                    qtab if gq.red_size > 1 else None, out["qkv"], out["attn"],
                                    out["lse"], otab if go.red_size > 1 else None, out["o"],
                                    comm_stream=torch.cuda.Stream())
        F[c] = out
    torch.cuda.synchronize()

    ref = O.attention_block_global(X, Wq, bq, Wo, bo, batch, seq, HD)
    # the core reads the reduced QKV block in bf16 (its first-order response),
    # and out-proj reads the core's output in bf16
    sens_a = np.zeros((T, h))
    for j in range(heads):
        cq = 3 * HD * j
        for b in range(batch):
            r = slice(b * seq, (b + 1) * seq)
            qkv_h = [ref["qkv"][r, cq + e * HD:cq + (e + 1) * HD] for e in range(3)]
            sens_a[r, j * HD:(j + 1) * HD] = bounds.attention_qkv_sensitivity(
                *qkv_h, *[bounds.rounding_var(t_) for t_ in qkv_h])
    var_a = bounds.rounding_var(ref["attn"]) + sens_a
    extra_attn = bounds.SIGMAS * np.sqrt(sens_a)
    extra_o = bounds.left(var_a, O._f64(Wo))
    for c in coords:
        l_, gq, go, out = L[c], L[c]["gq"], L[c]["go"], F[c]
        # the chained call gives the single-step sequence's bits
        assert torch.equal(_bits(out["qkv"]), _bits(Qred[c])), c
        assert torch.equal(_bits(out["attn"]), _bits(Ag[_key(c, qax)])), c
        assert torch.equal(_bits(out["lse"]), _bits(lse[c])), c
        # against the unsharded block
        assert_close(out["qkv"], ref["qkv"][:, gq.n_off:gq.n_off + gq.n_loc], f"qkv {c}")
        ka = slice(go.k_off, go.k_off + go.k_loc)
        assert_close(out["attn"], ref["attn"][:, ka], f"attn {c}", extra=extra_attn[:, ka])
        heads_lo = gq.n_off // (3 * HD) + l_["first"]
        np.testing.assert_allclose(to64(out["lse"]), ref["lse"][heads_lo:heads_lo + l_["hd"]],
                                   rtol=0, atol=2e-3)
        no = slice(go.n_off, go.n_off + go.n_loc)
        assert_close(out["o"], ref["o"][:, no], f"o {c}", extra=extra_o[:, no])
        for p in _group(c, oax, go.red_size):
            assert torch.equal(_bits(F[p]["o"]), _bits(out["o"])), (c, p)

    # ---- the peers' backward data, from the single-step calls
    Qa, Dred, Dq, Qx = {}, {}, {}, {}
    for c in coords:
        l_, go = L[c], L[c]["go"]
        Qa[c] = torch.empty((T, go.k_loc), device=DEV)
        scratch_w = torch.empty((go.k_loc, go.n_loc), device=DEV)
        atp.atp_shard_linear_bwd(l_["m"], mode_of(go), T, h, h, chunks, Ag[_key(c, qax)],
                                 l_["wo"], l_["do"], Qa[c], scratch_w)
    for c in coords:
        l_, gq, go = L[c], L[c]["gq"], L[c]["go"]
        Dred[c] = bf(T, go.k_loc)
        atp.atp_chunked_partial_reduce(go.bwd_size, T, go.k_loc, chunks,
                                       [Qa[p] for p in _group(c, obax, go.bwd_size)], None,
                                       atp.ATP_EPI_NONE, Dred[c])
        k = _key(c, qax)
        if k not in Dq:
            Dq[k] = torch.full((T, gq.n_loc), -9.0, dtype=torch.bfloat16, device=DEV)
        delta = torch.empty(l_["hd"] * T, device=DEV)
        atp.atp_attention_bwd(l_["m"], bm, batch, seq, h, heads, Qred[c], Ag[k], lse[c],
                              Dred[c], Dq[k], delta)
    for c in coords:
        l_, gq = L[c], L[c]["gq"]
        Qx[c] = torch.empty((T, gq.k_loc), device=DEV)
        scratch_w = torch.empty((gq.k_loc, gq.n_loc), device=DEV)
        atp.atp_shard_linear_bwd(l_["m"], mode_of(gq), T, h, 3 * h, chunks, l_["x"], l_["wq"],
                                 Dq[_key(c, qax)], Qx[c], scratch_w)
    torch.cuda.synchronize()

    # ---- the chained backward on every device
    B = {}
    for c in coords:
        l_, gq, go = L[c], L[c]["gq"], L[c]["go"]
        own_a = nan(T, go.k_loc) if go.bwd_size > 1 else None
        own_x = nan(T, gq.k_loc) if gq.bwd_size > 1 else None
        atab = [own_a if p == c else Qa[p] for p in _group(c, obax, go.bwd_size)]
        xtab = [own_x if p == c else Qx[p] for p in _group(c, qbax, gq.bwd_size)]
        d_qkv = Dq[_key(c, qax)].clone()
        qcols = slice(l_["first"] * 3 * HD, (l_["first"] + l_["hd"]) * 3 * HD)
        d_qkv[:, qcols] = float("nan")
        out = dict(d_attn=nan(T, go.k_loc, torch.bfloat16), d_qkv=d_qkv,
                   dx=nan(T, gq.k_loc, torch.bfloat16),
                   dw=[nan(gq.k_loc, gq.n_loc), nan(go.k_loc, go.n_loc)],
                   db=[torch.full((gq.n_loc,), float("nan"), device=DEV),
                       torch.full((go.n_loc,), float("nan"), device=DEV)])
        delta = torch.empty(l_["hd"] * T, device=DEV)
        atp.atp_attention_block_bwd(l_["m"], bm, batch, seq, h, heads, chunks,
                                    [l_["wq"], l_["wo"]], [l_["bq"], l_["bo"]], l_["x"],
                                    F[c]["qkv"], F[c]["attn"], F[c]["lse"], l_["do"],
                                    atab if go.bwd_size > 1 else None, out["d_attn"], delta,
                                    out["d_qkv"], xtab if gq.bwd_size > 1 else None, out["dx"],
                                    out["dw"], out["db"], comm_stream=torch.cuda.Stream())
        B[c] = out
        # the same call with a workspace (dW from transposed copies, db from
        # the dY transpose) gives the same bits; the workspace starts as
        # all-ones bytes (NaN in both dtypes), so nothing may be read from it
        # before the call writes it
        nb = atp.atp_block_workspace_bytes(l_["m"], bm, T, h, chunks, atp.ATP_W_KN)
        assert atp.atp_block_workspace_path(l_["m"], bm, T, h, atp.ATP_W_KN, nb, 1) == 1
        ws = torch.full((nb,), 255, dtype=torch.uint8, device=DEV)
        d_qkv2 = Dq[_key(c, qax)].clone()
        d_qkv2[:, qcols] = float("nan")
        own_a2 = nan(T, go.k_loc) if go.bwd_size > 1 else None
        own_x2 = nan(T, gq.k_loc) if gq.bwd_size > 1 else None
        out2 = dict(d_attn=nan(T, go.k_loc, torch.bfloat16), d_qkv=d_qkv2,
                    dx=nan(T, gq.k_loc, torch.bfloat16),
                    dw=[nan(gq.k_loc, gq.n_loc), nan(go.k_loc, go.n_loc)],
                    db=[torch.full((gq.n_loc,), float("nan"), device=DEV),
                        torch.full((go.n_loc,), float("nan"), device=DEV)])
        atp.atp_attention_block_bwd(
            l_["m"], bm, batch, seq, h, heads, chunks, [l_["wq"], l_["wo"]],
            [l_["bq"], l_["bo"]], l_["x"], F[c]["qkv"], F[c]["attn"], F[c]["lse"], l_["do"],
            [own_a2 if p == c else Qa[p] for p in _group(c, obax, go.bwd_size)]
            if go.bwd_size > 1 else None, out2["d_attn"], torch.empty(l_["hd"] * T, device=DEV),
            out2["d_qkv"], [own_x2 if p == c else Qx[p] for p in _group(c, qbax, gq.bwd_size)]
            if gq.bwd_size > 1 else None, out2["dx"], out2["dw"], out2["db"], workspace=ws,
            comm_stream=torch.cuda.Stream())
        torch.cuda.synchronize()
        for key in ("d_attn", "d_qkv", "dx"):
            assert torch.equal(_bits(out2[key]), _bits(out[key])), (c, key)
        for i in range(2):
            assert torch.equal(_bits(out2["dw"][i]), _bits(out["dw"][i])), (c, "dw", i)
            assert torch.equal(_bits(out2["db"][i]), _bits(out["db"][i])), (c, "db", i)
    torch.cuda.synchronize()

    g = O.attention_block_global_bwd(X, Wq, Wo, ref, dO, batch, seq, HD)
    # the attention backward's delta term, per head over the whole layer
    bq_all, bk_all = np.zeros((T, h)), np.zeros((T, h))
    for j in range(heads):
        cq = 3 * HD * j
        for b in range(batch):
            r = slice(b * seq, (b + 1) * seq)
            q_, k_, v_ = (ref["qkv"][r, cq + e * HD:cq + (e + 1) * HD] for e in range(3))
            e_q, e_k = bounds.delta_bounds(q_, k_, v_, g["d_attn"][r, j * HD:(j + 1) * HD])
            bq_all[r, j * HD:(j + 1) * HD] = e_q
            bk_all[r, j * HD:(j + 1) * HD] = e_k
    # the core's backward reads d_attn in bf16: its exact linear response
    # (per element, and for the token sums that the bias gradient takes)
    var_delta = np.zeros((T, 3 * h))
    var_prop, sum_prop = np.zeros((T, 3 * h)), np.zeros(3 * h)
    for j in range(heads):
        cq = 3 * HD * j
        var_delta[:, cq:cq + HD] = (bq_all[:, j * HD:(j + 1) * HD] / bounds.SIGMAS) ** 2
        var_delta[:, cq + HD:cq + 2 * HD] = (bk_all[:, j * HD:(j + 1) * HD] / bounds.SIGMAS) ** 2
        for b in range(batch):
            r = slice(b * seq, (b + 1) * seq)
            q_, k_, v_ = (ref["qkv"][r, cq + e * HD:cq + (e + 1) * HD] for e in range(3))
            sens = bounds.attention_dout_sensitivity(
                q_, k_, v_, bounds.rounding_var(g["d_attn"][r, j * HD:(j + 1) * HD]))
            for e, key in enumerate(("dq", "dk", "dv")):
                var_prop[r, cq + e * HD:cq + (e + 1) * HD] = sens[key]
                sum_prop[cq + e * HD:cq + (e + 1) * HD] += sens["sum_" + key]
    extra_dqkv = bounds.SIGMAS * np.sqrt(var_delta + var_prop)
    # d_qkv reaches QKV's products in bf16, carrying the terms above
    var_dqkv = bounds.rounding_var(g["d_qkv"]) + var_delta + var_prop
    Wq64, X64 = O._f64(Wq), O._f64(X)
    extra_dx = bounds.left(var_dqkv, Wq64.T)
    extra_dw = bounds.right(X64, var_dqkv)
    extra_db = bounds.SIGMAS * np.sqrt(
        (bounds.rounding_var(g["d_qkv"]) + var_delta).sum(0) + sum_prop)
    extra_dw_out = bounds.right_var(var_a, O._f64(dO))
    for c in coords:
        l_, gq, go, out = L[c], L[c]["gq"], L[c]["go"], B[c]
        assert torch.equal(_bits(out["d_attn"]), _bits(Dred[c])), c
        assert torch.equal(_bits(out["d_qkv"]), _bits(Dq[_key(c, qax)])), c
        kq, nq = slice(gq.k_off, gq.k_off + gq.k_loc), slice(gq.n_off, gq.n_off + gq.n_loc)
        ko, no = slice(go.k_off, go.k_off + go.k_loc), slice(go.n_off, go.n_off + go.n_loc)
        assert_close(out["d_attn"], g["d_attn"][:, ko], f"d_attn {c}")
        qc = slice(gq.n_off + l_["first"] * 3 * HD, gq.n_off + (l_["first"] + l_["hd"]) * 3 * HD)
        lc = slice(l_["first"] * 3 * HD, (l_["first"] + l_["hd"]) * 3 * HD)
        assert_close(out["d_qkv"][:, lc], g["d_qkv"][:, qc], f"d_qkv {c}", extra=extra_dqkv[:, qc])
        assert_close(out["dx"], g["dx"][:, kq], f"dx {c}", extra=extra_dx[:, kq])
        assert_close(out["dw"][0], g["dw_qkv"][kq, nq], f"dw_qkv {c}", extra=extra_dw[kq, nq])
        assert_close(out["db"][0], g["db_qkv"][nq], f"db_qkv {c}", extra=extra_db[nq])
        assert_close(out["dw"][1], g["dw_out"][ko, no], f"dw_out {c}", extra=extra_dw_out[ko, no])
        assert_close(out["db"][1], g["db_out"][no], f"db_out {c}")
        for p in _group(c, qbax, gq.bwd_size):
            assert torch.equal(_bits(B[p]["dx"]), _bits(out["dx"])), (c, p)


def test_attention_block_nk_weights_and_bf16_partials():
    """One device with seeded peers (bench mode): [n][k] weights give the
    bits of [k][n] weights, and both partial dtypes match the oracle's chain
    on the same inputs (bf16 partials: each own partial rounded once, the
    derived single-rounding term added)."""
    mesh, c, h, heads, batch, seq, chunks = (2, 2), (1, 0), 1024, 8, 1, 256, 2
    m = atp.mesh(*mesh, *c)
    bm = atp.ATP_BLOCK_COL
    gq, go = atp.block_geometry(m, bm, h)[:2]
    first, hd, _ = atp.attention_heads(m, bm, h, heads)
    T = batch * seq
    x = S.randn_bf16((T, gq.k_loc), 1.0, 82, 1)
    wq = S.randn_bf16((gq.k_loc, gq.n_loc), 0.02, 82, 2)
    wo = S.randn_bf16((go.k_loc, go.n_loc), 0.02, 82, 3)
    bq = S.randn_bf16((gq.n_loc,), 0.02, 82, 4)
    bo = S.randn_bf16((go.n_loc,), 0.02, 82, 5)
    peer_q = S.randn_bf16((T, gq.n_loc), 0.5, 82, 6)
    peer_o = S.randn_bf16((T, go.n_loc), 0.5, 82, 7)
    gathered = S.randn_bf16((T, go.k_loc), 0.5, 82, 8)

    def run(layout, pdt):
        wts = [wq, wo] if layout == atp.ATP_W_KN else [wq.t().contiguous(), wo.t().contiguous()]
        qt = group_table(torch.empty((T, gq.n_loc), dtype=pdt, device=DEV),
                         [peer_q.to(DEV, pdt)], gq.red_index)
        ot = group_table(torch.empty((T, go.n_loc), dtype=pdt, device=DEV),
                         [peer_o.to(DEV, pdt)], go.red_index)
        out = dict(qkv=torch.empty((T, gq.n_loc), dtype=torch.bfloat16, device=DEV),
                   attn=gathered.to(DEV), lse=torch.empty((hd, T), device=DEV),
                   o=torch.empty((T, go.n_loc), dtype=torch.bfloat16, device=DEV))
        atp.atp_attention_block_fwd(m, bm, batch, seq, h, heads, chunks,
                                    [w_.to(DEV) for w_ in wts], [bq.to(DEV), bo.to(DEV)],
                                    x.to(DEV), qt, out["qkv"], out["attn"], out["lse"], ot,
                                    out["o"], comm_stream=torch.cuda.Stream(),
                                    weight_layout=layout)
        return out

    print("attention block options", flush=True)
    a = run(atp.ATP_W_KN, torch.float32)
    b = run(atp.ATP_W_NK, torch.float32)
    z = run(atp.ATP_W_KN, torch.bfloat16)
    torch.cuda.synchronize()
    for key in ("qkv", "attn", "lse", "o"):
        assert torch.equal(_bits(a[key]), _bits(b[key])), key
    # the oracle's chain on the same inputs (peers exact in either dtype)
    own_q = O.matmul(x, wq)
    qkv = O.partial_reduce(group_table(own_q, [peer_q], gq.red_index), bq, O.EPI_BIAS)[0]
    attn = O._f64(gathered)
    cols = slice(first * HD, (first + hd) * HD)
    attn[:, cols] = O.attention_core_local(qkv, batch, seq, HD, gq.red_size, gq.red_index)[0]
    own_o = O.matmul(attn, wo)
    o = O.partial_reduce(group_table(own_o, [peer_o], go.red_index), bo, O.EPI_BIAS)[0]
    for out, pb16 in ((a, False), (z, True)):
        assert_close(out["qkv"], qkv, "qkv", extra=bounds.single(own_q) if pb16 else None)
        assert_close(out["attn"], attn, "attn")
        # out-proj reads the bf16 attention output (and, with bf16 partials,
        # its own partial is rounded once)
        var_a = np.zeros_like(attn)
        var_a[:, cols] = bounds.rounding_var(attn[:, cols])
        e = bounds.left(var_a, O._f64(wo)) + (bounds.single(own_o) if pb16 else 0.0)
        assert_close(out["o"], o, "o", extra=e)


def test_attention_block_workspace_path_full_size():
    """The benchmark's attention block (h = 20480 on DeviceMesh(8, 1), 2 x 2048
    tokens, 8 forward chunks, one device with seeded peers): the backward with
    a workspace (dW from transposed copies on the 256-wide NT tiles, db from
    the dY transpose) gives the bits of the backward without one, on every
    output.  The path without a workspace is checked against the oracle on
    every coordinate above."""
    w = S.WORKLOADS["wide_h20480_col_8x1"]
    d1, d2 = w["mesh"]
    h, T, chunks, sw = w["h"], w["tokens"], w["chunks"], w["sigma_w"]
    heads, seq = h // HD, 2048
    batch = T // seq
    m = atp.mesh(d1, d2, d1 - 1, 0)
    bm = atp.ATP_BLOCK_COL
    gq, go = atp.block_geometry(m, bm, h)[:2]
    _, hd, _ = atp.attention_heads(m, bm, h, heads)
    rnd = lambda shape, std, tid, dt=torch.bfloat16: S.randn_device(  # noqa: E731
        shape, std, 83, tid, DEV, dtype=dt)
    nan = lambda r, c_, dt=torch.float32: torch.full((r, c_), float("nan"), dtype=dt,  # noqa
                                                     device=DEV)

    def table(size, cols, tid0):
        return None if size == 1 else [rnd((T, cols), 0.5, tid0 + j, torch.float32)
                                       for j in range(size)]
    x = rnd((T, gq.k_loc), 1.0, 1)
    wts = [rnd((gq.k_loc, gq.n_loc), sw, 2), rnd((go.k_loc, go.n_loc), sw, 3)]
    bs = [rnd((gq.n_loc,), 0.02, 4), rnd((go.n_loc,), 0.02, 5)]
    qkv = torch.empty((T, gq.n_loc), dtype=torch.bfloat16, device=DEV)
    attn = rnd((T, go.k_loc), 1.0, 6)
    lse = torch.empty((hd, T), device=DEV)
    o = torch.empty((T, go.n_loc), dtype=torch.bfloat16, device=DEV)
    print(f"attention block full size, forward (h={h}, T={T}, {hd} heads)", flush=True)
    atp.atp_attention_block_fwd(m, bm, batch, seq, h, heads, chunks, wts, bs, x,
                                table(gq.red_size, gq.n_loc, 10), qkv, attn, lse,
                                table(go.red_size, go.n_loc, 30), o,
                                comm_stream=torch.cuda.Stream())
    d_o = rnd((T, go.n_loc), 1.0, 7)
    dq0 = rnd((T, gq.n_loc), 1.0, 8)
    atab, xtab = table(go.bwd_size, go.k_loc, 50), table(gq.bwd_size, gq.k_loc, 70)
    nb = atp.atp_block_workspace_bytes(m, bm, T, h, chunks, atp.ATP_W_KN)
    assert atp.atp_block_workspace_path(m, bm, T, h, atp.ATP_W_KN, nb, 1) == 1
    res = []
    for ws in (None, torch.full((nb,), 255, dtype=torch.uint8, device=DEV)):
        print(f"attention block full size, backward, workspace {ws is not None}", flush=True)
        def own(tab, idx):
            """The group's table with a fresh own entry (written by the call)."""
            return None if tab is None else [nan(T, t.shape[1]) if j == idx else t
                                             for j, t in enumerate(tab)]
        out = dict(d_attn=nan(T, go.k_loc, torch.bfloat16), d_qkv=dq0.clone(),
                   dx=nan(T, gq.k_loc, torch.bfloat16),
                   dw=[nan(gq.k_loc, gq.n_loc), nan(go.k_loc, go.n_loc)],
                   db=[torch.full((gq.n_loc,), float("nan"), device=DEV),
                       torch.full((go.n_loc,), float("nan"), device=DEV)])
        atp.atp_attention_block_bwd(m, bm, batch, seq, h, heads, 1, wts, bs, x, qkv, attn, lse,
                                    d_o, own(atab, go.bwd_index), out["d_attn"],
                                    torch.empty(hd * T, device=DEV), out["d_qkv"],
                                    own(xtab, gq.bwd_index), out["dx"], out["dw"], out["db"],
                                    workspace=ws, comm_stream=torch.cuda.Stream())
        torch.cuda.synchronize()
        res.append(out)
    a, b = res
    for key in ("d_attn", "d_qkv", "dx"):
        assert not torch.isnan(a[key].float()).any(), key
        assert torch.equal(_bits(a[key]), _bits(b[key])), key
    for i in range(2):
        assert not torch.isnan(a["dw"][i]).any() and not torch.isnan(a["db"][i]).any(), i
        assert torch.equal(_bits(a["dw"][i]), _bits(b["dw"][i])), ("dw", i)
        assert torch.equal(_bits(a["db"][i]), _bits(b["db"][i])), ("db", i)


@pytest.mark.parametrize("mode,mesh,coord,h,heads,batch,seq,chunks", [
    ("col", (2, 4), (1, 2), 2048, 16, 2, 512, 2),
    ("col", (8, 1), (3, 0), 2048, 16, 1, 512, 4),
    ("row", (2, 2), (1, 1), 1024, 8, 2, 128, 2)])
def test_attention_block_forward_workspace_path(mode, mesh, coord, h, heads, batch, seq, chunks):
    """The forward with a workspace (chunk products split over k into slabs
    where the chunk has too few tiles, from W^T copies) against the forward
    without one: the split sums in another order, so the outputs agree to
    fp32 rounding (bf16 outputs within two units in the last place), and the
    split kernels run only on the workspace path."""
    from helpers import assert_paths_agree
    bm = block_mode_code(mode)
    m = atp.mesh(*mesh, *coord)
    gq, go = atp.block_geometry(m, bm, h)[:2]
    _, hd, _ = atp.attention_heads(m, bm, h, heads)
    T = batch * seq
    rnd = lambda shape, std, tid, dt=torch.bfloat16: S.randn_device(  # noqa: E731
        shape, std, 84, tid, DEV, dtype=dt)
    x = rnd((T, gq.k_loc), 1.0, 1)
    wts = [rnd((gq.k_loc, gq.n_loc), 0.02, 2), rnd((go.k_loc, go.n_loc), 0.02, 3)]
    bs = [rnd((gq.n_loc,), 0.02, 4), rnd((go.n_loc,), 0.02, 5)]
    peers = [None if g.red_size == 1 else [rnd((T, g.n_loc), 0.5, 10 * i + j, torch.float32)
                                           for j in range(g.red_size)]
             for i, g in enumerate((gq, go))]
    gathered = rnd((T, go.k_loc), 1.0, 6)
    nb = atp.atp_block_workspace_bytes(m, bm, T, h, chunks, atp.ATP_W_KN)
    res, names = [], []
    for ws in (None, torch.full((nb,), 255, dtype=torch.uint8, device=DEV)):
        print(f"attention block forward {mode} {mesh} workspace {ws is not None}", flush=True)
        tabs = [None if p is None else [torch.full_like(t, float("nan")) if j == g.red_index
                                        else t for j, t in enumerate(p)]
                for p, g in zip(peers, (gq, go))]
        out = dict(qkv=torch.full((T, gq.n_loc), float("nan"), dtype=torch.bfloat16, device=DEV),
                   attn=gathered.clone(), lse=torch.full((hd, T), float("nan"), device=DEV),
                   o=torch.full((T, go.n_loc), float("nan"), dtype=torch.bfloat16, device=DEV))
        atp.atp_profile_enable(2)
        try:
            atp.atp_attention_block_fwd(m, bm, batch, seq, h, heads, chunks, wts, bs, x, tabs[0],
                                        out["qkv"], out["attn"], out["lse"], tabs[1], out["o"],
                                        workspace=ws, comm_stream=torch.cuda.Stream())
            torch.cuda.synchronize()
            names.append([r["name"] for r in atp.atp_profile_collect(256)])
        finally:
            atp.atp_profile_enable(0)
        res.append(out)
    a, b = res
    for key in ("qkv", "attn", "o"):
        assert not torch.isnan(a[key].float()).any() and not torch.isnan(b[key].float()).any()
        assert_paths_agree(a[key], b[key], key)
    assert_paths_agree(a["lse"], b["lse"], "lse")
    assert not any(n.startswith("gemm_nt_splitk") for n in names[0]), names[0]
    if mode == "col" and mesh == (2, 4):
        assert any(n.startswith("gemm_nt_splitk") for n in names[1]), names[1]
