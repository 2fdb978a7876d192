"""GPU parity of the whole shard block (Sec. 3.2.1 forward, Sec. 4.2
backward) with chunk-based overlapping (Sec. 4.1).

* bench mode: the other group members' partial buffers are seeded inputs;
  the oracle receives the same buffers.
* mesh simulation: every coordinate of the mesh is run on the one GPU with
  the true partials of its group members; the reduced blocks must equal the
  unsharded layer (the spec invariant) and be identical bit for bit
  across each reduction group.
* chunking, stream overlap and the ROW/COL transposition never change a bit
  (on the workspace path chunking keeps the bits while every chunk product
  keeps its split-K plan, as it does for the shapes here).
* full-size workloads are checked on sampled token rows (rows are
  independent in every step) and, for dW, on sampled columns.
"""
import itertools

import numpy as np
import pytest
import torch

import oracle as O
import paper_2301_08658_amd as atp
import synth_inputs as S
import bounds
from helpers import (DEV, LIN, assert_close, block_mode_code, check_bwd, check_fwd,
                     make_block_inputs, oracle_block_bwd, oracle_block_fwd, run_block_bwd,
                     run_block_fwd, to64)

pytestmark = pytest.mark.gpu

TINY = S.WORKLOADS["tiny_mlp_h512_col_2x2"]


# ------------------------------------------------------------------ tiny, bench mode
@pytest.mark.parametrize("mode", ["col", "row"])
@pytest.mark.parametrize("bias_std", [0.0, 0.02])
def test_block_fwd_tiny_every_coordinate(mode, bias_std):
    w = TINY
    d1, d2 = w["mesh"]
    for coord in itertools.product(range(d1), range(d2)):
        inp = make_block_inputs(mode, w["mesh"], coord, w["tokens"], w["h"], w["sigma_w"],
                                seed=1, bias_std=bias_std)
        out = run_block_fwd(inp, w["chunks"])
        torch.cuda.synchronize()
        ref, extra = oracle_block_fwd(O, inp)
        check_fwd(out, ref, extra, what=f"{mode} {coord}")
        # the own partial buffer holds x_loc @ w_loc (fc2's input is a GPU
        # output, so only the three linears fed by seeded inputs are checked)
        for i, g in enumerate(inp["G"][:3]):
            if g.red_size > 1:
                xin = inp["a"] if i == 1 else inp["x"]
                assert_close(out["own"][i], O.matmul(xin.cpu(), inp["wkn"][i].cpu()),
                             f"own partial {LIN[i]}")


@pytest.mark.parametrize("mesh", [(1, 1), (1, 4), (4, 1), (3, 2)])
def test_block_fwd_degenerate_meshes(mesh):
    """Groups of one (bias/GeLU fused in the GEMM), Megatron's (N,1) mesh and
    a non-power-of-two mesh."""
    T, h = 96, 384 if mesh != (3, 2) else 768
    for coord in [(0, 0), (mesh[0] - 1, mesh[1] - 1)]:
        inp = make_block_inputs("col", mesh, coord, T, h, 0.02, seed=2)
        out = run_block_fwd(inp, 2)
        torch.cuda.synchronize()
        check_fwd(out, *oracle_block_fwd(O, inp), what=f"{mesh} {coord}")


# ------------------------------------------------------------------ mesh simulation
def _simulate_mesh(mode, mesh, T, h, chunks, X, A, W, B):
    """Run every coordinate's share on the one GPU with true peer partials.
    Returns {coord: outputs}."""
    d1, d2 = mesh
    bm = block_mode_code(mode)
    coords = list(itertools.product(range(d1), range(d2)))
    omodes = O.block_linear_modes(O.BLOCK_COL if mode == "col" else O.BLOCK_ROW)
    loc = {}
    for c in coords:
        m = atp.mesh(d1, d2, *c)
        G = atp.block_geometry(m, bm, h)
        xs, _, _ = O.linear_specs(omodes["qkv"])
        xr = O.spec_block(mesh, c, xs, (T, h))[1]
        xo, _, _ = O.linear_specs(omodes["out"])
        ar = O.spec_block(mesh, c, xo, (T, h))[1]
        w = [W[n][g.k_off:g.k_off + g.k_loc, g.n_off:g.n_off + g.n_loc].contiguous().to(DEV)
             for g, n in zip(G, LIN)]
        b = [B[n][g.n_off:g.n_off + g.n_loc].contiguous().to(DEV) for g, n in zip(G, LIN)]
        loc[c] = dict(m=m, G=G, x=X[:, xr[0]:xr[1]].contiguous().to(DEV),
                      a=A[:, ar[0]:ar[1]].contiguous().to(DEV), w=w, b=b)
    part = {c: [torch.empty((T, g.n_loc), device=DEV) for g in loc[c]["G"]] for c in coords}
    # phase 1: partials of qkv, out, fc1 on every device
    for c in coords:
        L = loc[c]
        for i, xin in ((0, L["x"]), (1, L["a"]), (2, L["x"])):
            g = L["G"][i]
            mode_i = atp.ATP_COL_FIRST if g.red_axis == 1 else atp.ATP_ROW_FIRST
            if g.red_size > 1:
                atp.atp_shard_linear_fwd(L["m"], mode_i, T, *(h, h, h)[i:i + 1],
                                         (3 * h, h, 4 * h)[i], chunks, xin, L["w"][i], None, 0,
                                         part[c][i])

    def group(c, g):
        return [tuple(c[:g.red_axis]) + (j,) + tuple(c[g.red_axis + 1:])
                for j in range(g.red_size)]

    # phase 2: every device's reduced H (fc1), then its fc2 partial
    Hd = {}
    for c in coords:
        L = loc[c]
        g = L["G"][2]
        Hd[c] = torch.empty((T, g.n_loc), dtype=torch.bfloat16, device=DEV)
        if g.red_size > 1:
            atp.atp_chunked_partial_reduce(g.red_size, T, g.n_loc, chunks,
                                           [part[p][2] for p in group(c, g)], L["b"][2],
                                           atp.ATP_EPI_BIAS_GELU, Hd[c])
        else:
            mode_i = atp.ATP_COL_FIRST if g.red_axis == 1 else atp.ATP_ROW_FIRST
            atp.atp_shard_linear_fwd(L["m"], mode_i, T, h, 4 * h, chunks, L["x"], L["w"][2],
                                     L["b"][2], atp.ATP_EPI_BIAS_GELU, Hd[c])
    for c in coords:
        L = loc[c]
        g = L["G"][3]
        if g.red_size > 1:
            mode_i = atp.ATP_COL_FIRST if g.red_axis == 1 else atp.ATP_ROW_FIRST
            atp.atp_shard_linear_fwd(L["m"], mode_i, T, 4 * h, h, chunks, Hd[c], L["w"][3], None,
                                     0, part[c][3])
    # phase 3: the block call on every device, with the true group tables
    res = {}
    for c in coords:
        L = loc[c]
        G = L["G"]
        tabs = [[part[p][i] for p in group(c, G[i])] if G[i].red_size > 1 else None
                for i in range(4)]
        out = dict(qkv=torch.empty((T, G[0].n_loc), dtype=torch.bfloat16, device=DEV),
                   o=torch.empty((T, G[1].n_loc), dtype=torch.bfloat16, device=DEV),
                   h=torch.empty((T, G[2].n_loc), dtype=torch.bfloat16, device=DEV),
                   pre=torch.empty((T, G[2].n_loc), dtype=torch.bfloat16, device=DEV),
                   z=torch.empty((T, G[3].n_loc), dtype=torch.bfloat16, device=DEV))
        atp.atp_block_fwd(L["m"], bm, T, h, chunks, L["w"], L["b"], L["x"], L["a"], tabs,
                          out["qkv"], out["o"], out["h"], out["pre"], out["z"],
                          comm_stream=torch.cuda.Stream())
        torch.cuda.synchronize()
        res[c] = out
    return res


@pytest.mark.parametrize("mode,mesh", [("col", (2, 2)), ("row", (2, 2)), ("col", (2, 4)),
                                       ("row", (4, 2))])
def test_mesh_simulation_equals_unsharded_layer(mode, mesh):
    T, h = 256, 512
    shapes = O.block_shapes(h)
    X = S.randn_bf16((T, h), 1.0, 3, 1)
    A = S.randn_bf16((T, h), 1.0, 3, 2)
    W = {n: S.randn_bf16(shapes[n], 0.02, 3, 10 + i) for i, n in enumerate(LIN)}
    B = {n: S.randn_bf16((shapes[n][1],), 0.02, 3, 20 + i) for i, n in enumerate(LIN)}
    res = _simulate_mesh(mode, mesh, T, h, 2, X, A, W, B)
    bm = O.BLOCK_COL if mode == "col" else O.BLOCK_ROW
    # fc2 reads every group member's bf16 H: z carries the rounding of the
    # whole H row through all of W2 (derived from the reference's own H)
    H = O.gelu(O.matmul(X, W["fc1"]) + O._f64(B["fc1"])[None, :])
    z_extra = bounds.left(bounds.rounding_var(H), O._f64(W["fc2"]))
    zs = O.linear_specs(O.block_linear_modes(bm)["fc2"])[2]
    zs = tuple(O.REPLICATE if p == O.PARTIAL_SUM else p for p in zs)
    for c, out in res.items():
        ref = O.block_fwd_global(bm, mesh, c, X, A, W, B)
        extra = dict(z=O.local_tensor(z_extra, mesh, c, zs))
        check_fwd(out, ref, extra, what=f"{mode} {mesh} {c}")
    # every member of a reduction group holds the same bits
    G0 = atp.block_geometry(atp.mesh(*mesh, 0, 0), block_mode_code(mode), h)
    for key, i in (("qkv", 0), ("o", 1), ("h", 2), ("z", 3)):
        axis = G0[i].red_axis
        for c in res:
            c2 = list(c)
            c2[axis] = (c[axis] + 1) % mesh[axis]
            assert torch.equal(res[c][key], res[tuple(c2)][key]), (key, c, c2)


# ------------------------------------------------------------------ invariances
@pytest.mark.parametrize("workspace", [False, True], ids=["direct", "workspace"])
def test_chunk_count_never_changes_a_bit(workspace):
    base = None
    inp = make_block_inputs("col", (2, 4), (1, 2), 512, 1024, 0.02, seed=4)
    for chunks in (1, 2, 4, 8):
        out = run_block_fwd(inp, chunks, workspace=workspace)
        torch.cuda.synchronize()
        if base is None:
            base = out
            continue
        for key in ("qkv", "o", "h", "pre", "z"):
            assert torch.equal(out[key], base[key]), (chunks, key)


@pytest.mark.parametrize("mode,mesh,coord", [("row", (4, 2), (3, 1)), ("col", (8, 1), (5, 0)),
                                             ("col", (1, 4), (0, 2))])
def test_serialized_equals_pipelined(mode, mesh, coord):
    """One stream, and compute + comm streams, give the same bits (groups of
    one and of several members)."""
    inp = make_block_inputs(mode, mesh, coord, 512, 1024, 0.02, seed=5, bwd=True)
    runs = [dict(same_stream=True), dict()]
    fw = [run_block_fwd(inp, 4, **kw) for kw in runs]
    torch.cuda.synchronize()
    for other in fw[1:]:
        for key in ("qkv", "o", "h", "pre", "z"):
            assert torch.equal(fw[0][key], other[key]), key
    bw = [run_block_bwd(inp, 4, **kw) for kw in runs]
    torch.cuda.synchronize()
    for other in bw[1:]:
        for key in ("dh_pre", "dx_qkv", "dx_fc1", "d_attn"):
            assert torch.equal(bw[0][key], other[key]), key
        for i in range(4):
            assert torch.equal(bw[0]["dw"][i], other["dw"][i])
            assert torch.equal(bw[0]["db"][i], other["db"][i])


def test_row_on_transposed_mesh_equals_col():
    """ROW on (4,2) at (i1,i2) has the local shapes and groups of COL on (2,4)
    at (i2,i1); fed the same local data the outputs match bit for bit."""
    T, h = 512, 1024
    for (i1, i2) in [(0, 0), (3, 1), (2, 0)]:
        a = make_block_inputs("row", (4, 2), (i1, i2), T, h, 0.02, seed=6)
        b = make_block_inputs("col", (2, 4), (i2, i1), T, h, 0.02, seed=6)
        for key in ("x", "a"):
            assert torch.equal(a[key], b[key])
        oa = run_block_fwd(a, 4)
        ob = run_block_fwd(b, 4)
        torch.cuda.synchronize()
        for key in ("qkv", "o", "h", "pre", "z"):
            assert torch.equal(oa[key], ob[key]), key


# ------------------------------------------------------------------ backward
@pytest.mark.parametrize("workspace", [False, True], ids=["direct", "workspace"])
@pytest.mark.parametrize("mode,mesh,coord", [("col", (2, 2), (1, 0)), ("row", (2, 4), (1, 3)),
                                             ("col", (4, 1), (2, 0))])
def test_block_fwd_bwd_integer_chain_bit_exact(mode, mesh, coord, workspace):
    """Integer inputs, integer peers and pre = 0 (GeLU'(0) = 1/2 exactly): every
    value before a bf16 store is exact on both sides, so the chained backward
    (fc2 dX -> reduce * GeLU' -> fc1 dX / dW) must match bit for bit, with the
    oracle's bf16-stored outputs rounded the same way."""
    inp = make_block_inputs(mode, mesh, coord, 192, 256, 0.0, seed=10, bwd=True, integer=True)
    out = run_block_bwd(inp, 2, workspace=workspace)
    torch.cuda.synchronize()
    # the oracle's diagnostic mirror rounds fc1's dY to bf16 as the GPU
    # stores it, so every value of this integer chain is exact on both sides
    ref, _ = oracle_block_bwd(O, inp, round_dpre=O.round_bf16)
    for key in ("dh_pre", "dx_qkv", "dx_fc1", "d_attn"):
        rk = {"d_attn": "da"}.get(key, key)
        np.testing.assert_array_equal(to64(out[key]), O.round_bf16(ref[rk]), err_msg=key)
    for i, n in enumerate(LIN):
        np.testing.assert_array_equal(to64(out["dw"][i]), ref["dw_" + n], err_msg=n)
        np.testing.assert_array_equal(to64(out["db"][i]), ref["db_" + n], err_msg=n)


@pytest.mark.parametrize("workspace", [False, True], ids=["direct", "workspace"])
@pytest.mark.parametrize("mode", ["col", "row"])
def test_block_bwd_tiny_every_coordinate(mode, workspace):
    w = TINY
    d1, d2 = w["mesh"]
    for coord in itertools.product(range(d1), range(d2)):
        inp = make_block_inputs(mode, w["mesh"], coord, w["tokens"], w["h"], w["sigma_w"],
                                seed=7, bwd=True)
        out = run_block_bwd(inp, w["chunks"], workspace=workspace)
        torch.cuda.synchronize()
        check_bwd(out, *oracle_block_bwd(O, inp), what=f"{mode} {coord}")


@pytest.mark.parametrize("mesh", [(1, 1), (4, 1), (1, 4)])
def test_block_bwd_groups_of_one(mesh):
    inp = make_block_inputs("col", mesh, (0, 0), 128, 256, 0.02, seed=8, bwd=True)
    out = run_block_bwd(inp, 2)
    torch.cuda.synchronize()
    check_bwd(out, *oracle_block_bwd(O, inp), what=f"{mesh}")


@pytest.mark.parametrize("workspace", [False, True], ids=["direct", "workspace"])
def test_block_bwd_chunk_invariance(workspace):
    inp = make_block_inputs("col", (2, 4), (1, 3), 512, 1024, 0.02, seed=9, bwd=True)
    base = run_block_bwd(inp, 1, workspace=workspace)
    for chunks in (2, 4, 8):
        out = run_block_bwd(inp, chunks, workspace=workspace)
        torch.cuda.synchronize()
        for key in ("dh_pre", "dx_qkv", "dx_fc1", "d_attn"):
            assert torch.equal(out[key], base[key]), (chunks, key)
        for i in range(4):
            assert torch.equal(out["dw"][i], base["dw"][i])


@pytest.mark.parametrize("workspace", [False, True], ids=["direct", "workspace"])
def test_block_without_tokens(workspace):
    """No tokens: the forward has nothing to write; dW and db are sums over no
    tokens, so they must come back as exact zeros (the buffers start as NaN)."""
    print(f"block without tokens workspace={workspace}", flush=True)
    inp = make_block_inputs("col", (2, 2), (1, 0), 0, 512, 0.02, seed=92, bwd=True)
    run_block_fwd(inp, 2, workspace=workspace)
    out = run_block_bwd(inp, 2, workspace=workspace)
    torch.cuda.synchronize()
    for i, n in enumerate(LIN):
        assert torch.all(out["dw"][i] == 0), f"dw_{n}"
        assert torch.all(out["db"][i] == 0), f"db_{n}"


# ------------------------------------------------------------------ options
def _bits(t):
    return t.contiguous().view(torch.int16 if t.element_size() == 2 else torch.int32)


OPT_CASES = [("col", (2, 4), (1, 2), 512, 1024, 4), ("row", (2, 2), (1, 0), 256, 512, 2),
             ("col", (8, 1), (3, 0), 256, 2048, 2), ("col", (2, 2), (0, 1), 256, 2000, 2)]
OPT_IDS = [f"{c[0]}{c[1][0]}x{c[1][1]}_h{c[4]}" for c in OPT_CASES]


@pytest.mark.parametrize("workspace", [False, True], ids=["direct", "workspace"])
@pytest.mark.parametrize("case", OPT_CASES, ids=OPT_IDS)
def test_weights_stored_nk(case, workspace):
    """Weights kept as [n_loc, k_loc] (torch.nn.Linear's order): the forward
    reads them as they are, the backward's dX reads them directly or from a
    [k_loc, n_loc] copy in the workspace, and dW comes back as [n_loc, k_loc].
    Every product sums in the same order as with [k_loc, n_loc] weights, so
    the two layouts give the same bits; both match the oracle."""
    mode, mesh, coord, T, h, chunks = case
    print(f"nk weights {case} workspace={workspace}", flush=True)
    kn = make_block_inputs(mode, mesh, coord, T, h, 0.02, seed=61, bwd=True)
    nk = make_block_inputs(mode, mesh, coord, T, h, 0.02, seed=61, bwd=True,
                           layout=atp.ATP_W_NK)
    fa, fb = run_block_fwd(kn, chunks, workspace=workspace), run_block_fwd(nk, chunks,
                                                                           workspace=workspace)
    ba, bb = run_block_bwd(kn, chunks, workspace=workspace), run_block_bwd(nk, chunks,
                                                                           workspace=workspace)
    torch.cuda.synchronize()
    for key in ("qkv", "o", "h", "pre", "z"):
        assert torch.equal(_bits(fa[key]), _bits(fb[key])), key
    for key in ("dh_pre", "dx_qkv", "dx_fc1", "d_attn"):
        assert torch.equal(_bits(ba[key]), _bits(bb[key])), key
    for i in range(4):
        assert torch.equal(_bits(ba["db"][i]), _bits(bb["db"][i])), f"db {i}"
    check_fwd(fb, *oracle_block_fwd(O, nk), what="nk")
    check_bwd(bb, *oracle_block_bwd(O, nk), what="nk")


@pytest.mark.parametrize("workspace", [False, True], ids=["direct", "workspace"])
@pytest.mark.parametrize("case", OPT_CASES, ids=OPT_IDS)
def test_bf16_partials(case, workspace):
    """Partial(SUM) blocks in bf16 (Sec. 5's 16-bit all-reduce): the own
    partial is the product rounded once (the split slabs are summed in fp32
    first), the group's values are summed in fp32 in group order.  Checked
    against the strict fp64 oracle with the derived rounding terms, the own
    partials within one rounding, and chunking never changes a bit on the
    direct path."""
    mode, mesh, coord, T, h, chunks = case
    print(f"bf16 partials {case} workspace={workspace}", flush=True)
    inp = make_block_inputs(mode, mesh, coord, T, h, 0.02, seed=62, bwd=True,
                            partial_dtype=torch.bfloat16)
    out = run_block_fwd(inp, chunks, workspace=workspace)
    bout = run_block_bwd(inp, chunks, workspace=workspace)
    torch.cuda.synchronize()
    check_fwd(out, *oracle_block_fwd(O, inp), what="bf16 partials")
    check_bwd(bout, *oracle_block_bwd(O, inp), what="bf16 partials")
    for i, g in enumerate(inp["G"][:3]):
        if g.red_size > 1:
            xin = inp["a"] if i == 1 else inp["x"]
            ref = O.matmul(xin.cpu(), inp["wkn"][i].cpu())
            assert out["own"][i].dtype == torch.bfloat16
            assert_close(out["own"][i], ref, f"own partial {LIN[i]}", extra=bounds.single(ref))
    if not workspace:
        one = run_block_fwd(inp, 1)
        torch.cuda.synchronize()
        for key in ("qkv", "o", "h", "pre", "z"):
            assert torch.equal(_bits(one[key]), _bits(out[key])), key


def test_concurrent_calls_from_two_threads():
    """Two host threads run block calls on their own streams at the same
    time.  Each thread keeps its own synchronisation events, so every call
    gives the bits of the same call made alone."""
    import threading
    cases = [make_block_inputs("col", (2, 4), (1, 2), 512, 1024, 0.02, seed=71 + i)
             for i in range(2)]
    ref = [run_block_fwd(c, 4) for c in cases]
    torch.cuda.synchronize()
    results, errs = [None, None], []

    def worker(i):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                outs = [run_block_fwd(cases[i], 4, compute=s) for _ in range(4)]
            s.synchronize()
            results[i] = outs
        except Exception as e:  # noqa: BLE001
            errs.append(e)

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=60)
    assert not errs, errs
    for i in range(2):
        assert results[i] is not None
        for out in results[i]:
            for key in ("qkv", "o", "h", "pre", "z"):
                assert torch.equal(_bits(out[key]), _bits(ref[i][key])), (i, key)
