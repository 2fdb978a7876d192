"""Parity at the full workload sizes, in the launch configuration the
benchmark times (same block calls, chunk counts and streams).

The oracle cannot run these layers whole in fp64, so it checks sampled
outputs it can compute one by one: token rows for everything that is
row-local (all forward outputs and the input gradients), and columns of
dW / db (each column is a product over all tokens)."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2301_08658_amd as atp
import synth_inputs as S
from helpers import (LIN, assert_close, group_table, make_block_inputs, oracle_block_fwd,
                     run_block_bwd, run_block_fwd)

pytestmark = pytest.mark.gpu

BIG = [k for k in S.WORKLOADS if not k.startswith("tiny")]


def _rows(T, chunks, n=8, seed=0):
    """Sampled token rows: the first and last row, chunk edges, and random rows."""
    rng = np.random.default_rng(seed)
    mc = T // chunks
    edge = {0, T - 1, mc - 1, mc, T - mc}
    extra = set(rng.choice(T, size=n, replace=False).tolist())
    return sorted(r for r in edge | extra if 0 <= r < T)


def _cols(n_loc, n=4, seed=1):
    rng = np.random.default_rng(seed)
    return sorted(set([0, n_loc - 1] + rng.choice(n_loc, size=n, replace=False).tolist()))


@pytest.mark.parametrize("workspace", [False, True], ids=["direct", "workspace"])
@pytest.mark.parametrize("name", BIG)
def test_workload_forward_sampled_rows(name, workspace):
    w = S.WORKLOADS[name]
    d1, d2 = w["mesh"]
    coord = (d1 - 1, d2 - 1)
    inp = make_block_inputs(w["mode"], w["mesh"], coord, w["tokens"], w["h"], w["sigma_w"],
                            seed=11, on_device=True)
    print(f"[{name}] forward, coord {coord}, workspace {workspace}", flush=True)
    out = run_block_fwd(inp, w["chunks"], workspace=workspace)
    torch.cuda.synchronize()
    rows = _rows(w["tokens"], w["chunks"])
    ref = oracle_block_fwd(O, inp, rows)
    for key in ("qkv", "o", "h", "pre", "z"):
        assert_close(out[key][rows], ref[key], f"{name} {key}")


def _oracle_bwd_sampled(inp, rows, cols):
    """Oracle backward of the device share on sampled rows (input gradients)
    and sampled columns (dW, db)."""
    cpu = lambda t: t.detach().cpu()  # noqa: E731
    G = inp["G"]
    W = [cpu(t) for t in inp["w"]]
    x, a, hs, pres = cpu(inp["x"]), cpu(inp["a"]), cpu(inp["hs"]), cpu(inp["pres"])
    dz, dq, do = cpu(inp["dz"]), cpu(inp["dqkv"]), cpu(inp["do"])
    peers = [[cpu(p) for p in inp["dx_peers"][i]] for i in range(4)]

    def red(i, own, sel_rows=None, sel_cols=None, epi=O.EPI_NONE, pre=None):
        ps = peers[i]
        if sel_rows is not None:
            ps = [p[sel_rows] for p in ps]
        if sel_cols is not None:
            ps = [p[:, sel_cols] for p in ps]
        return O.partial_reduce(group_table(own, ps, G[i].bwd_index), None, epi, pre)[0]

    r = {}
    dh_rows = red(3, O.matmul(dz[rows], W[3].T), sel_rows=rows, epi=O.EPI_GELU_BWD,
                  pre=pres[rows])
    r["dh_pre"] = dh_rows
    # fc1's backward reads dh_pre as a 16-bit tensor (Sec. 5)
    r["dx_fc1"] = red(2, O.matmul(O.round_bf16(dh_rows), W[2].T), sel_rows=rows)
    r["d_attn"] = red(1, O.matmul(do[rows], W[1].T), sel_rows=rows)
    r["dx_qkv"] = red(0, O.matmul(dq[rows], W[0].T), sel_rows=rows)
    c3, c2, c1, c0 = cols
    r["dw3"] = O.matmul(hs.T, dz[:, c3])
    r["db3"] = O.colsum(dz[:, c3])
    # fc1's dY columns over all tokens: (dz W2^T)[:, c2] reduced, times GeLU'(pre)
    dh_c = red(3, O.matmul(dz, W[3][c2, :].T), sel_cols=c2, epi=O.EPI_GELU_BWD,
               pre=pres[:, c2])
    r["dw2"] = O.matmul(x.T, O.round_bf16(dh_c))
    r["db2"] = O.colsum(dh_c)
    r["dw1"] = O.matmul(a.T, do[:, c1])
    r["db1"] = O.colsum(do[:, c1])
    r["dw0"] = O.matmul(x.T, dq[:, c0])
    r["db0"] = O.colsum(dq[:, c0])
    return r


@pytest.mark.parametrize("workspace", [False, True], ids=["direct", "workspace"])
@pytest.mark.parametrize("name", [k for k in BIG if S.WORKLOADS[k]["bwd"]])
def test_workload_backward_sampled(name, workspace):
    w = S.WORKLOADS[name]
    d1, d2 = w["mesh"]
    coord = (0, d2 - 1)
    inp = make_block_inputs(w["mode"], w["mesh"], coord, w["tokens"], w["h"], w["sigma_w"],
                            seed=12, on_device=True, bwd=True)
    print(f"[{name}] backward, coord {coord}, workspace {workspace}", flush=True)
    out = run_block_bwd(inp, w["chunks"], workspace=workspace)
    torch.cuda.synchronize()
    rows = _rows(w["tokens"], w["chunks"], n=6)
    cols = [_cols(g.n_loc, n=3, seed=i) for i, g in enumerate(inp["G"])]
    ref = _oracle_bwd_sampled(inp, rows, (cols[3], cols[2], cols[1], cols[0]))
    for key in ("dh_pre", "dx_fc1", "d_attn", "dx_qkv"):
        assert_close(out[key][rows], ref[key], f"{name} {key}")
    for i in range(4):
        fl = "rms" if LIN[i] == "fc1" else 1.0    # token-sums of the bf16 dh_pre
        assert_close(out["dw"][i][:, cols[i]], ref[f"dw{i}"], f"{name} dw_{LIN[i]}", floor=fl)
        assert_close(out["db"][i][cols[i]], ref[f"db{i}"], f"{name} db_{LIN[i]}", floor=fl)


def test_literal_row_first_fc1_shape():
    """The GPT-3-shaped workload's stated fc1 shape 2048 x 3072 x 24576 is the
    row-first fc1 on mesh 4x2 (K/d1 = 12288/4, N/d2 = 49152/2)."""
    T, h, chunks = 2048, 12288, 4
    m = atp.mesh(4, 2, 1, 1)
    g = atp.atp_shard_geometry(m, atp.ATP_ROW_FIRST, h, 4 * h)
    assert (g.k_loc, g.n_loc, g.red_size) == (3072, 24576, 4)
    dev = "cuda:0"
    x = S.randn_device((T, g.k_loc), 1.0, 13, 1, dev)
    wt = S.randn_device((g.k_loc, g.n_loc), 0.02, 13, 2, dev)
    y = torch.empty((T, g.n_loc), device=dev)
    atp.atp_shard_linear_fwd(m, atp.ATP_ROW_FIRST, T, h, 4 * h, chunks, x, wt, None, 0, y)
    torch.cuda.synchronize()
    rows = _rows(T, chunks)
    ref = O.matmul(x[rows].cpu(), wt.cpu())
    assert_close(y[rows], ref, "row-first fc1 partial")
