"""Parity at the full workload sizes, in the launch configuration the
benchmark times (same block calls, chunk counts and streams), against the
strict fp64 oracle with the derived terms of the GPU's 16-bit handoffs
(tests/bounds.py).  Every output buffer starts as NaN, so an element a
kernel never wrote fails.

* The two h = 4096 GPT layers (2 x 4 column-first forward; 4 x 2 row-first
  forward and backward) are checked on their whole outputs, the row-first
  layer at every chunk count of its sweep (Sec. 4.1; Table 3 runs 1, 2 and 4
  chunks).  The oracle runs once per layer and serves every GPU run.
* The GPT-3-shaped layer and the two h = 20480 layers are too large for an
  fp64 CPU pass in a test: the oracle checks 256 seeded token rows of every
  row-local output (rows are independent in every step; the chunk edges are
  among them) and 32 seeded columns of each dW and db (a column is a sum
  over all tokens)."""
import functools

import numpy as np
import pytest
import torch

import bounds
import oracle as O
import paper_2301_08658_amd as atp
import synth_inputs as S
from helpers import (LIN, assert_close, check_bwd, check_fwd, group_table, make_block_inputs,
                     oracle_block_bwd, oracle_block_fwd, run_block_bwd, run_block_fwd)

pytestmark = pytest.mark.gpu

FULL = ("gpt_h4096_col_2x4", "gpt_h4096_row_4x2")
SAMPLED = ("gpt3_h12288_col_4x2", "wide_h20480_col_8x1", "wide_h20480_col_2x4")
N_ROWS, N_COLS = 256, 32


def _rows(T, chunks, n=N_ROWS, seed=0):
    """Seeded token rows: the first and last row, every chunk edge of the
    chunk counts 1..8, and random rows up to n."""
    rng = np.random.default_rng(seed)
    edge = {0, T - 1}
    for c in (2, 4, 8, chunks):
        mc = T // c
        edge |= {k * mc for k in range(c)} | {k * mc - 1 for k in range(1, c + 1)}
    edge = {r for r in edge if 0 <= r < T}
    rest = [r for r in rng.permutation(T).tolist() if r not in edge][:max(0, n - len(edge))]
    return sorted(edge | set(rest))


def _cols(n_loc, n=N_COLS, seed=1):
    rng = np.random.default_rng(seed)
    rest = [c for c in rng.permutation(n_loc).tolist() if c not in (0, n_loc - 1)]
    return sorted([0, n_loc - 1] + rest[:n - 2])


def _inputs(name, seed, bwd):
    w = S.WORKLOADS[name]
    d1, d2 = w["mesh"]
    coord = (d1 - 1, d2 - 1) if not bwd else (0, d2 - 1)
    return w, make_block_inputs(w["mode"], w["mesh"], coord, w["tokens"], w["h"], w["sigma_w"],
                                seed=seed, on_device=True, bwd=bwd)


# ------------------------------------------------------------------ whole outputs
@functools.lru_cache(maxsize=2)
def _full_case(name):
    """Inputs and the oracle's whole forward (and backward) of the layer,
    computed once for every GPU run of it."""
    has_bwd = S.WORKLOADS[name]["bwd"]
    w, inp = _inputs(name, 31, has_bwd)
    print(f"[{name}] oracle, whole outputs", flush=True)
    fwd = oracle_block_fwd(O, inp)
    bwd = oracle_block_bwd(O, inp) if has_bwd else None
    return w, inp, fwd, bwd


@pytest.fixture(scope="module", autouse=True)
def _release_cached_oracle():
    yield
    _full_case.cache_clear()


def _full_cases():
    """(workload, workspace, chunks): both paths at the workload's chunk
    count, and the workspace path (the benchmark's) at every chunk count of
    its sweep; one workload's cases stay together so its oracle is reused."""
    cases = []
    for name in FULL:
        w = S.WORKLOADS[name]
        cases.append((name, False, w["chunks"]))
        for c in w.get("chunk_sweep", (w["chunks"],)):
            cases.append((name, True, c))
    return cases


@pytest.mark.parametrize("case", _full_cases(),
                         ids=lambda c: f"{c[0]}-{'workspace' if c[1] else 'direct'}-c{c[2]}")
def test_workload_whole_outputs(case):
    name, workspace, chunks = case
    w, inp, fwd, bwd = _full_case(name)
    print(f"[{name}] whole outputs, chunks {chunks}, workspace {workspace}", flush=True)
    out = run_block_fwd(inp, chunks, workspace=workspace)
    torch.cuda.synchronize()
    check_fwd(out, *fwd, what=f"{name} c={chunks}")
    del out
    if bwd is not None:
        bout = run_block_bwd(inp, chunks, workspace=workspace)
        torch.cuda.synchronize()
        check_bwd(bout, *bwd, what=f"{name} c={chunks}")


# ------------------------------------------------------------------ sampled
@pytest.mark.parametrize("workspace", [False, True], ids=["direct", "workspace"])
@pytest.mark.parametrize("name", SAMPLED)
def test_workload_forward_sampled_rows(name, workspace):
    w, inp = _inputs(name, 11, False)
    print(f"[{name}] forward, workspace {workspace}", flush=True)
    out = run_block_fwd(inp, w["chunks"], workspace=workspace)
    torch.cuda.synchronize()
    rows = _rows(w["tokens"], w["chunks"])
    check_fwd(out, *oracle_block_fwd(O, inp, rows), rows=rows, what=name)


def _oracle_bwd_sampled(inp, rows, cols):
    """Strict oracle backward of the device share on sampled rows (input
    gradients) and sampled columns (dW, db), with the derived terms of the
    bf16 dh_pre that fc1's backward reads."""
    cpu = lambda t: t.detach().cpu()  # noqa: E731
    G = inp["G"]
    W = [O._f64(cpu(t)) for t in inp["wkn"]]
    x, a, hs, pres = (O._f64(cpu(inp[k])) for k in ("x", "a", "hs", "pres"))
    dz, dq, do = (O._f64(cpu(inp[k])) for k in ("dz", "dqkv", "do"))
    peers = [[cpu(p) for p in inp["dx_peers"][i]] for i in range(4)]

    def red(i, own, sel_rows=None, sel_cols=None, epi=O.EPI_NONE, pre=None):
        ps = peers[i]
        if sel_rows is not None:
            ps = [p[sel_rows] for p in ps]
        if sel_cols is not None:
            ps = [p[:, sel_cols] for p in ps]
        return O.partial_reduce(group_table(own, ps, G[i].bwd_index), None, epi, pre)[0]

    r, e = {}, {}
    dh_rows = red(3, O.matmul(dz[rows], W[3].T), sel_rows=rows, epi=O.EPI_GELU_BWD,
                  pre=pres[rows])
    r["dh_pre"] = dh_rows
    r["dx_fc1"] = red(2, O.matmul(dh_rows, W[2].T), sel_rows=rows)
    e["dx_fc1"] = bounds.left(bounds.rounding_var(dh_rows), W[2].T)
    r["da"] = red(1, O.matmul(do[rows], W[1].T), sel_rows=rows)
    r["dx_qkv"] = red(0, O.matmul(dq[rows], W[0].T), sel_rows=rows)
    c3, c2, c1, c0 = cols
    r["dw_fc2"] = O.matmul(hs.T, dz[:, c3])
    r["db_fc2"] = O.colsum(dz[:, c3])
    # fc1's dY columns over all tokens: (dz W2^T)[:, c2] reduced, times GeLU'(pre)
    dh_c = red(3, O.matmul(dz, W[3][c2, :].T), sel_cols=c2, epi=O.EPI_GELU_BWD,
               pre=pres[:, c2])
    r["dw_fc1"] = O.matmul(x.T, dh_c)
    r["db_fc1"] = O.colsum(dh_c)
    e["dw_fc1"] = bounds.right(x, bounds.rounding_var(dh_c))
    e["db_fc1"] = bounds.colsum(bounds.rounding_var(dh_c))
    r["dw_out"] = O.matmul(a.T, do[:, c1])
    r["db_out"] = O.colsum(do[:, c1])
    r["dw_qkv"] = O.matmul(x.T, dq[:, c0])
    r["db_qkv"] = O.colsum(dq[:, c0])
    return r, e


@pytest.mark.parametrize("workspace", [False, True], ids=["direct", "workspace"])
@pytest.mark.parametrize("name", SAMPLED)
def test_workload_backward_sampled(name, workspace):
    w, inp = _inputs(name, 12, True)
    print(f"[{name}] backward, workspace {workspace}", flush=True)
    out = run_block_bwd(inp, w["chunks"], workspace=workspace)
    torch.cuda.synchronize()
    rows = _rows(w["tokens"], w["chunks"], seed=2)
    cols = [_cols(g.n_loc, seed=3 + i) for i, g in enumerate(inp["G"])]
    ref, extra = _oracle_bwd_sampled(inp, rows, (cols[3], cols[2], cols[1], cols[0]))
    for key in ("dh_pre", "dx_fc1", "d_attn", "dx_qkv"):
        rk = {"d_attn": "da"}.get(key, key)
        assert_close(out[key][rows], ref[rk], f"{name} {key}", extra=extra.get(rk))
    for i, n in enumerate(LIN):
        assert_close(out["dw_kn"][i][:, cols[i]], ref[f"dw_{n}"], f"{name} dw_{n}",
                     extra=extra.get(f"dw_{n}"))
        assert_close(out["db"][i][cols[i]], ref[f"db_{n}"], f"{name} db_{n}",
                     extra=extra.get(f"db_{n}"))


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
    y = torch.full((T, g.n_loc), float("nan"), device=dev)
    atp.atp_shard_linear_fwd(m, atp.ATP_ROW_FIRST, T, h, 4 * h, chunks, x, wt, None, 0, y)
    torch.cuda.synchronize()
    rows = _rows(T, chunks)
    ref = O.matmul(x[rows].cpu(), wt.cpu())
    assert_close(y[rows], ref, "row-first fc1 partial")
